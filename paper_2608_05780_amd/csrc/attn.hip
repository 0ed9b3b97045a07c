// Block-sparse prefill attention for gfx950 with fused query-frame evidence
// partials.
//
// Work item = one query block (a region block of <= 64 tokens), up to two
// query heads sharing one kv head, and a run of the block's active key
// blocks (CSR). A work-group has four wavefronts: waves 0-1 take the first
// head's rows 0-31 / 32-63, waves 2-3 the second head's. Each key/value tile
// is staged once in LDS for both heads. Two work-groups fit a CU, so every
// SIMD interleaves two wavefronts and part of one's softmax VALU work hides
// under the other's MFMAs.
// A kv group with an odd number of query heads (7 for 28/4) leaves one head
// over; it runs as paired items, in which waves 2-3 take a second query
// block for the same head (the region's next block, or the same chunk of the
// video's next query-token block). The item's key tiles are the two blocks'
// lists merged, and each half computes only the tiles active for its rows.
//
// Key/value tiles go straight from global memory to LDS (16-byte
// global_load_lds per lane, no staging registers), double-buffered: tile j+1
// is in flight while tile j is computed, one barrier per tile. The K and V
// operand reads of a tile run eight ahead of the MFMAs that consume them.
// Rows are XOR-swizzled in 16-byte chunks so the MFMA operand reads below are
// free of LDS bank conflicts.
//
// Per key tile (64 keys):
//   S^T = K Q^T        32x32x16 bf16 MFMA (fp32 inputs: 32x32x2 f32 MFMA);
//                      computing the transpose leaves one query row per lane
//                      (lane % 32); a row max or sum is an in-lane reduction
//                      plus one v_permlane32_swap with lane ^ 32.
//   mask               only on tiles reaching past the first query row or
//                      shorter than 64 keys: keys after the row (causal) and
//                      past the block end.
//   online softmax     base-2 with log2(e) folded into the scale. A row's
//                      running reference m_ref is set from the exact row max
//                      of its first tile; later tiles take their
//                      probabilities against m_ref directly, with no row max,
//                      and only when one of them exceeds 2^64 (or is not
//                      finite) is the tile recomputed from the staged K tile,
//                      its row max taken and m_ref moved (accumulators
//                      rescaled). The reference is never above the true
//                      running max, so the row sum stays >= 1; fp32
//                      accumulators and bf16 P keep their relative precision
//                      at any such scale.
//   evidence           query-token rows only: the fp32 probabilities of each
//                      anchor frame's keys (frames of N_v | 64 keys never cross
//                      a tile) are summed and written once per (row, frame) as
//                      a log2 partial mass m_ref + log2(sum); non-visual keys
//                      (system prefix, query tokens) accumulate into one
//                      running partial per item.
//   O^T += V^T P^T     P rounded to bf16 (RNE) as the B operand straight from
//                      the S^T registers; the V^T operand comes from the
//                      row-major V tile through ds_read_b64_tr_b16 (LDS
//                      transpose read: within 16 lanes, lane i receives
//                      element i % 4 of the rows addressed by lanes i/4 + 4k).
//
// bf16 Q and O pass through LDS in the K-tile layout: the item's Q rows go
// by direct global -> LDS loads, as whole 256-byte rows, into the second
// buffer pair (free until the first loop iteration refills it after a
// barrier), in the same round trip as the first key/value tile (the item
// record carries the descriptors both need), and the normalised O rows are
// written back as whole rows after the last tile. Read or written straight
// from the MFMA layout, every such instruction touches 32 rows 7 KB apart,
// 16-32 bytes each.
//
// Visual and system rows finish in the kernel (O, LSE). Query-token rows are
// split into chunks of key blocks (longest-first balance across the chip);
// each chunk leaves an unnormalised partial (acc, m_ref, row sum, non-visual
// mass) in the workspace, and the combine part of combine_evidence_kernel
// merges them.
#include <algorithm>
#include <type_traits>

#include "attn_tiles.h"
#include "kernels.h"

namespace evisel {
namespace {

// ---------------------------------------------------------------------------
template <class P, int D, bool TOPP>
__global__ __attribute__((amdgpu_flat_work_group_size(kThreads, kThreads),
                          amdgpu_waves_per_eu(2, 2))) void
attn_kernel(const DevPlan pl, const Workspace ws, const AttnCall ac) {
  using T = typename P::T;
  constexpr int TB = kTile * P::RC * 16;   // bytes of one tile
  constexpr int VSWZ = sizeof(T) == 2 ? kSwzV : kSwzNone;
  __shared__ __attribute__((aligned(1024))) char smem[4 * TB];
  EV_LDS char* lds = (EV_LDS char*)smem;   // [K0 | K1 | V0 | V1]
  // top-p: CSR positions of the item's key tiles that some row retained
  __shared__ short clist[TOPP ? kMaxItemCandidates : 1];
  __shared__ int n_kept;

  const WorkItem it = pl.items[blockIdx.x];
  if (it.qblock < 0) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform
  const int l32 = lane & 31, g = lane >> 5;
  const int hsub = wave >> 1;
  // A paired item gives the second half of the work-group its own query
  // block (same head); otherwise the halves take heads head, head + 1.
  const bool uni = it.qblock2 >= 0;
  const int nhalf = uni ? 2 : it.nheads;   // halves with rows
  const bool active = hsub < nhalf;
  const int hd1 = uni ? it.head : it.head + 1;   // the second half's head
  const int h = active && hsub ? hd1 : it.head;
  const int kvh = it.head / (pl.hq / pl.hkv);
  const BlockDesc qb0 = pl.blocks[it.qblock];
  const BlockDesc qb1 = uni ? pl.blocks[it.qblock2] : qb0;
  const BlockDesc qb = hsub ? qb1 : qb0;
  const int qbid = uni && hsub ? it.qblock2 : it.qblock;   // the wave's block
  const bool is_text = it.slot >= 0;
  const int qrow = 32 * (wave & 1) + l32;
  const bool qvalid = active && qrow < qb.len;
  const int qpos = qb.start + qrow;
  int n = it.kb_end - it.kb_begin;
  const float c2 = ac.scale_log2;
  const T* kg = (const T*)ac.k;
  const T* vg = (const T*)ac.v;

  typename P::QFrag qf;
  if constexpr (!P::kStaged) P::load_q(qf, ac.q, qpos, qvalid, h, pl.hq, g);

  float m_ref = neg_inf(), l_part = 0.f, nv_part = 0.f;
  f32x16 o[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) o[i] = f32x16{};

  TileLoader<T, D, kSwzK> kload;
  TileLoader<T, D, VSWZ> vload;
  typename P::PvOff pvo;
  P::pv_offsets(pvo, lane);
  kload.init(pl.hkv, wave, lane);
  vload.init(pl.hkv, wave, lane);
  // LDS layout: [K0 | K1 | V0 | V1], tile t in buffers t % 2.
  EV_LDS char* const kbuf0 = lds;
  EV_LDS char* const vbuf0 = lds + 2 * TB;
  auto kbuf = [&](int t) { return kbuf0 + (t & 1) * TB; };
  auto vbuf = [&](int t) { return vbuf0 + (t & 1) * TB; };

  const int b0 = it.kb_begin;

  // Descriptors of this item's key tiles, 64 at a time: lane t holds the
  // BlockDesc of tile 64*batch + t, and the loop reads tile j's with
  // v_readlane. (Loading them per tile would put two dependent global round
  // trips in front of every tile's K/V loads.) dsc_pos is the tile's CSR
  // position in the row of the wave's query block (paired items: -1 when
  // the key block is not active for it).
  // Top-p: dsc_loc is the tile's local history index, or -1 when the tile
  // is always visible.
  int dsc_start = 0, dsc_len = 1, dsc_region = 0, dsc_aux = 0, dsc_loc = -1,
      dsc_pos = 0;
  auto load_batch = [&](int batch) {
    const int t = batch * 64 + lane;
    if (t < n) {
      const int pos = TOPP ? (int)clist[t] : t;
      const BlockDesc bd =
          uni ? pl.ptile_desc[b0 + pos] : pl.col_desc[b0 + pos];
      dsc_start = bd.start;
      dsc_len = bd.len;
      dsc_region = bd.region;
      dsc_aux = bd.aux;
      if (uni) {
        const PairedTile pt = pl.ptile[b0 + pos];
        dsc_pos = pt.pos[hsub];
        if (TOPP) {
          // top-p: a history block no row of this half retained is skipped
          const int loc = pl.blk_local[pt.block];
          dsc_loc = pt.block == qbid ? -1 : loc;
          if (dsc_pos >= 0 && dsc_loc >= 0 &&
              !((ws.ubits[((size_t)it.head * pl.nb + qbid) * pl.W +
                          (loc >> 5)] >> (loc & 31)) & 1u))
            dsc_pos = -1;
        }
      } else {
        dsc_pos = b0 + pos;
        if (TOPP) {
          const int bid = pl.col[b0 + pos];
          dsc_loc = bid == it.qblock ? -1 : pl.blk_local[bid];
        }
      }
    }
  };
  auto desc = [&](int t) {
    const int l = t & 63;
    BlockDesc d;
    d.start = __builtin_amdgcn_readlane(dsc_start, l);
    d.len = __builtin_amdgcn_readlane(dsc_len, l);
    d.region = __builtin_amdgcn_readlane(dsc_region, l);
    d.aux = __builtin_amdgcn_readlane(dsc_aux, l);
    return d;
  };

  // The item's Q rows go straight to the second buffer pair (K1 for the
  // first half, V1 for the second) in the K-tile layout, which the first
  // loop iteration refills only after a barrier; rows past a block's length
  // repeat its last row (their results are never stored). The query blocks
  // and the first key tile come with the item record, so these loads and
  // the first tile's start one round trip after the kernel does. Without
  // top-p the first descriptor batch is fetched in the same round trip.
  if constexpr (!TOPP) load_batch(0);
  if constexpr (P::kStaged) {
    TileLoader<T, D, kSwzK> qload;
    qload.init(pl.hq, wave, lane);
    qload.issue(kbuf(1), (const T*)ac.q, it.q0start, it.q0len, it.head, wave);
    if (nhalf > 1)
      qload.issue(vbuf(1), (const T*)ac.q, it.q1start, it.q1len, hd1, wave);
  }

  // Top-p: a candidate tile is kept when it is always visible (system
  // prefix, the query block itself) or some row of the item's heads
  // retained it; wave 0 compacts the kept CSR positions into clist.
  if constexpr (TOPP) {
    if (wave == 0) {
      const uint32_t* ub =
          ws.ubits + ((size_t)it.head * pl.nb + it.qblock) * pl.W;
      const size_t hstride = (size_t)pl.nb * pl.W;
      int base = 0;
      for (int c0 = 0; c0 < n; c0 += 64) {
        const int t = c0 + lane;
        bool keep = false;
        if (t < n && uni) {
          // paired item: kept when either half's rows need it
          const PairedTile pt = pl.ptile[b0 + t];
          const int loc = pl.blk_local[pt.block];
          for (int k = 0; k < 2; ++k) {
            const int own = k ? it.qblock2 : it.qblock;
            if (pt.pos[k] < 0) continue;
            if (loc < 0 || pt.block == own) {
              keep = true;
            } else {
              const unsigned wd =
                  ws.ubits[((size_t)it.head * pl.nb + own) * pl.W +
                           (loc >> 5)];
              keep = keep || ((wd >> (loc & 31)) & 1u);
            }
          }
        } else if (t < n) {
          const int bid = pl.col[b0 + t];
          const int loc = pl.blk_local[bid];
          if (loc < 0 || bid == it.qblock) {
            keep = true;
          } else {
            unsigned wd = 0u;
            for (int i = 0; i < it.nheads; ++i)
              wd |= ub[i * hstride + (loc >> 5)];
            keep = (wd >> (loc & 31)) & 1u;
          }
        }
        const unsigned long long m = __ballot(keep);
        const int pos = __builtin_amdgcn_mbcnt_hi(
            (unsigned)(m >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)m, 0u));
        if (keep) clist[base + pos] = (short)t;
        base += __popcll(m);
      }
      if (lane == 0) n_kept = base;
    }
    __syncthreads();
    n = __builtin_amdgcn_readfirstlane(n_kept);
  }

  // Per tile, in three parts:
  //   pre:  causal / length mask (only on tiles that need it), row max and
  //         the (rare) lazy rescale of the accumulators;
  //   main: p = exp2(s * scale - m_ref) in place, row-sum partial;
  //   post: evidence partials of query-token rows, then O^T += V^T P^T.
  // Top-p: the rows of the wave that did not retain this history block
  // (rloc >= 0) are masked whole. Only the exact path needs this; the fast
  // path below drops such rows through their exponent offset.
  auto row_mask = [&](f32x16 (&s)[2], unsigned rbit, int rloc) {
    if (TOPP && rloc >= 0) {
      const bool kept = (rbit >> (rloc & 31)) & 1u;
      if (__any(!kept)) {
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
          for (int r = 0; r < 16; ++r) s[c][r] = kept ? s[c][r] : neg_inf();
      }
    }
  };
  auto tile_mask = [&](f32x16 (&s)[2], const BlockDesc& cur) {
    if (cur.len < kTile || cur.start + cur.len - 1 > qb.start) {
      // key kl = 32c + 8(r/4) + 4g + r%4 is masked when kl >= len or
      // start + kl > qpos, i.e. when its lane-free part exceeds x
      const int x = min(qpos - cur.start, cur.len - 1) - 4 * g;
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (32 * c + 8 * (r >> 2) + (r & 3) > x) s[c][r] = neg_inf();
    }
  };
  auto tile_ref = [&](const f32x16 (&s)[2]) {
    float mx = neg_inf();
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[c][r]);
    mx = pair_max(mx);
    const float m_new = fmaxf(m_ref, mx * c2);
    const bool need = m_new > m_ref + kRescaleSlack;
    // While m_ref is -inf nothing has been accumulated yet (the item's
    // first tile with a finite score): then only the reference moves.
    const bool resc = need && m_ref != neg_inf();
    if (__any(resc)) {
      const float alpha = resc ? exp2_(m_ref - m_new) : 1.f;
      l_part *= alpha;
      nv_part *= alpha;
#pragma unroll
      for (int i = 0; i < D / 32; ++i) o[i] *= alpha;
    }
    m_ref = need ? m_new : m_ref;
  };
  auto tile_main = [&](f32x16 (&s)[2], float mu) -> float {
    float ts = 0.f;
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = exp2_(fmaf(s[c][r], c2, -mu));
        s[c][r] = p;
        ts += p;
      }
    return ts;
  };
  // query-token rows: this video's offsets (read once, outside the loop)
  SeqDesc sq{};
  if (is_text) sq = pl.seqs[it.seq];
  const int trow = qb.aux + qrow - sq.textrow0;
  float* const seg_row = ws.seg + (size_t)h * pl.segtot + sq.segbase +
                         (size_t)trow * sq.n_frames - sq.frame0;
  // Frame cues: visual rows also leave one log2 partial mass per (row, key
  // frame) of every computed visual tile, at the tile's CSR position.
  const bool vis_ff = ac.segv != nullptr && !is_text && qb.region == kVis;
  const int fpt = kTile / pl.Nv;                    // frames per key tile
  float* const segv_row =
      vis_ff ? ac.segv + (size_t)h * pl.nnz * fpt * kTile + qrow : nullptr;
  auto tile_post = [&](f32x16 (&s)[2], const BlockDesc& cur, float ts,
                       const EV_LDS char* vt, int cpos) {
    if (is_text || vis_ff) {
      const float mu = m_ref == neg_inf() ? 0.f : m_ref;
      if (cur.region == kVis && pl.Nv == kTile) {
        // one frame per key tile: its partial is the row's tile sum
        float* dst = is_text ? seg_row + cur.aux
                             : segv_row + (size_t)cpos * kTile;
        const float t = pair_sum(ts);
        if (g == 0 && qvalid) *dst = mu + log2_(t);
      } else if (cur.region == kVis) {
        // per 8-key group partial sums, completed across the lane pair
        float g8[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) g8[q] = 0.f;
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
          for (int r = 0; r < 16; ++r) g8[4 * c + (r >> 2)] += s[c][r];
#pragma unroll
        for (int q = 0; q < 8; ++q) g8[q] = pair_sum(g8[q]);
        const int lg = __builtin_ctz((unsigned)pl.Nv) - 3;  // log2(N_v / 8)
        const int nseg = kTile / pl.Nv;
        float* dst = is_text ? seg_row + cur.aux
                             : segv_row + (size_t)cpos * fpt * kTile;
        const int dstride = is_text ? 1 : kTile;
        for (int si = 0; si < nseg; ++si) {
          float t = 0.f;
#pragma unroll
          for (int q = 0; q < 8; ++q) t += (q >> lg) == si ? g8[q] : 0.f;
          if (g == 0 && qvalid && si * pl.Nv < cur.len)
            dst[si * dstride] = mu + log2_(t);
        }
      } else if (is_text) {
        nv_part += ts;
      }
    }
    P::pv(o, vt, s, pvo);
  };

  // Top-p: the row's retained-history word of a tile, fetched with the
  // tile's key/value loads.
  const uint32_t* rrow =
      TOPP ? ws.rbits + ((size_t)h * pl.nb + qbid) * pl.W * 64 + qrow
           : nullptr;
  auto row_bits = [&](int loc) -> unsigned {
    return loc < 0 ? ~0u : rrow[(size_t)(loc >> 5) * 64];
  };
  auto loc_of = [&](int t) {
    return TOPP ? __builtin_amdgcn_readlane(dsc_loc, t & 63) : -1;
  };
  auto pos_of = [&](int t) {   // CSR position of tile t for the wave's rows
    return TOPP || uni ? __builtin_amdgcn_readlane(dsc_pos, t & 63) : b0 + t;
  };

  // Tile j+1 streams into the other buffer pair while tile j is computed.
  if constexpr (TOPP) load_batch(0);
  BlockDesc kb;
  if constexpr (TOPP) {
    kb = desc(0);
  } else {
    kb.start = it.k0start;
    kb.len = it.k0len;
  }
  if (n > 0) {
    kload.issue(kbuf(0), kg, kb.start, kb.len, kvh, wave);
    vload.issue(vbuf(0), vg, kb.start, kb.len, kvh, wave);
  }
  if constexpr (!TOPP) kb = desc(0);
  int lnext = loc_of(0), pnext = pos_of(0);
  unsigned wnext = 0u;
  if (TOPP && n > 0) wnext = row_bits(lnext);
  if constexpr (P::kStaged) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();   // Q rows visible to every wave
    P::load_q_lds(qf, hsub ? vbuf(1) : kbuf(1), qrow, g);
  }
  // Tile j lives in buffer pair j % 2. The loop is unrolled by two so that
  // each copy addresses fixed buffers: their LDS offsets become instruction
  // immediates instead of a VALU add per operand read.
  auto step = [&](int j, auto parity) {
    constexpr int pb = decltype(parity)::value;
    EV_LDS char* const kc = kbuf0 + pb * TB;
    EV_LDS char* const vc = vbuf0 + pb * TB;
    EV_LDS char* const kn = kbuf0 + (1 - pb) * TB;
    EV_LDS char* const vn = vbuf0 + (1 - pb) * TB;
    const BlockDesc cur = kb;
    const int lcur = lnext, pcur = pnext;
    if (((j + 1) & 63) == 0 && j + 1 < n) load_batch((j + 1) >> 6);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    const unsigned wcur = wnext;
    __syncthreads();
    if (j + 1 < n) {
      kb = desc(j + 1);
      kload.issue(kn, kg, kb.start, kb.len, kvh, wave);
      vload.issue(vn, vg, kb.start, kb.len, kvh, wave);
      if (TOPP) {
        lnext = loc_of(j + 1);
        wnext = row_bits(lnext);
      }
      pnext = pos_of(j + 1);
    }
    if (active && pcur >= 0) {
      f32x16 s[2] = {f32x16{}, f32x16{}};
      P::qk(s, kc, qf, l32, g);
      tile_mask(s, cur);
      // Once every row of the wave has a reference, the tile's
      // probabilities are taken against it without the tile's row max; the
      // max is needed only if some probability exceeds 2^kFastSlack (or is
      // not finite), and then the tile is recomputed from the staged K tile.
      bool exact = __any(m_ref == neg_inf());
      float ts = 0.f;
      if (!exact) {
        // top-p: a row that did not retain this history block gets an
        // offset of +inf, so all its probabilities are 0
        const bool drop =
            TOPP && lcur >= 0 && !((wcur >> (lcur & 31)) & 1u);
        ts = tile_main(s, drop ? __builtin_inff() : m_ref);
        exact = __any(!(ts <= kFastBound));
        if (exact) {
          s[0] = f32x16{};
          s[1] = f32x16{};
          P::qk(s, kc, qf, l32, g);
          tile_mask(s, cur);
        }
      }
      if (exact) {
        row_mask(s, wcur, lcur);
        tile_ref(s);
        ts = tile_main(s, m_ref == neg_inf() ? 0.f : m_ref);
      }
      l_part += ts;
      tile_post(s, cur, ts, vc, pcur);
    }
  };
  for (int j = 0; j < n; j += 2) {
    step(j, std::integral_constant<int, 0>{});
    if (j + 1 < n) step(j + 1, std::integral_constant<int, 1>{});
  }
  const float l_tot = pair_sum(l_part);
  if (P::kStaged && !is_text) {
    // O rows through LDS (K0 for the first head, K1 for the second), then
    // whole-row stores by every thread of the work-group
    __syncthreads();   // every wave is done with the last tile
    if (active) P::o_to_lds(kbuf(hsub), o, qvalid ? 1.f / l_tot : 0.f, qrow, g);
    __syncthreads();
    for (int hh = 0; hh < nhalf; ++hh)
      P::o_from_lds(ac.o, kbuf(hh), hh ? qb1.start : qb0.start,
                    hh ? qb1.len : qb0.len, hh ? hd1 : it.head, pl.hq, tid);
  }
  if (!active) return;

  if (!is_text) {
    if (qvalid) {
      if constexpr (!P::kStaged) {
        const float inv = 1.f / l_tot;
#pragma unroll
        for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
          for (int r4 = 0; r4 < 4; ++r4) {
            f32x4 v = {o[mt][4 * r4] * inv, o[mt][4 * r4 + 1] * inv,
                       o[mt][4 * r4 + 2] * inv, o[mt][4 * r4 + 3] * inv};
            P::store_o(ac.o, qpos, h, pl.hq, 32 * mt + 8 * r4 + 4 * g, v);
          }
      }
      if (g == 0 && ac.lse)
        ac.lse[(size_t)h * pl.S + qpos] = (m_ref + log2_(l_tot)) * kLn2;
      if (g == 0 && ac.lse2v)
        ac.lse2v[(size_t)h * pl.S + qpos] = m_ref + log2_(l_tot);
    }
  } else {
    const float nv_tot = pair_sum(nv_part);
    const int slot =
        uni ? (hsub ? it.slot2 : it.slot) : it.slot + hsub * it.nch;
    if (qvalid) {
      float* po = ws.pO + ((size_t)slot * kTile + qrow) * D;
#pragma unroll
      for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          f32x4 v = {o[mt][4 * r4], o[mt][4 * r4 + 1], o[mt][4 * r4 + 2],
                     o[mt][4 * r4 + 3]};
          *(f32x4*)(po + 32 * mt + 8 * r4 + 4 * g) = v;
        }
      if (g == 0) {
        const size_t ix = (size_t)slot * kTile + qrow;
        ws.pM[ix] = m_ref;
        ws.pL[ix] = l_tot;
        ws.pNV[ix] = nv_tot > 0.f ? m_ref + log2_(nv_tot) : neg_inf();
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Intra-frame cue: per visual block and kv head, the probabilities among
// the tokens of each frame, P_im = exp2(s_im * scale - lse2_i) for key m <=
// query i in i's frame (the block's diagonal tile, recomputed with the same
// MFMA contraction as the attention pass and normalised by the row LSE it
// saved), summed over the kv head's query heads. The K tile is staged in
// LDS once; waves 0-1 take the even heads of each head pair, waves 2-3 the
// odd ones, the next pair's Q and LSE are fetched while the current pair is
// computed, and the two wave groups' sums are added in a fixed order. The
// result is a partial per kv head; intra_reduce_kernel adds the kv heads in
// order and divides by Hq.
template <class P, int D>
__global__ __attribute__((amdgpu_flat_work_group_size(kThreads, kThreads)))
void intra_kernel(const DevPlan pl, const Workspace ws, const AttnCall ac) {
  using T = typename P::T;
  constexpr int TB = kTile * P::RC * 16;
  constexpr int RB = 2 * 64 * 32 * 4;              // wave-pair hand-off
  // bf16: the key tile, then both heads' query rows of the current pair
  // (staged like a key tile); fp32 rows are read from global memory
  constexpr bool kStageQ = sizeof(T) == 2;
  constexpr int SM = kStageQ ? 3 * TB : (TB > RB ? TB : RB);
  static_assert(SM >= RB, "hand-off buffer");
  __shared__ __attribute__((aligned(1024))) char smem[SM];
  EV_LDS char* kt = (EV_LDS char*)smem;
  const BlockDesc qb = pl.blocks[blockIdx.x];
  if (qb.region != kVis) return;
  const int kvh = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, g = lane >> 5;
  const int qrow = 32 * (wave & 1) + l32;
  const bool qvalid = qrow < qb.len;
  const int qpos = qb.start + qrow;
  const int Nv = pl.Nv;
  const int group = pl.hq / pl.hkv;
  const int npair = (group + 1) / 2;
  const float c2 = ac.scale_log2;
  TileLoader<T, D, kSwzK> kload;
  kload.init(pl.hkv, wave, lane);
  kload.issue(kt, (const T*)ac.k, qb.start, qb.len, kvh, wave);

  f32x16 acc[2] = {f32x16{}, f32x16{}};
  // head of pair pi for this wave (or -1 past an odd group's end)
  auto head = [&](int pi) {
    const int hi = 2 * pi + (wave >> 1);
    return pi < npair && hi < group ? kvh * group + hi : -1;
  };
  auto fetch = [&](typename P::QFrag& qf, float& l2, int h) {
    if (h < 0) return;
    P::load_q(qf, ac.q, qpos, qvalid, h, pl.hq, g);
    l2 = qvalid ? ws.lse2v[(size_t)h * pl.S + qpos] : 0.f;
  };
  auto accumulate = [&](const typename P::QFrag& qf, float l2, int h) {
    if (h < 0) return;
    f32x16 s[2] = {f32x16{}, f32x16{}};
    P::qk(s, kt, qf, l32, g);
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int kl = 32 * c + 8 * (r >> 2) + 4 * g + (r & 3);
        const bool ok = qvalid && kl <= qrow && kl / Nv == qrow / Nv;
        acc[c][r] += ok ? exp2_(fmaf(s[c][r], c2, -l2)) : 0.f;
      }
  };
  if constexpr (kStageQ) {
    // pair pi's query rows: head 2 pi + s of the group to slot s, in whole
    // 16-byte chunks of each row; wave w reads slot w / 2
    EV_LDS char* qs = kt + TB;
    TileLoader<T, D, kSwzK> qload;
    qload.init(pl.hq, wave, lane);
    auto stage = [&](int pi) {
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2)
        if (pi < npair && 2 * pi + s2 < group)
          qload.issue(qs + s2 * TB, (const T*)ac.q, qb.start, qb.len,
                      kvh * group + 2 * pi + s2, wave);
    };
    stage(0);
    for (int pi = 0; pi < npair; ++pi) {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();                             // K tile, pair pi's rows
      const int h = head(pi);
      typename P::QFrag qf;
      float l2 = 0.f;
      if (h >= 0) {
        P::load_q_lds(qf, qs + (wave >> 1) * TB, qrow, g);
        l2 = qvalid ? ws.lse2v[(size_t)h * pl.S + qpos] : 0.f;
      }
      __syncthreads();                             // the slots may refill
      stage(pi + 1);
      accumulate(qf, l2, h);
    }
  } else {
    typename P::QFrag qa, qb2;
    float la = 0.f, lb = 0.f;
    fetch(qa, la, head(0));
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();                               // K tile in LDS
    for (int pi = 0; pi < npair; pi += 2) {
      fetch(qb2, lb, head(pi + 1));
      accumulate(qa, la, head(pi));
      fetch(qa, la, head(pi + 2));
      accumulate(qb2, lb, head(pi + 1));
    }
  }
  // waves 2-3 hand their sums to waves 0-1 through LDS (lane-contiguous)
  __syncthreads();
  float* red = (float*)smem;                       // [2][32][64 lanes]
  if (wave >= 2) {
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        red[((wave & 1) * 32 + 16 * c + r) * 64 + lane] = acc[c][r];
  }
  __syncthreads();
  if (wave >= 2 || !qvalid) return;
  const int fr = qrow / Nv, ii = qrow % Nv;
  float* dst = ws.intra_part +
               (((size_t)kvh * pl.T + qb.aux + fr) * Nv + ii) * Nv;
#pragma unroll
  for (int c = 0; c < 2; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int kl = 32 * c + 8 * (r >> 2) + 4 * g + (r & 3);
      if (kl / Nv != fr || kl >= qb.len) continue;
      dst[kl % Nv] =
          acc[c][r] + red[((wave & 1) * 32 + 16 * c + r) * 64 + lane];
    }
}

__global__ __launch_bounds__(256) void intra_reduce_kernel(
    const DevPlan pl, const Workspace ws, float* __restrict__ out) {
  const size_t n = (size_t)pl.T * pl.Nv * pl.Nv;
  const float inv = 1.f / (float)pl.hq;
  for (size_t e = (size_t)blockIdx.x * 256 + threadIdx.x; e < n;
       e += (size_t)gridDim.x * 256) {
    float t = 0.f;
    for (int kvh = 0; kvh < pl.hkv; ++kvh) t += ws.intra_part[kvh * n + e];
    out[e] = t * inv;
  }
}

}  // namespace

hipError_t launch_attention(const DevPlan& p, const Workspace& w,
                            const AttnCall& c, hipStream_t s) {
  if (p.n_items == 0) return hipSuccess;
  if (attention_pipe_supported(p, c)) return launch_attention_pipe(p, w, c, s);
  dim3 grid(p.n_items), block(kThreads);
  if (p.topp) {
    if (c.fp32) {
      if (c.d == 64)
        attn_kernel<F32Path<64>, 64, true><<<grid, block, 0, s>>>(p, w, c);
      else
        attn_kernel<F32Path<128>, 128, true><<<grid, block, 0, s>>>(p, w, c);
    } else {
      if (c.d == 64)
        attn_kernel<Bf16Path<64>, 64, true><<<grid, block, 0, s>>>(p, w, c);
      else
        attn_kernel<Bf16Path<128>, 128, true><<<grid, block, 0, s>>>(p, w,
                                                                     c);
    }
    return hipGetLastError();
  }
  if (c.fp32) {
    if (c.d == 64)
      attn_kernel<F32Path<64>, 64, false><<<grid, block, 0, s>>>(p, w, c);
    else
      attn_kernel<F32Path<128>, 128, false><<<grid, block, 0, s>>>(p, w, c);
  } else {
    if (c.d == 64)
      attn_kernel<Bf16Path<64>, 64, false><<<grid, block, 0, s>>>(p, w, c);
    else
      attn_kernel<Bf16Path<128>, 128, false><<<grid, block, 0, s>>>(p, w, c);
  }
  return hipGetLastError();
}

hipError_t launch_intra_frame(const DevPlan& p, const Workspace& w,
                              const AttnCall& c, float* out, hipStream_t s) {
  dim3 grid(p.nb, p.hkv), block(kThreads);
  if (c.fp32) {
    if (c.d == 64)
      intra_kernel<F32Path<64>, 64><<<grid, block, 0, s>>>(p, w, c);
    else
      intra_kernel<F32Path<128>, 128><<<grid, block, 0, s>>>(p, w, c);
  } else {
    if (c.d == 64)
      intra_kernel<Bf16Path<64>, 64><<<grid, block, 0, s>>>(p, w, c);
    else
      intra_kernel<Bf16Path<128>, 128><<<grid, block, 0, s>>>(p, w, c);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t n = (size_t)p.T * p.Nv * p.Nv;
  const int blocks = (int)std::min<size_t>((n + 255) / 256, 4096);
  intra_reduce_kernel<<<dim3(blocks), dim3(256), 0, s>>>(p, w, out);
  return hipGetLastError();
}

}  // namespace evisel
