// Software-pipelined block-sparse prefill attention for gfx950 (bf16 inputs,
// static sparse rule, no frame-cue outputs) with the fused query-frame
// evidence partials. Same work items, LDS tile layout, loaders and outputs
// as attn_kernel (attn.hip); what differs is the order of work inside a
// wavefront.
//
// A wave (32 query rows of one head) keeps its MFMA pipe busy by running the
// VALU work of one tile beside the MFMAs of another. Per loop iteration j:
//   block 1  S(j+1) = K(j+1) Q^T, keys 0-31 then 32-63 (16 MFMAs), with the
//            exponentials of tile j's keys 32-63 (whose logits were left in
//            registers by the previous iteration) between them;
//   block 2  O^T += V(j)^T P(j)^T (16 MFMAs), with the exponentials of tile
//            j+1's keys 0-31.
// Each MFMA then has about two exponentials, two fused multiply-adds and two
// adds beside it, which issue while it executes. Probabilities are rounded
// to bf16 for the PV product only; a row's normaliser and, for query-token
// rows, its per-frame partial masses are fp32 sums of the fp32
// probabilities, as in attn_kernel.
//
// The softmax reference of a row is the exact row max of its first tile and
// never moves in this loop: no tile max, no rescale. A tile whose row sum
// exceeds 2^64 (or is not finite) marks the wave; after the last tile the
// work-group votes, and if any wave was marked the whole item is computed
// again by a plain per-tile exact loop (row max per tile, lazy rescale),
// which rewrites every output the first pass wrote. On ordinary inputs no
// row's logits rise 64 log2 units above its first tile's.
//
// LDS: [K0 | K1 | V0 | V1], one 64-key tile each, as attn_kernel. Key tile
// t lives in K(t % 2) and value tile t in V(t % 2); K(j+2) and V(j+1) are
// loaded during iteration j, so each arrives one iteration before it is
// read and one barrier per iteration orders the buffer reuse. The item's
// query rows are staged in K1 (first half) and V1 (second half) in the same
// round trip as K0 and V0; key tile 1 is fetched once they are in
// registers. After the last tile V0 carries the waves' votes.
#include <type_traits>

#include "attn_tiles.h"
#include "kernels.h"

namespace evisel {
namespace {

// The scalar arguments the kernel reads.
struct PipeArgs {
  const WorkItem* items;
  const BlockDesc* blocks;
  const BlockDesc* col_desc;
  const PairedTile* ptile;
  const BlockDesc* ptile_desc;
  const SeqDesc* seqs;
  const __bf16* q;
  const __bf16* k;
  const __bf16* v;
  __bf16* o;
  float* lse;     // may be null
  float* pO;      // split query-row partials and per-frame partial masses
  float* pM;
  float* pL;
  float* pNV;
  float* seg;
  int64_t segtot;
  int32_t hq, hkv, Nv, S;
  float c2;       // softmax scale * log2(e)
  // frame cues (the kernel's CUE form): visual rows' log2 partial masses
  // per key frame of each computed visual tile at its CSR position, or
  // null, and the log2 LSE of every non-query row, or null
  float* segv;
  float* lse2v;
  int32_t nnz;
};

// A key tile as the loop sees it (wave-uniform).
struct Tile {
  int start, len, region, aux;
  bool act;   // some row of this wave's half attends to it
  int pos;    // CSR position of the tile for this half (CUE form only)
};

// Instruction order requested from the scheduler (sched_group_barrier
// masks: 0x008 MFMA, 0x100 LDS read, 0x002 VALU).
// M MFMAs, each reading R operands from LDS, the reads four MFMAs ahead.
template <int M, int R>
__device__ __forceinline__ void sched_reads_ahead() {
  __builtin_amdgcn_sched_group_barrier(0x100, 4 * R, 0);
#pragma unroll
  for (int i = 0; i < M - 4; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, R, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
}
// Block 1: 2M MFMAs of QK with their K operand reads four ahead; the first
// M MFMAs each get V1 VALU instructions (the softmax), the rest one.
template <int M, int V1>
__device__ __forceinline__ void sched_block1() {
  __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
  for (int i = 0; i < M; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, V1, 0);
  }
#pragma unroll
  for (int i = 0; i < M - 4; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);
  }
}
// Block 2: M MFMAs of PV, two V^T reads per operand, four operands ahead;
// each MFMA gets V VALU instructions.
template <int M, int V>
__device__ __forceinline__ void sched_block2() {
  __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
#pragma unroll
  for (int i = 0; i < M - 4; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, V, 0);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, V, 0);
  }
}

template <int D, bool CUE>
__global__ __attribute__((amdgpu_flat_work_group_size(kThreads, kThreads),
                          amdgpu_waves_per_eu(2, 2))) void
attn_pipe_kernel(const PipeArgs a) {
  using P = Bf16Path<D>;
  constexpr int RC = P::RC;             // 16-byte chunks per row
  constexpr int TB = kTile * RC * 16;   // bytes of one tile
  constexpr int KK = D / 16;            // k-steps of one QK half
  constexpr int NMT = D / 32;           // d-tiles of O^T
  __shared__ __attribute__((aligned(1024))) char smem[4 * TB];
  EV_LDS char* const kb0 = (EV_LDS char*)smem;   // [K0 | K1 | V0 | V1]
  EV_LDS char* const vb0 = kb0 + 2 * TB;

  const WorkItem it = a.items[blockIdx.x];
  if (it.qblock < 0) return;
  const int n = it.kb_end - it.kb_begin;   // key tiles of the item
  if (n <= 0) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, g = lane >> 5;
  const int hsub = wave >> 1;
  // paired item: the second half takes a second query block of one head
  const bool uni = it.qblock2 >= 0;
  const int nhalf = uni ? 2 : it.nheads;
  const bool active = hsub < nhalf;
  const int hd1 = uni ? it.head : it.head + 1;
  const int h = active && hsub ? hd1 : it.head;
  const int kvh = it.head / (a.hq / a.hkv);
  const int qbid = uni && hsub ? it.qblock2 : it.qblock;
  const BlockDesc qb = a.blocks[qbid];
  const bool is_text = it.slot >= 0;
  const int qrow = 32 * (wave & 1) + l32;
  const bool qvalid = active && qrow < qb.len;
  const int qpos = qb.start + qrow;
  const int b0 = it.kb_begin;
  const float c2 = a.c2;

  // Tile descriptors, 64 at a time: lane t holds tile 64 * batch + t's
  // first token, aux field and (length | region << 8 | active << 10).
  int dsc_start = 0, dsc_aux = 0, dsc_meta = 1, dsc_pos = -1;
  auto load_batch = [&](int batch) {
    const int t = batch * 64 + lane;
    if (t < n) {
      const BlockDesc bd = uni ? a.ptile_desc[b0 + t] : a.col_desc[b0 + t];
      const int act = uni ? (a.ptile[b0 + t].pos[hsub] >= 0 ? 1 : 0) : 1;
      dsc_start = bd.start;
      dsc_aux = bd.aux;
      dsc_meta = bd.len | bd.region << 8 | act << 10;
      if (CUE) dsc_pos = uni ? a.ptile[b0 + t].pos[hsub] : b0 + t;
    }
  };
  auto desc = [&](int t) {
    const int l = t & 63;
    Tile d;
    d.start = __builtin_amdgcn_readlane(dsc_start, l);
    d.aux = __builtin_amdgcn_readlane(dsc_aux, l);
    const int meta = __builtin_amdgcn_readlane(dsc_meta, l);
    d.len = meta & 255;
    d.region = (meta >> 8) & 3;
    d.act = (meta >> 10) & 1;
    d.pos = CUE ? __builtin_amdgcn_readlane(dsc_pos, l) : -1;
    return d;
  };
  const Tile none = {0, 1, 0, 0, false, -1};

  TileLoader<__bf16, D, kSwzK> kload;
  TileLoader<__bf16, D, kSwzV> vload;
  kload.init(a.hkv, wave, lane);
  vload.init(a.hkv, wave, lane);
  typename P::PvOff pvo;
  P::pv_offsets(pvo, lane);

  // Prologue: descriptors, both halves' query rows (staged in K1 and V1)
  // and key/value tile 0 in one round trip; key tile 1 follows once the
  // query rows are in registers.
  load_batch(0);
  {
    TileLoader<__bf16, D, kSwzK> qload;
    qload.init(a.hq, wave, lane);
    qload.issue(kb0 + TB, a.q, it.q0start, it.q0len, it.head, wave);
    if (nhalf > 1)
      qload.issue(vb0 + TB, a.q, it.q1start, it.q1len, hd1, wave);
  }
  kload.issue(kb0, a.k, it.k0start, it.k0len, kvh, wave);
  vload.issue(vb0, a.v, it.k0start, it.k0len, kvh, wave);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  typename P::QFrag qf;
  P::load_q_lds(qf, hsub ? vb0 + TB : kb0 + TB, qrow, g);
  __syncthreads();   // every wave has its query rows: K1 and V1 are free
  if (n > 1) kload.issue(kb0 + TB, a.k, it.k1start, it.k1len, kvh, wave);

  // query-token rows: this video's offsets
  SeqDesc sq{};
  if (is_text) sq = a.seqs[it.seq];
  const int trow = qb.aux + qrow - sq.textrow0;
  float* const seg_row = a.seg + (size_t)h * a.segtot + sq.segbase +
                         (size_t)trow * sq.n_frames - sq.frame0;

  float m_ref = neg_inf(), l_part = 0.f, nv_part = 0.f;
  f32x16 o[NMT];
#pragma unroll
  for (int i = 0; i < NMT; ++i) o[i] = f32x16{};

  auto need_mask = [&](const Tile& t) {
    return t.len < kTile || t.start + t.len - 1 > qb.start;
  };
  // keys of half c past the row (causal) or past the tile's end -> -inf:
  // key 32c + 8(r/4) + 4g + r%4 is masked when its lane-free part exceeds x
  auto mask_half = [&](f32x16& s, int c, const Tile& t) {
    const int x = min(qpos - t.start, t.len - 1) - 4 * g;
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (32 * c + 8 * (r >> 2) + (r & 3) > x) s[r] = neg_inf();
  };
  // K operand of key half c, k-step kk (lane: key 32c + lane % 32)
  auto k_operand = [&](const EV_LDS char* kt, int c, int kk) {
    const int key = 32 * c + l32;
    return *(const EV_LDS bf16x8*)(kt + (key * RC + ((2 * kk + g) ^
                                                     swz<kSwzK, RC>(key))) *
                                            16);
  };
  // V^T operand of k-step cs (keys 16cs .. 16cs + 15), d-tile mt
  auto v_operand = [&](const EV_LDS char* vt, int cs, int mt) {
    const int c = cs >> 1, s = cs & 1;
    const EV_LDS char* a0 = vt + pvo.v[mt] + (32 * c + 16 * s) * RC * 16;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((EV_LDS i16x4*)a0);
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (EV_LDS i16x4*)(a0 + 8 * RC * 16));
    const i16x4 lohi[2] = {lo, hi};
    return __builtin_bit_cast(bf16x8, lohi);
  };
  // S^T for keys 32c .. 32c + 31 of the tile at kt
  auto qk_half = [&](f32x16& s, const EV_LDS char* kt, int c) {
    bf16x8 kf[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) kf[kk] = k_operand(kt, c, kk);
    s = f32x16{};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kk], qf.x[kk], s, 0, 0,
                                                  0);
    sched_reads_ahead<KK, 1>();
  };
  // probabilities of one half against the reference, as two bf16 groups;
  // returns their fp32 sum
  auto soft_half = [&](const f32x16& s, bf16x8& p0, bf16x8& p1,
                       float mu) -> float {
    f32x16 p;
    float sum = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      p[r] = exp2_(fmaf(s[r], c2, -mu));
      sum += p[r];
    }
    p0 = __builtin_convertvector(
        __builtin_shufflevector(p, p, 0, 1, 2, 3, 4, 5, 6, 7), bf16x8);
    p1 = __builtin_convertvector(
        __builtin_shufflevector(p, p, 8, 9, 10, 11, 12, 13, 14, 15), bf16x8);
    return sum;
  };
  // O^T += V^T P^T over the tile at vt
  auto pv_tile = [&](const EV_LDS char* vt, const bf16x8 (&pb)[4]) {
    bf16x8 va[4 * NMT];
#pragma unroll
    for (int i = 0; i < 4 * NMT; ++i) va[i] = v_operand(vt, i / NMT, i % NMT);
#pragma unroll
    for (int i = 0; i < 4 * NMT; ++i)
      o[i % NMT] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
          va[i], pb[i / NMT], o[i % NMT], 0, 0, 0);
    sched_reads_ahead<4 * NMT, 2>();
  };
  // end of a tile for query-token rows: per-frame log2 partial masses of
  // visual keys (each (row, frame) slot written once), or the running
  // non-visual mass
  auto text_tile = [&](const Tile& t, float (&g8)[8]) {
    if (t.region == kVis) {
      if (a.Nv == kTile) {
        float s = 0.f;
#pragma unroll
        for (int q = 0; q < 8; ++q) s += g8[q];
        s = pair_sum(s);
        if (g == 0 && qvalid) seg_row[t.aux] = m_ref + log2_(s);
      } else {
#pragma unroll
        for (int q = 0; q < 8; ++q) g8[q] = pair_sum(g8[q]);
        const int lg = __builtin_ctz((unsigned)a.Nv) - 3;   // log2(N_v / 8)
        const int nseg = kTile / a.Nv;
        for (int si = 0; si < nseg; ++si) {
          float s = 0.f;
#pragma unroll
          for (int q = 0; q < 8; ++q) s += (q >> lg) == si ? g8[q] : 0.f;
          if (g == 0 && qvalid && si * a.Nv < t.len)
            seg_row[t.aux + si] = m_ref + log2_(s);
        }
      }
    } else {
      float s = 0.f;
#pragma unroll
      for (int q = 0; q < 8; ++q) s += g8[q];
      nv_part += s;
    }
  };

  // The same for the pipelined loop, where frames hold 32 or 64 keys: h0 and
  // h1 are the row's fp32 sums over keys 0-31 and 32-63.
  auto text_tile_halves = [&](const Tile& t, float h0, float h1) {
    if (t.region == kVis) {
      if (a.Nv == kTile) {
        const float s = pair_sum(h0 + h1);
        if (g == 0 && qvalid) seg_row[t.aux] = m_ref + log2_(s);
      } else {
        const float s0 = pair_sum(h0), s1 = pair_sum(h1);
        if (g == 0 && qvalid) {
          seg_row[t.aux] = m_ref + log2_(s0);
          if (t.len > 32) seg_row[t.aux + 1] = m_ref + log2_(s1);
        }
      }
    } else {
      nv_part += h0 + h1;
    }
  };

  // Frame cues (CUE form): a visual row's log2 partial mass on each key
  // frame of a computed visual tile, written at the tile's CSR position
  // ([h][nnz][64 / N_v][64 rows]); frames hold 32 or 64 keys, h0 and h1 are
  // the row's sums over keys 0-31 and 32-63.
  const bool vis_ff =
      CUE && a.segv != nullptr && !is_text && qb.region == kVis;
  float* const segv_row =
      vis_ff ? a.segv + (size_t)h * a.nnz * (kTile / a.Nv) * kTile + qrow
             : nullptr;
  auto vis_tile_halves = [&](const Tile& t, float h0, float h1) {
    if (!vis_ff || t.region != kVis || t.pos < 0) return;
    if (a.Nv == kTile) {
      const float s = pair_sum(h0 + h1);
      if (g == 0 && qvalid) segv_row[(size_t)t.pos * kTile] = m_ref + log2_(s);
    } else {
      const float s0 = pair_sum(h0), s1 = pair_sum(h1);
      if (g == 0 && qvalid) {
        float* const dst = segv_row + (size_t)t.pos * 2 * kTile;
        dst[0] = m_ref + log2_(s0);
        if (t.len > 32) dst[kTile] = m_ref + log2_(s1);
      }
    }
  };

  // Exact recomputation of the whole item (row max per tile, accumulators
  // rescaled when it rises by more than kRescaleSlack), used when some row's
  // probabilities exceeded 2^64 against its first-tile reference.
  auto exact_item = [&](auto txt) {
    constexpr bool TXT = decltype(txt)::value;
    m_ref = neg_inf();
    l_part = 0.f;
    nv_part = 0.f;
#pragma unroll
    for (int i = 0; i < NMT; ++i) o[i] = f32x16{};
    load_batch(0);
    kload.issue(kb0, a.k, it.k0start, it.k0len, kvh, wave);
    vload.issue(vb0, a.v, it.k0start, it.k0len, kvh, wave);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    Tile cur = desc(0);
    for (int t = 0; t < n; ++t) {
      if (t + 1 < n && ((t + 1) & 63) == 0) load_batch((t + 1) >> 6);
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
      const int pt = t & 1;
      Tile nxt = none;
      if (t + 1 < n) {
        nxt = desc(t + 1);
        kload.issue(kb0 + (1 - pt) * TB, a.k, nxt.start, nxt.len, kvh, wave);
        vload.issue(vb0 + (1 - pt) * TB, a.v, nxt.start, nxt.len, kvh, wave);
      }
      if (active && cur.act) {
        f32x16 s[2];
        qk_half(s[0], kb0 + pt * TB, 0);
        qk_half(s[1], kb0 + pt * TB, 1);
        if (need_mask(cur)) {
          mask_half(s[0], 0, cur);
          mask_half(s[1], 1, cur);
        }
        float mx = neg_inf();
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
          for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[c][r]);
        mx = pair_max(mx);
        const float m_new = fmaxf(m_ref, mx * c2);
        const bool need = m_new > m_ref + kRescaleSlack;
        const bool resc = need && m_ref != neg_inf();
        if (__any(resc)) {
          const float alpha = resc ? exp2_(m_ref - m_new) : 1.f;
          l_part *= alpha;
          nv_part *= alpha;
#pragma unroll
          for (int i = 0; i < NMT; ++i) o[i] *= alpha;
        }
        m_ref = need ? m_new : m_ref;
        const float mu = m_ref == neg_inf() ? 0.f : m_ref;
        bf16x8 pb[4];
        float g8[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          f32x16 p;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            p[r] = exp2_(fmaf(s[c][r], c2, -mu));
            g8[4 * c + (r >> 2)] += p[r];
          }
          pb[2 * c] = __builtin_convertvector(
              __builtin_shufflevector(p, p, 0, 1, 2, 3, 4, 5, 6, 7), bf16x8);
          pb[2 * c + 1] = __builtin_convertvector(
              __builtin_shufflevector(p, p, 8, 9, 10, 11, 12, 13, 14, 15),
              bf16x8);
        }
        float ts = 0.f;
#pragma unroll
        for (int q = 0; q < 8; ++q) ts += g8[q];
        l_part += ts;
        if (TXT) text_tile(cur, g8);
        if (CUE && !TXT)
          vis_tile_halves(cur, g8[0] + g8[1] + g8[2] + g8[3],
                          g8[4] + g8[5] + g8[6] + g8[7]);
        pv_tile(vb0 + pt * TB, pb);
      }
      cur = nxt;
    }
  };

  auto pipeline = [&](auto txt) {
    constexpr bool TXT = decltype(txt)::value;
    // Carried between iterations, for the tile in flight (tile j at the top
    // of iteration j): the logits of its keys 32-63 (s1), the bf16
    // probabilities of its keys 0-31 (pb[0..1]) and their fp32 sum (th).
    // A tile that is not active for this wave's rows (half of a paired item)
    // takes its probabilities against +inf, so they are all 0 and its PV
    // product adds nothing; only a wave's first active tile needs a branch
    // (its row max sets the reference).
    f32x16 s0, s1;
    bf16x8 pb[4];
    float th = 0.f;   // fp32 sum of the probabilities of keys 0-31
    bool started = false, bad = false;
    const float pinf = __builtin_inff();

    // keys 0-31 of a tile (logits in s0) to pb[0..1] and their sum
    auto start_half = [&](float mu) {
      th = soft_half(s0, pb[0], pb[1], mu);
    };
    // a wave's first active tile: the exact row max of its logits (both
    // halves, masked) is the reference
    auto first_tile = [&](const Tile& t) {
      if (need_mask(t)) mask_half(s1, 1, t);
      float mx = neg_inf();
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, fmaxf(s0[r], s1[r]));
      mx = pair_max(mx);
      m_ref = mx == neg_inf() ? 0.f : mx * c2;
      started = true;
    };
    // end of tile t once its keys 32-63 are in pb[2..3] (h1: their sum)
    auto finish = [&](const Tile& t, float h1) {
      const float ts = th + h1;
      if (TXT && t.act) text_tile_halves(t, th, h1);
      if (CUE && !TXT && t.act) vis_tile_halves(t, th, h1);
      bad = bad || __any(active && !(ts <= kFastBound));
      l_part += ts;
    };

    // Tile 0: its key and value tiles and key tile 1 came with the query
    // rows.
    Tile tc = none, tn = desc(0), tnn = n > 1 ? desc(1) : none;
    qk_half(s0, kb0, 0);
    qk_half(s1, kb0, 1);
    if (need_mask(tn)) mask_half(s0, 0, tn);
    if (active && tn.act) first_tile(tn);
    start_half(tn.act && started ? m_ref : pinf);

    // top of iteration j: key tile j+1 and value tile j have landed; every
    // wave is past iteration j-1, so K(j % 2) and V((j+1) % 2) may be
    // refilled with key tile j+2 and value tile j+1
    auto top = [&](int j) {
      if (j + 2 < n && ((j + 2) & 63) == 0) load_batch((j + 2) >> 6);
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
      tc = tn;
      tn = tnn;
      tnn = j + 2 < n ? desc(j + 2) : none;
      if (j + 2 < n)
        kload.issue(kb0 + (j & 1) * TB, a.k, tnn.start, tnn.len, kvh, wave);
      if (j + 1 < n)
        vload.issue(vb0 + ((j + 1) & 1) * TB, a.v, tn.start, tn.len, kvh,
                    wave);
    };
    // Iteration j (j + 1 < n): finish tile j, start tile j+1.
    auto iter = [&](int j, auto par) {
      constexpr int pj = decltype(par)::value;   // j & 1
      constexpr int pn = 1 - pj;
      const EV_LDS char* const kn = kb0 + pn * TB;   // key tile j + 1
      const EV_LDS char* const vc = vb0 + pj * TB;   // value tile j
      top(j);
      const Tile cur = tc, nxt = tn;
      const float mu_c = cur.act ? m_ref : pinf;
      if (need_mask(cur)) mask_half(s1, 1, cur);
      // block 1: QK(j+1) beside the exponentials of tile j, keys 32-63.
      // The 16 K operand reads run four ahead of their MFMAs; the first
      // chain (keys 0-31) carries the softmax VALU work.
      {
        bf16x8 kf[2 * KK];
#pragma unroll
        for (int i = 0; i < 2 * KK; ++i) kf[i] = k_operand(kn, i / KK, i % KK);
        f32x16 n0 = f32x16{}, n1 = f32x16{};
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
          n0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kk], qf.x[kk], n0,
                                                       0, 0, 0);
        const float h1 = soft_half(s1, pb[2], pb[3], mu_c);
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
          n1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[KK + kk], qf.x[kk],
                                                       n1, 0, 0, 0);
        sched_block1<KK, 40 / KK>();
        s0 = n0;
        s1 = n1;
        finish(cur, h1);
      }
      if (need_mask(nxt)) mask_half(s0, 0, nxt);
      if (!started && active && nxt.act) first_tile(nxt);
      const float mu_n = nxt.act && started ? m_ref : pinf;
      // block 2: PV(j) beside the exponentials of tile j+1, keys 0-31,
      // which replace pb[0..1] once the PV MFMAs have read them. The V^T
      // operand reads (two per MFMA) run four MFMAs ahead.
      {
        bf16x8 va[4 * NMT];
#pragma unroll
        for (int i = 0; i < 4 * NMT; ++i) va[i] = v_operand(vc, i / NMT, i % NMT);
        const bf16x8 pc[4] = {pb[0], pb[1], pb[2], pb[3]};
#pragma unroll
        for (int i = 0; i < 4 * NMT; ++i)
          o[i % NMT] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              va[i], pc[i / NMT], o[i % NMT], 0, 0, 0);
        start_half(mu_n);
        // keep the exponentials in this block (they would otherwise be
        // sunk to their first use, past the next barrier)
        asm volatile("" ::"v"(pb[0]), "v"(pb[1]), "v"(th));
        sched_block2<4 * NMT, 48 / (4 * NMT) + 1>();
      }
    };
    int j = 0;
    for (; j + 2 < n; j += 2) {
      iter(j, std::integral_constant<int, 0>{});
      iter(j + 1, std::integral_constant<int, 1>{});
    }
    if (j + 1 < n) {
      iter(j, std::integral_constant<int, 0>{});
      ++j;
    }
    // last tile (j = n - 1): keys 32-63 and PV
    top(j);
    {
      const Tile cur = tc;
      if (need_mask(cur)) mask_half(s1, 1, cur);
      finish(cur, soft_half(s1, pb[2], pb[3], cur.act ? m_ref : pinf));
      pv_tile(vb0 + (j & 1) * TB, pb);
    }
    // votes, in V0 (the O rows are staged in K0 and K1 afterwards): every
    // wave is done with the tiles
    __syncthreads();
    if (lane == 0) ((EV_LDS int*)vb0)[wave] = bad ? 1 : 0;
    __syncthreads();
    const EV_LDS int* votes = (const EV_LDS int*)vb0;
    if ((votes[0] | votes[1] | votes[2] | votes[3]) != 0) {
      __syncthreads();   // every wave has read the votes
      exact_item(txt);
      __syncthreads();   // every wave is done with the tiles
    }
  };

  // The "top" of the first iteration is the prologue's wait and barrier: the
  // loop driver's top(j) runs from j = 0 and expects tile descriptors 0 and
  // 1 in tn / tnn before iteration -1, which sets them up itself.
  if (!is_text) {
    pipeline(std::false_type{});
  } else if (a.Nv >= 32) {
    pipeline(std::true_type{});
  } else {
    // frames of 8 or 16 keys: the per-frame sums need eight groups per
    // tile, which the pipelined loop does not keep; the exact loop does
    exact_item(std::true_type{});
  }

  const float l_tot = pair_sum(l_part);
  if (!is_text) {
    // O rows through LDS (K0 for the first half, K1 for the second), then
    // whole-row stores by every thread
    if (active)
      P::o_to_lds(kb0 + hsub * TB, o, qvalid ? 1.f / l_tot : 0.f, qrow, g);
    __syncthreads();
    for (int hh = 0; hh < nhalf; ++hh)
      P::o_from_lds(a.o, kb0 + hh * TB, hh ? it.q1start : it.q0start,
                    hh ? it.q1len : it.q0len, hh ? hd1 : it.head, a.hq, tid);
    if (qvalid && g == 0 && a.lse)
      a.lse[(size_t)h * a.S + qpos] = (m_ref + log2_(l_tot)) * kLn2;
    if (CUE && qvalid && g == 0 && a.lse2v)
      a.lse2v[(size_t)h * a.S + qpos] = m_ref + log2_(l_tot);
  } else if (active) {
    const float nv_tot = pair_sum(nv_part);
    const int slot =
        uni ? (hsub ? it.slot2 : it.slot) : it.slot + hsub * it.nch;
    if (qvalid) {
      float* po = a.pO + ((size_t)slot * kTile + qrow) * D;
#pragma unroll
      for (int mt = 0; mt < NMT; ++mt)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          f32x4 x = {o[mt][4 * r4], o[mt][4 * r4 + 1], o[mt][4 * r4 + 2],
                     o[mt][4 * r4 + 3]};
          *(f32x4*)(po + 32 * mt + 8 * r4 + 4 * g) = x;
        }
      if (g == 0) {
        const size_t ix = (size_t)slot * kTile + qrow;
        a.pM[ix] = m_ref;
        a.pL[ix] = l_tot;
        a.pNV[ix] = nv_tot > 0.f ? m_ref + log2_(nv_tot) : neg_inf();
      }
    }
  }
}

}  // namespace

bool attention_pipe_supported(const DevPlan& p, const AttnCall& c) {
  // frame cues: frames of 32 or 64 keys (the loop keeps two half-tile sums)
  const bool cues = c.segv != nullptr || c.lse2v != nullptr;
  return !c.fp32 && !p.topp && (!cues || p.Nv >= 32) &&
         (c.d == 64 || c.d == 128);
}

hipError_t launch_attention_pipe(const DevPlan& p, const Workspace& w,
                                 const AttnCall& c, hipStream_t s) {
  if (p.n_items == 0) return hipSuccess;
  PipeArgs a;
  a.items = p.items;
  a.blocks = p.blocks;
  a.col_desc = p.col_desc;
  a.ptile = p.ptile;
  a.ptile_desc = p.ptile_desc;
  a.seqs = p.seqs;
  a.q = (const __bf16*)c.q;
  a.k = (const __bf16*)c.k;
  a.v = (const __bf16*)c.v;
  a.o = (__bf16*)c.o;
  a.lse = c.lse;
  a.pO = w.pO;
  a.pM = w.pM;
  a.pL = w.pL;
  a.pNV = w.pNV;
  a.seg = w.seg;
  a.segtot = p.segtot;
  a.hq = p.hq;
  a.hkv = p.hkv;
  a.Nv = p.Nv;
  a.S = p.S;
  a.c2 = c.scale_log2;
  a.segv = c.segv;
  a.lse2v = c.lse2v;
  a.nnz = p.nnz;
  const bool cue = c.segv != nullptr || c.lse2v != nullptr;
  dim3 grid(p.n_items), block(kThreads);
  if (c.d == 64 && cue)
    attn_pipe_kernel<64, true><<<grid, block, 0, s>>>(a);
  else if (c.d == 64)
    attn_pipe_kernel<64, false><<<grid, block, 0, s>>>(a);
  else if (cue)
    attn_pipe_kernel<128, true><<<grid, block, 0, s>>>(a);
  else
    attn_pipe_kernel<128, false><<<grid, block, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace evisel
