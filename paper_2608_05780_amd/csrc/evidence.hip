// Query-row merge, evidence reduction and frame aggregation (gfx950).
//
// combine_evidence_kernel: one launch, three independent parts (ranges of
//   the block index), so that no part waits for another:
//   combine    one work-group per (query-token tile, head): merges the
//              tile's chunk partials into O and the LSE, sixteen threads per
//              row (each a contiguous D/16 slice);
//   evidence   one work-group per (64 frames, head): E[h, f] = sum over the
//              query rows r of f's video of exp2(seg[h, r, f] - lse2[h, r]),
//              i.e. each row's softmax mass on frame f (the query-frame cue
//              of Evidence Decomposition, kept as a raw sum over the query
//              rows). 16 row groups sum strided rows and are added in a fixed
//              order in LDS, one store per output: no atomics, bitwise
//              reproducible. Adjacent threads read adjacent frames of the
//              same row, so every load is coalesced;
//   text mass  one work-group per (head, video), only when requested: the
//              video's query-row mass on non-visual keys (system prefix and
//              query tokens); one wavefront per tile, rows and then tiles
//              added in a fixed order.
//   Every part that needs a row's log2 LSE rebuilds it from the chunk
//   partials the same way: the largest chunk reference, then the rescaled
//   chunk row sums added in chunk order. The evidence part computes the
//   LSE of the rows its frames read once into LDS (when they fit).
// frame_mean_kernel: E_qf[l, t] = sum_h E[l, h, t] / (Hq * n_text) and the
//   mean over layers (heads averaged per layer, layer kept); 32 frames x 32
//   layer groups per work-group, layers added in a fixed order.
// topk_kernel: per video, rank r(t) = #{t' : e(t') > e(t) or (e(t') == e(t)
//   and t' < t)}; frames with r(t) < k land at topk[offset + r(t)]. Ranks of a
//   strict total order are a permutation, so every slot gets one writer.
#include "kernels.h"

namespace evisel {
namespace {

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kTile = 64;
constexpr float kLn2 = 0.69314718055994530942f;

__device__ __forceinline__ float neg_inf() { return -__builtin_inff(); }
__device__ __forceinline__ float exp2_(float x) {
  return __builtin_amdgcn_exp2f(x);
}
__device__ __forceinline__ float log2_(float x) {
  return __builtin_amdgcn_logf(x);
}

// log2 LSE of row r of a query-token tile from its chunk partials (chunk
// slots slot0 .. slot0 + nch - 1).
__device__ __forceinline__ float row_lse2(const Workspace& ws, int slot0,
                                          int nch, int r) {
  float M = neg_inf();
  for (int c = 0; c < nch; ++c)
    M = fmaxf(M, ws.pM[(size_t)(slot0 + c) * kTile + r]);
  float L = 0.f;
  for (int c = 0; c < nch; ++c) {
    const size_t ix = (size_t)(slot0 + c) * kTile + r;
    const float m = ws.pM[ix];
    const float w = m == neg_inf() ? 0.f : exp2_(m - M);
    L += w * ws.pL[ix];
  }
  return M + log2_(L);
}

// Sum over the 64 lanes of a wavefront, in a fixed butterfly order (the
// same result on every lane, reproducible run to run).
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

// Row `rr` (0-based) of video sq's query tokens, head h.
__device__ __forceinline__ float text_row_lse2(const DevPlan& pl,
                                               const Workspace& ws,
                                               const SeqDesc& sq, int h,
                                               int rr) {
  const TextTile tt = pl.tiles[sq.tile0 + (rr >> 6)];
  return row_lse2(ws, tt.slot0 + h * tt.n_chunks, tt.n_chunks, rr & 63);
}

constexpr int kCeThreads = 1024;
constexpr int kEvFrames = 64, kEvRows = kCeThreads / kEvFrames;   // 16
constexpr int kLseCache = 4096;   // query rows whose LSE the evidence part
                                  // keeps in LDS

template <int D, bool F32>
__global__ __launch_bounds__(kCeThreads) void combine_evidence_kernel(
    const DevPlan pl, const Workspace ws, const AttnCall ac,
    float* __restrict__ ev, float* __restrict__ tm) {
  __shared__ float red[kEvRows][kEvFrames];
  __shared__ float l2c[kLseCache];
  const int tid = threadIdx.x;
  const int n_comb = pl.n_tiles * pl.hq;
  const int n_fb = (pl.T + kEvFrames - 1) / kEvFrames;
  int bid = blockIdx.x;

  if (bid < n_comb) {
    // ---- combine: tile bid % n_tiles, head bid / n_tiles
    constexpr int DP = D / 16;
    const TextTile tt = pl.tiles[bid % pl.n_tiles];
    const int h = bid / pl.n_tiles;
    const BlockDesc qb = pl.blocks[tt.qblock];
    const int r = tid >> 4, part = tid & 15;
    if (r >= qb.len) return;
    const int slot0 = tt.slot0 + h * tt.n_chunks;
    float M = neg_inf();
    for (int c = 0; c < tt.n_chunks; ++c)
      M = fmaxf(M, ws.pM[(size_t)(slot0 + c) * kTile + r]);
    float L = 0.f;
    float acc[DP];
#pragma unroll
    for (int i = 0; i < DP; ++i) acc[i] = 0.f;
    for (int c = 0; c < tt.n_chunks; ++c) {
      const size_t ix = (size_t)(slot0 + c) * kTile + r;
      const float m = ws.pM[ix];
      const float w = m == neg_inf() ? 0.f : exp2_(m - M);
      L += w * ws.pL[ix];
      const float* po = ws.pO + ix * D + part * DP;
#pragma unroll
      for (int i = 0; i < DP; i += 4) {
        const f32x4 t = *(const f32x4*)(po + i);
        acc[i] += w * t[0];
        acc[i + 1] += w * t[1];
        acc[i + 2] += w * t[2];
        acc[i + 3] += w * t[3];
      }
    }
    const float inv = 1.f / L;
    const int qpos = qb.start + r;
#pragma unroll
    for (int i = 0; i < DP; i += 4) {
      const f32x4 v = {acc[i] * inv, acc[i + 1] * inv, acc[i + 2] * inv,
                       acc[i + 3] * inv};
      const size_t off = ((size_t)qpos * pl.hq + h) * D + part * DP + i;
      if (F32)
        *(f32x4*)((float*)ac.o + off) = v;
      else
        *(bf16x4*)((__bf16*)ac.o + off) = __builtin_convertvector(v, bf16x4);
    }
    if (part == 0 && ac.lse)
      ac.lse[(size_t)h * pl.S + qpos] = (M + log2_(L)) * kLn2;
    return;
  }
  bid -= n_comb;

  if (bid < n_fb * pl.hq) {
    // ---- evidence: frames [f0, f0 + 64) of head h
    const int h = bid / n_fb, f0 = (bid % n_fb) * kEvFrames;
    const int fl = tid % kEvFrames, rg = tid / kEvFrames;
    const int f = f0 + fl, fv = min(f, pl.T - 1);
    const int n0 = pl.frame_seq[f0];
    const int n1 = pl.frame_seq[min(f0 + kEvFrames, pl.T) - 1];
    const SeqDesc sq = pl.seqs[pl.frame_seq[fv]];
    const float* src = ws.seg + (size_t)h * pl.segtot + sq.segbase +
                       (fv - sq.frame0);
    // the first rows' partial masses are in flight while the LSEs are built
    constexpr int kPre = 8;
    float pre[kPre];
#pragma unroll
    for (int i = 0; i < kPre; ++i) {
      const int r = rg + i * kEvRows;
      pre[i] = r < sq.n_text ? src[(size_t)r * sq.n_frames] : 0.f;
    }
    // the query rows of the videos these frames belong to are consecutive
    const SeqDesc s0 = pl.seqs[n0], s1 = pl.seqs[n1];
    const int r0 = s0.textrow0, nrows = s1.textrow0 + s1.n_text - r0;
    const bool cached = nrows <= kLseCache;
    if (cached) {
      for (int n = n0; n <= n1; ++n) {
        const SeqDesc sn = pl.seqs[n];
        for (int rr = tid; rr < sn.n_text; rr += kCeThreads)
          l2c[sn.textrow0 - r0 + rr] = text_row_lse2(pl, ws, sn, h, rr);
      }
      __syncthreads();
    }
    float acc = 0.f;
    if (f < pl.T) {
      const float* l2 = l2c + (sq.textrow0 - r0);
      auto lse = [&](int r) {
        return cached ? l2[r] : text_row_lse2(pl, ws, sq, h, r);
      };
#pragma unroll
      for (int i = 0; i < kPre; ++i) {
        const int r = rg + i * kEvRows;
        if (r < sq.n_text) acc += exp2_(pre[i] - lse(r));
      }
#pragma unroll 4
      for (int r = rg + kPre * kEvRows; r < sq.n_text; r += kEvRows)
        acc += exp2_(src[(size_t)r * sq.n_frames] - lse(r));
    }
    red[rg][fl] = acc;
    __syncthreads();
    if (rg == 0 && f < pl.T) {
      float t = 0.f;
#pragma unroll
      for (int i = 0; i < kEvRows; ++i) t += red[i][fl];
      ev[(size_t)h * pl.T + f] = t;
    }
    return;
  }
  bid -= n_fb * pl.hq;

  // ---- text mass of (head, video): wave w takes the video's tiles w,
  // w + 16, ...; lane = row of the tile
  const int h = bid / pl.n_seq, n = bid % pl.n_seq;
  const SeqDesc sq = pl.seqs[n];
  const int lane = tid & 63, wave = tid >> 6;
  float wsum = 0.f;
  for (int i = wave; i < sq.n_tiles; i += kCeThreads / 64) {
    const TextTile tt = pl.tiles[sq.tile0 + i];
    float nv = 0.f;
    if (lane < pl.blocks[tt.qblock].len) {
      const int slot0 = tt.slot0 + h * tt.n_chunks;
      const float l2 = row_lse2(ws, slot0, tt.n_chunks, lane);
      for (int c = 0; c < tt.n_chunks; ++c)
        nv += exp2_(ws.pNV[(size_t)(slot0 + c) * kTile + lane] - l2);
    }
    wsum += wave_sum(nv);
  }
  float* part = &red[0][0];
  if (lane == 0) part[wave] = wsum;
  __syncthreads();
  if (wave == 0) {
    const float t = wave_sum(lane < kCeThreads / 64 ? part[lane] : 0.f);
    if (lane == 0) tm[(size_t)h * pl.n_seq + n] = t;
  }
}

constexpr int kFmFrames = 32, kFmLayers = 32;

__global__ __launch_bounds__(kFmFrames * kFmLayers) void frame_mean_kernel(
    const DevPlan pl, const float* __restrict__ ev, int n_layers,
    float* __restrict__ e_layer, float* __restrict__ e_qf) {
  __shared__ float red[kFmLayers][kFmFrames];
  const int tl = threadIdx.x % kFmFrames, lg = threadIdx.x / kFmFrames;
  const int t = blockIdx.x * kFmFrames + tl;
  float part = 0.f;
  if (t < pl.T) {
    const SeqDesc sq = pl.seqs[pl.frame_seq[t]];
    const float denom = (float)pl.hq * (float)sq.n_text;
    for (int l = lg; l < n_layers; l += kFmLayers) {
      float s = 0.f;
#pragma unroll 4
      for (int h = 0; h < pl.hq; ++h)
        s += ev[((size_t)l * pl.hq + h) * pl.T + t];
      const float v = s / denom;
      if (e_layer) e_layer[(size_t)l * pl.T + t] = v;
      part += v;
    }
  }
  red[lg][tl] = part;
  __syncthreads();
  if (lg == 0 && t < pl.T) {
    float pooled = 0.f;
#pragma unroll
    for (int i = 0; i < kFmLayers; ++i) pooled += red[i][tl];
    e_qf[t] = pooled / (float)n_layers;
  }
}

constexpr int kTopkThreads = 1024;
constexpr int kTopkLds = 16384;   // frames held in LDS per video

__device__ __forceinline__ float rank_key(float x) {
  return x != x ? -__builtin_inff() : x;   // NaN ranks like -inf
}

__global__ __launch_bounds__(kTopkThreads) void topk_kernel(
    const DevPlan pl, const float* __restrict__ e_qf,
    const int* __restrict__ kps, int* __restrict__ topk) {
  __shared__ float vals[kTopkLds];
  const int n = blockIdx.x;
  const SeqDesc sq = pl.seqs[n];
  const int F = sq.n_frames;
  int off = 0;
  for (int i = 0; i < n; ++i) off += min(max(kps[i], 0), pl.seqs[i].n_frames);
  const int k = min(max(kps[n], 0), F);
  if (k == 0) return;
  const float* src = e_qf + sq.frame0;
  const bool in_lds = F <= kTopkLds;
  if (in_lds) {
    for (int t = threadIdx.x; t < F; t += kTopkThreads)
      vals[t] = rank_key(src[t]);
    __syncthreads();
  }
  for (int t = threadIdx.x; t < F; t += kTopkThreads) {
    const float v = in_lds ? vals[t] : rank_key(src[t]);
    int rank = 0;
    for (int u = 0; u < F; ++u) {
      const float w = in_lds ? vals[u] : rank_key(src[u]);
      rank += (w > v) || (w == v && u < t);
    }
    if (rank < k) topk[off + rank] = t;
  }
}

// Cross-frame cue of one layer: one wavefront per frame pair (a, b). Lane r
// < N_v owns row r of frame a; it adds, over the heads in order, the row's
// normalised mass on frame b, exp2(partial - LSE), from the partial the
// attention pass left for that key tile. A top-p tile that no row of head
// h's work item kept was never computed and adds nothing. The lanes are
// then summed by a butterfly (every lane ends with the same bits) and the
// pair gets the mean over heads and frame a's rows.
constexpr int kPairWaves = 4;

constexpr int kPairHeads = 8;

__global__ __launch_bounds__(64 * kPairWaves) void frame_pairs_kernel(
    const DevPlan pl, const Workspace ws, float* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int pi = blockIdx.x * kPairWaves + (threadIdx.x >> 6);
  if (pi >= pl.n_pairs) return;
  const FramePair fp = pl.pairs[pi];
  const int fpt = 64 / pl.Nv;
  const BlockDesc qb = pl.blocks[fp.qblock];
  const int kb = pl.col[fp.pos];
  const int loc = pl.blk_local[kb];
  const bool always = !pl.topp || kb == fp.qblock || loc < 0;
  const int group = pl.hq / pl.hkv;
  const bool rv = lane < pl.Nv;
  const int row = fp.roff + (rv ? lane : 0);
  // heads in groups of kPairHeads: the group's loads go out together, the
  // sum still runs in head order
  float acc = 0.f;
  for (int hb = 0; hb < pl.hq; hb += kPairHeads) {
    float sv[kPairHeads], l2[kPairHeads];
    bool dn[kPairHeads];
#pragma unroll
    for (int u = 0; u < kPairHeads; ++u) {
      const int h = hb + u;
      bool done = always;
      if (!always && h < pl.hq) {
        const int g0 = (h / group) * group;
        const int h0 = g0 + ((h - g0) / kHeadsPerItem) * kHeadsPerItem;
        const int nh = min(kHeadsPerItem, g0 + group - h0);
        unsigned wd = 0u;
        for (int i = 0; i < nh; ++i)
          wd |= ws.ubits[((size_t)(h0 + i) * pl.nb + fp.qblock) * pl.W +
                         (loc >> 5)];
        done = (wd >> (loc & 31)) & 1u;
      }
      dn[u] = done && rv && h < pl.hq;
      sv[u] = dn[u] ? ws.segv[(((size_t)h * pl.nnz + fp.pos) * fpt +
                                fp.koff) * 64 + row]
                    : 0.f;
      l2[u] = dn[u] ? ws.lse2v[(size_t)h * pl.S + qb.start + row] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kPairHeads; ++u)
      if (dn[u]) acc += exp2_(sv[u] - l2[u]);
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) acc += __shfl_xor(acc, o);
  if (lane == 0) out[pi] = acc / ((float)pl.hq * (float)pl.Nv);
}

// E_ff[l, t]: the mean over t's earlier frames of A_ff[t, b] and the mean
// over its later frames of A_ff[a, t], averaged over the sides that exist
// (pairs outside the sparse pattern are 0). One wavefront per (layer,
// frame): lanes take strided pairs, then a butterfly adds the lanes (fixed
// order, every lane ends with the same bits).
constexpr int kEffWaves = 4;

__global__ __launch_bounds__(64 * kEffWaves) void e_ff_kernel(
    const DevPlan pl, const float* __restrict__ pr, float* __restrict__ e_ff) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * kEffWaves + (threadIdx.x >> 6), l = blockIdx.y;
  if (t >= pl.T) return;
  const SeqDesc sq = pl.seqs[pl.frame_seq[t]];
  const int tl = t - sq.frame0, F = sq.n_frames;
  const float* p = pr + (size_t)l * pl.n_pairs;
  float o = 0.f, in = 0.f;
  for (int i = pl.ff_out_ptr[t] + lane; i < pl.ff_out_ptr[t + 1]; i += 64)
    o += p[pl.ff_out_idx[i]];
  for (int i = pl.ff_in_ptr[t] + lane; i < pl.ff_in_ptr[t + 1]; i += 64)
    in += p[pl.ff_in_idx[i]];
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    o += __shfl_xor(o, m);
    in += __shfl_xor(in, m);
  }
  if (lane) return;
  float acc = 0.f;
  int ns = 0;
  if (tl > 0) {
    acc += o / (float)tl;
    ++ns;
  }
  if (tl < F - 1) {
    acc += in / (float)(F - 1 - tl);
    ++ns;
  }
  e_ff[(size_t)l * pl.T + t] = ns ? acc / (float)ns : 0.f;
}

}  // namespace

hipError_t launch_frame_pairs(const DevPlan& p, const Workspace& w,
                              float* pairs_out, hipStream_t s) {
  if (p.n_pairs == 0) return hipSuccess;
  frame_pairs_kernel<<<dim3((p.n_pairs + kPairWaves - 1) / kPairWaves),
                       dim3(64 * kPairWaves), 0, s>>>(p, w, pairs_out);
  return hipGetLastError();
}

hipError_t launch_e_ff(const DevPlan& p, const float* pairs,
                       int32_t n_layers, float* e_ff, hipStream_t s) {
  e_ff_kernel<<<dim3((p.T + kEffWaves - 1) / kEffWaves, n_layers),
                dim3(64 * kEffWaves), 0, s>>>(p, pairs, e_ff);
  return hipGetLastError();
}

hipError_t launch_combine_evidence(const DevPlan& p, const Workspace& w,
                                   const AttnCall& c, float* ev, float* tm,
                                   hipStream_t s) {
  const int n_fb = (p.T + kEvFrames - 1) / kEvFrames;
  const int blocks =
      p.n_tiles * p.hq + n_fb * p.hq + (tm ? p.hq * p.n_seq : 0);
  dim3 grid(blocks), block(kCeThreads);
  if (c.fp32) {
    if (c.d == 64)
      combine_evidence_kernel<64, true><<<grid, block, 0, s>>>(p, w, c, ev, tm);
    else
      combine_evidence_kernel<128, true><<<grid, block, 0, s>>>(p, w, c, ev,
                                                                tm);
  } else {
    if (c.d == 64)
      combine_evidence_kernel<64, false><<<grid, block, 0, s>>>(p, w, c, ev,
                                                                tm);
    else
      combine_evidence_kernel<128, false><<<grid, block, 0, s>>>(p, w, c, ev,
                                                                 tm);
  }
  return hipGetLastError();
}

hipError_t launch_frame_evidence(const DevPlan& p, const float* evidence,
                                 int32_t n_layers, float* e_qf_layer,
                                 float* e_qf, const int32_t* k_per_seq,
                                 int32_t* topk, hipStream_t s) {
  frame_mean_kernel<<<dim3((p.T + kFmFrames - 1) / kFmFrames),
                      dim3(kFmFrames * kFmLayers), 0, s>>>(
      p, evidence, n_layers, e_qf_layer, e_qf);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !k_per_seq) return e;
  topk_kernel<<<dim3(p.n_seq), dim3(kTopkThreads), 0, s>>>(p, e_qf, k_per_seq,
                                                           topk);
  return hipGetLastError();
}

}  // namespace evisel
