// Evidence reduction and frame aggregation (gfx950).
//
// evidence_kernel: E[h, f] = sum over the query rows r of f's video of
//   exp2(seg[h, r, f] - lse2[h, r]), i.e. each row's softmax mass on frame f
//   (the query-frame cue of Evidence Decomposition, kept as a raw sum over the
//   query rows). A work-group takes 64 frames of one head; 16 row groups sum
//   strided rows and are added in a fixed order in LDS, one store per
//   output: no atomics, bitwise reproducible. Adjacent threads read adjacent
//   frames of the same row, so every load is coalesced.
// frame_mean_kernel: E_qf[l, t] = sum_h E[l, h, t] / (Hq * n_text) and the
//   mean over layers (heads averaged per layer, layer kept); 32 frames x 32
//   layer groups per work-group, layers added in a fixed order.
// topk_kernel: per video, rank r(t) = #{t' : e(t') > e(t) or (e(t') == e(t)
//   and t' < t)}; frames with r(t) < k land at topk[offset + r(t)]. Ranks of a
//   strict total order are a permutation, so every slot gets one writer.
#include "kernels.h"

namespace evisel {
namespace {

__device__ __forceinline__ float exp2_(float x) {
  return __builtin_amdgcn_exp2f(x);
}

constexpr int kEvFrames = 64, kEvRows = 16;

__global__ __launch_bounds__(kEvFrames * kEvRows) void evidence_kernel(
    const DevPlan pl, const Workspace ws, float* __restrict__ ev,
    float* __restrict__ tm) {
  __shared__ float red[kEvRows][kEvFrames];
  const int h = blockIdx.y;
  const int fl = threadIdx.x % kEvFrames, rg = threadIdx.x / kEvFrames;
  const int f = blockIdx.x * kEvFrames + fl;
  float acc = 0.f;
  if (f < pl.T) {
    const SeqDesc sq = pl.seqs[pl.frame_seq[f]];
    const float* src = ws.seg + (size_t)h * pl.segtot + sq.segbase +
                       (f - sq.frame0);
    const float* l2 = ws.lse2t + (size_t)h * pl.n_text_rows + sq.textrow0;
#pragma unroll 4
    for (int r = rg; r < sq.n_text; r += kEvRows)
      acc += exp2_(src[(size_t)r * sq.n_frames] - l2[r]);
  }
  red[rg][fl] = acc;
  __syncthreads();
  if (rg == 0 && f < pl.T) {
    float t = 0.f;
#pragma unroll
    for (int i = 0; i < kEvRows; ++i) t += red[i][fl];
    ev[(size_t)h * pl.T + f] = t;
  }
  if (tm && blockIdx.x == 0) {
    for (int n = threadIdx.x; n < pl.n_seq; n += kEvFrames * kEvRows) {
      const SeqDesc sq = pl.seqs[n];
      float t = 0.f;
      for (int i = 0; i < sq.n_tiles; ++i)
        t += ws.tmpart[(size_t)h * pl.n_tiles + sq.tile0 + i];
      tm[(size_t)h * pl.n_seq + n] = t;
    }
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
  float acc = 0.f;
  for (int h = 0; h < pl.hq; ++h) {
    bool done = always;
    if (!always) {
      const int g0 = (h / group) * group;
      const int h0 = g0 + ((h - g0) / kHeadsPerItem) * kHeadsPerItem;
      const int nh = min(kHeadsPerItem, g0 + group - h0);
      unsigned wd = 0u;
      for (int i = 0; i < nh; ++i)
        wd |= ws.ubits[((size_t)(h0 + i) * pl.nb + fp.qblock) * pl.W +
                       (loc >> 5)];
      done = (wd >> (loc & 31)) & 1u;
    }
    if (done && rv) {
      const float sv =
          ws.segv[(((size_t)h * pl.nnz + fp.pos) * fpt + fp.koff) * 64 + row];
      const float l2 = ws.lse2v[(size_t)h * pl.S + qb.start + row];
      acc += exp2_(sv - l2);
    }
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

hipError_t launch_evidence(const DevPlan& p, const Workspace& w, float* ev,
                           float* tm, hipStream_t s) {
  dim3 grid((p.T + kEvFrames - 1) / kEvFrames, p.hq),
      block(kEvFrames * kEvRows);
  evidence_kernel<<<grid, block, 0, s>>>(p, w, ev, tm);
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
