// Block-sparse prefill attention for gfx950 with fused query-frame evidence
// partials, and the combine step of split query-token rows.
//
// Work item = one query block (a region block of <= 64 tokens), one query
// head and a run of that block's active key blocks (CSR). A work-group of two
// wavefronts owns the item; each wavefront owns 32 query rows.
//
// Per key tile (64 keys):
//   S^T = K Q^T        32x32x16 bf16 MFMA (fp32 inputs: 32x32x2 f32 MFMA);
//                      computing the transpose leaves one query row per lane
//                      (lane % 32), so row reductions stay inside the lane
//                      plus one exchange with lane ^ 32.
//   mask               only on tiles reaching past the first query row or
//                      shorter than 64 keys: keys after the row (causal) and
//                      past the block end.
//   online softmax     base-2 with log2(e) folded into the scale; the running
//                      reference max is only moved when the tile max exceeds
//                      it by more than 2^8, which keeps every probability
//                      below 256 and skips almost all accumulator rescales.
//   evidence           query-token rows only: the fp32 probabilities of each
//                      anchor frame's keys (frames of N_v | 64 keys never cross
//                      a tile) are summed and written once per (row, frame) as
//                      a log2 partial mass m_ref + log2(sum); non-visual keys
//                      (system prefix, query tokens) accumulate into one
//                      running partial per item.
//   O^T += V^T P^T     P rounded to bf16 (RNE) as the B operand straight from
//                      the S^T registers; V^T staged transposed in LDS.
// Key/value tiles are prefetched into registers during the previous tile's
// math and written to LDS between two barriers.
//
// Visual and system rows finish in the kernel (O, LSE). Query-token rows are
// split into chunks of key blocks (longest-first balance across the chip);
// each chunk leaves an unnormalised partial (acc, m_ref, row sum, non-visual
// mass) in the workspace and the combine kernel merges them.
#include "kernels.h"

namespace evisel {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kTile = 64;
constexpr int kWaves = 2;
constexpr int kThreads = 64 * kWaves;
constexpr float kLn2 = 0.69314718055994530942f;
constexpr float kRescaleSlack = 8.0f;  // log2 units

__device__ __forceinline__ float neg_inf() { return -__builtin_inff(); }
__device__ __forceinline__ float exp2_(float x) {
  return __builtin_amdgcn_exp2f(x);
}
__device__ __forceinline__ float log2_(float x) {
  return __builtin_amdgcn_logf(x);
}
__device__ __forceinline__ float partner(float x) { return __shfl_xor(x, 32); }

// ---------------------------------------------------------------------------
// bf16 operands: Q fragment in registers, K [key][d] and V^T [d][key] in LDS.
template <int D>
struct Bf16Path {
  static constexpr int KS = D + 8;       // padded K row (elements)
  static constexpr int VS = kTile + 4;   // padded V^T row (elements)
  static constexpr int KCH = kTile * D / 8 / kThreads;  // 16-B K chunks
  static constexpr int VGR = 16 * (D / 8) / kThreads;   // 4x8 V groups
  struct Smem {
    __bf16 k[kTile * KS];
    __bf16 vt[D * VS];
  };
  struct Stage {
    bf16x8 k[KCH];
    bf16x8 v[VGR][4];
  };
  struct QFrag {
    bf16x8 x[D / 16];
  };

  __device__ static void load_q(QFrag& qf, const void* q, int qpos, bool ok,
                                int h, int hq, int g) {
    const __bf16* src = (const __bf16*)q + ((size_t)qpos * hq + h) * D;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      bf16x8 z = {};
      qf.x[kk] = ok ? *(const bf16x8*)(src + 16 * kk + 8 * g) : z;
    }
  }

  __device__ static void fetch(Stage& st, const void* k, const void* v,
                               int kstart, int klen, int kvh, int hkv,
                               int tid) {
    const __bf16* kb = (const __bf16*)k;
    const __bf16* vb = (const __bf16*)v;
#pragma unroll
    for (int r = 0; r < KCH; ++r) {
      const int c = tid + kThreads * r;
      const int row = c / (D / 8), c8 = c % (D / 8);
      bf16x8 z = {};
      st.k[r] = row < klen
                    ? *(const bf16x8*)(kb + ((size_t)(kstart + row) * hkv +
                                             kvh) * D + c8 * 8)
                    : z;
    }
#pragma unroll
    for (int r = 0; r < VGR; ++r) {
      const int gi = tid + kThreads * r;
      const int kq = gi % 16, cc = gi / 16;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = 4 * kq + i;
        bf16x8 z = {};
        st.v[r][i] = row < klen
                         ? *(const bf16x8*)(vb + ((size_t)(kstart + row) * hkv +
                                                  kvh) * D + cc * 8)
                         : z;
      }
    }
  }

  __device__ static void commit(Smem& sm, const Stage& st, const void*,
                                const void*, int, int, int, int, int tid) {
#pragma unroll
    for (int r = 0; r < KCH; ++r) {
      const int c = tid + kThreads * r;
      const int row = c / (D / 8), c8 = c % (D / 8);
      *(bf16x8*)&sm.k[row * KS + c8 * 8] = st.k[r];
    }
#pragma unroll
    for (int r = 0; r < VGR; ++r) {
      const int gi = tid + kThreads * r;
      const int kq = gi % 16, cc = gi / 16;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        bf16x4 t = {st.v[r][0][e], st.v[r][1][e], st.v[r][2][e],
                    st.v[r][3][e]};
        *(bf16x4*)&sm.vt[(8 * cc + e) * VS + 4 * kq] = t;
      }
    }
  }

  // S^T[key][q] for the two 32-key halves of the tile.
  __device__ static void qk(f32x16 (&s)[2], const Smem& sm, const QFrag& qf,
                            int l32, int g) {
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const bf16x8 kf =
            *(const bf16x8*)&sm.k[(32 * c + l32) * KS + 16 * kk + 8 * g];
        s[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf.x[kk], s[c], 0,
                                                        0, 0);
      }
    }
  }

  // O^T[d][q] += V^T[d][key] P^T[key][q]. The B operand of k-step (c, s)
  // is the lane's own s[c][8s .. 8s+7], i.e. keys 32c + 16s + 8(e/4) +
  // 4g + e%4 for e = 0..7; the A operand reads V^T at the same keys.
  __device__ static void pv(f32x16 (&o)[D / 32], const Smem& sm,
                            const f32x16 (&p)[2], int l32, int g) {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const f32x8 pf = s == 0 ? __builtin_shufflevector(p[c], p[c], 0, 1, 2,
                                                          3, 4, 5, 6, 7)
                                : __builtin_shufflevector(p[c], p[c], 8, 9, 10,
                                                          11, 12, 13, 14, 15);
        const bf16x8 pb = __builtin_convertvector(pf, bf16x8);
#pragma unroll
        for (int mt = 0; mt < D / 32; ++mt) {
          const __bf16* row = &sm.vt[(32 * mt + l32) * VS + 32 * c + 16 * s];
          const bf16x4 lo = *(const bf16x4*)(row + 4 * g);
          const bf16x4 hi = *(const bf16x4*)(row + 8 + 4 * g);
          const bf16x8 va = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5,
                                                    6, 7);
          o[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, o[mt], 0, 0,
                                                          0);
        }
      }
    }
  }

  __device__ static void store_o(void* out, int qpos, int h, int hq, int d0,
                                 f32x4 v) {
    bf16x4 b = __builtin_convertvector(v, bf16x4);
    *(bf16x4*)((__bf16*)out + ((size_t)qpos * hq + h) * D + d0) = b;
  }
};

// ---------------------------------------------------------------------------
// fp32 operands (32x32x2 f32 MFMA). The contraction over d pairs element t
// of lane half g with d = g*D/2 + t, so every lane reads contiguous runs.
// V needs no transpose: each lane contributes one value per k-step.
template <int D>
struct F32Path {
  static constexpr int KS = D + 4;
  static constexpr int VS = D + 4;
  struct Smem {
    float k[kTile * KS];
    float v[kTile * VS];
  };
  struct Stage {};
  struct QFrag {
    float x[D / 2];
  };

  __device__ static void load_q(QFrag& qf, const void* q, int qpos, bool ok,
                                int h, int hq, int g) {
    const float* src = (const float*)q + ((size_t)qpos * hq + h) * D + g * D / 2;
#pragma unroll
    for (int u = 0; u < D / 8; ++u) {
      f32x4 z = {};
      const f32x4 t = ok ? *(const f32x4*)(src + 4 * u) : z;
#pragma unroll
      for (int j = 0; j < 4; ++j) qf.x[4 * u + j] = t[j];
    }
  }

  __device__ static void fetch(Stage&, const void*, const void*, int, int, int,
                               int, int) {}

  __device__ static void commit(Smem& sm, const Stage&, const void* k,
                                const void* v, int kstart, int klen, int kvh,
                                int hkv, int tid) {
    const float* kb = (const float*)k;
    const float* vb = (const float*)v;
    for (int c = tid; c < kTile * D / 4; c += kThreads) {
      const int row = c / (D / 4), c4 = c % (D / 4);
      f32x4 z = {};
      const size_t off = ((size_t)(kstart + row) * hkv + kvh) * D + c4 * 4;
      *(f32x4*)&sm.k[row * KS + c4 * 4] =
          row < klen ? *(const f32x4*)(kb + off) : z;
      *(f32x4*)&sm.v[row * VS + c4 * 4] =
          row < klen ? *(const f32x4*)(vb + off) : z;
    }
  }

  __device__ static void qk(f32x16 (&s)[2], const Smem& sm, const QFrag& qf,
                            int l32, int g) {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
#pragma unroll
      for (int u = 0; u < D / 8; ++u) {
        const f32x4 kf =
            *(const f32x4*)&sm.k[(32 * c + l32) * KS + g * D / 2 + 4 * u];
#pragma unroll
        for (int j = 0; j < 4; ++j)
          s[c] = __builtin_amdgcn_mfma_f32_32x32x2f32(kf[j], qf.x[4 * u + j],
                                                      s[c], 0, 0, 0);
      }
    }
  }

  __device__ static void pv(f32x16 (&o)[D / 32], const Smem& sm,
                            const f32x16 (&p)[2], int l32, int g) {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = 32 * c + 8 * (r >> 2) + 4 * g + (r & 3);
#pragma unroll
        for (int mt = 0; mt < D / 32; ++mt)
          o[mt] = __builtin_amdgcn_mfma_f32_32x32x2f32(
              sm.v[key * VS + 32 * mt + l32], p[c][r], o[mt], 0, 0, 0);
      }
    }
  }

  __device__ static void store_o(void* out, int qpos, int h, int hq, int d0,
                                 f32x4 v) {
    *(f32x4*)((float*)out + ((size_t)qpos * hq + h) * D + d0) = v;
  }
};

// ---------------------------------------------------------------------------
template <class P, int D>
__global__ __launch_bounds__(kThreads) void attn_kernel(const DevPlan pl,
                                                        const Workspace ws,
                                                        const AttnCall ac) {
  __shared__ typename P::Smem sm;
  const WorkItem it = pl.items[blockIdx.x];
  if (it.qblock < 0) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, g = lane >> 5;
  const BlockDesc qb = pl.blocks[it.qblock];
  const int h = it.head, kvh = h / (pl.hq / pl.hkv);
  const bool is_text = it.slot >= 0;
  const int qrow = 32 * wave + l32;
  const bool qvalid = qrow < qb.len;
  const int qpos = qb.start + qrow;
  const int n = it.kb_end - it.kb_begin;
  const float c2 = ac.scale_log2;

  typename P::QFrag qf;
  P::load_q(qf, ac.q, qpos, qvalid, h, pl.hq, g);

  float m_ref = neg_inf(), l_part = 0.f, nv_part = 0.f;
  f32x16 o[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) o[i] = f32x16{};

  typename P::Stage st;
  BlockDesc kb = pl.blocks[pl.col[it.kb_begin]];
  P::fetch(st, ac.k, ac.v, kb.start, kb.len, kvh, pl.hkv, tid);

  for (int j = 0; j < n; ++j) {
    __syncthreads();
    P::commit(sm, st, ac.k, ac.v, kb.start, kb.len, kvh, pl.hkv, tid);
    __syncthreads();
    const BlockDesc cur = kb;
    if (j + 1 < n) {
      kb = pl.blocks[pl.col[it.kb_begin + j + 1]];
      P::fetch(st, ac.k, ac.v, kb.start, kb.len, kvh, pl.hkv, tid);
    }

    f32x16 s[2] = {f32x16{}, f32x16{}};
    P::qk(s, sm, qf, l32, g);

    if (cur.len < kTile || cur.start + cur.len - 1 > qb.start) {
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int kl = 32 * c + 8 * (r >> 2) + 4 * g + (r & 3);
          if (kl >= cur.len || cur.start + kl > qpos) s[c][r] = neg_inf();
        }
    }

    float mx = neg_inf();
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[c][r]);
    mx = fmaxf(mx, partner(mx));
    const float m_new = fmaxf(m_ref, mx * c2);
    const bool need = m_new > m_ref + kRescaleSlack;
    if (__any(need)) {
      const float alpha = need ? exp2_(m_ref - m_new) : 1.f;
      l_part *= alpha;
      nv_part *= alpha;
#pragma unroll
      for (int i = 0; i < D / 32; ++i) o[i] *= alpha;
      m_ref = need ? m_new : m_ref;
    }
    const float mu = m_ref == neg_inf() ? 0.f : m_ref;
    float ts = 0.f;
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = exp2_(fmaf(s[c][r], c2, -mu));
        s[c][r] = p;
        ts += p;
      }
    l_part += ts;

    if (is_text) {
      if (cur.region == kVis) {
        // per 8-key group partial sums, completed across the lane pair
        float g8[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) g8[q] = 0.f;
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
          for (int r = 0; r < 16; ++r) g8[4 * c + (r >> 2)] += s[c][r];
#pragma unroll
        for (int q = 0; q < 8; ++q) g8[q] += partner(g8[q]);
        const int lg = __builtin_ctz((unsigned)pl.Nv) - 3;  // log2(N_v / 8)
        const int nseg = kTile / pl.Nv;
        const SeqDesc sq = pl.seqs[it.seq];
        const int trow = qb.aux + qrow - sq.textrow0;
        float* dst = ws.seg + (size_t)h * pl.segtot + sq.segbase +
                     (size_t)trow * sq.n_frames + (cur.aux - sq.frame0);
        for (int si = 0; si < nseg; ++si) {
          float t = 0.f;
#pragma unroll
          for (int q = 0; q < 8; ++q) t += (q >> lg) == si ? g8[q] : 0.f;
          if (g == 0 && qvalid && si * pl.Nv < cur.len)
            dst[si] = mu + log2_(t);
        }
      } else {
        nv_part += ts;
      }
    }

    P::pv(o, sm, s, l32, g);
  }

  const float l_tot = l_part + partner(l_part);
  if (!is_text) {
    if (qvalid) {
      const float inv = 1.f / l_tot;
#pragma unroll
      for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          f32x4 v = {o[mt][4 * r4] * inv, o[mt][4 * r4 + 1] * inv,
                     o[mt][4 * r4 + 2] * inv, o[mt][4 * r4 + 3] * inv};
          P::store_o(ac.o, qpos, h, pl.hq, 32 * mt + 8 * r4 + 4 * g, v);
        }
      if (g == 0 && ac.lse)
        ac.lse[(size_t)h * pl.S + qpos] = (m_ref + log2_(l_tot)) * kLn2;
    }
  } else {
    const float nv_tot = nv_part + partner(nv_part);
    if (qvalid) {
      float* po = ws.pO + ((size_t)it.slot * kTile + qrow) * D;
#pragma unroll
      for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          f32x4 v = {o[mt][4 * r4], o[mt][4 * r4 + 1], o[mt][4 * r4 + 2],
                     o[mt][4 * r4 + 3]};
          *(f32x4*)(po + 32 * mt + 8 * r4 + 4 * g) = v;
        }
      if (g == 0) {
        const size_t ix = (size_t)it.slot * kTile + qrow;
        ws.pM[ix] = m_ref;
        ws.pL[ix] = l_tot;
        ws.pNV[ix] = nv_tot > 0.f ? m_ref + log2_(nv_tot) : neg_inf();
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Merge the chunks of a query-token tile: one work-group per (tile, head),
// four threads per row. Also leaves the rows' log2 LSE for the evidence
// reduction and the tile's non-visual mass.
template <int D, bool F32>
__global__ __launch_bounds__(256) void combine_kernel(const DevPlan pl,
                                                      const Workspace ws,
                                                      const AttnCall ac) {
  constexpr int DP = D / 4;
  __shared__ float red[kTile];
  const TextTile tt = pl.tiles[blockIdx.x];
  const int h = blockIdx.y;
  const BlockDesc qb = pl.blocks[tt.qblock];
  const int tid = threadIdx.x, r = tid >> 2, part = tid & 3;
  float nvmass = 0.f;
  if (r < qb.len) {
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
      f32x4 v = {acc[i] * inv, acc[i + 1] * inv, acc[i + 2] * inv,
                 acc[i + 3] * inv};
      const size_t off = ((size_t)qpos * pl.hq + h) * D + part * DP + i;
      if (F32) {
        *(f32x4*)((float*)ac.o + off) = v;
      } else {
        *(bf16x4*)((__bf16*)ac.o + off) = __builtin_convertvector(v, bf16x4);
      }
    }
    const float lse2 = M + log2_(L);
    if (part == 0) {
      if (ac.lse) ac.lse[(size_t)h * pl.S + qpos] = lse2 * kLn2;
      ws.lse2t[(size_t)h * pl.n_text_rows + qb.aux + r] = lse2;
      for (int c = 0; c < tt.n_chunks; ++c)
        nvmass += exp2_(ws.pNV[(size_t)(slot0 + c) * kTile + r] - lse2);
    }
  }
  if (part == 0) red[r] = nvmass;
  __syncthreads();
  if (tid == 0) {
    float t = 0.f;
    for (int i = 0; i < kTile; ++i) t += red[i];
    ws.tmpart[(size_t)h * pl.n_tiles + blockIdx.x] = t;
  }
}

}  // namespace

hipError_t launch_attention(const DevPlan& p, const Workspace& w,
                            const AttnCall& c, hipStream_t s) {
  if (p.n_items == 0) return hipSuccess;
  dim3 grid(p.n_items), block(kThreads);
  if (c.fp32) {
    if (c.d == 64)
      attn_kernel<F32Path<64>, 64><<<grid, block, 0, s>>>(p, w, c);
    else
      attn_kernel<F32Path<128>, 128><<<grid, block, 0, s>>>(p, w, c);
  } else {
    if (c.d == 64)
      attn_kernel<Bf16Path<64>, 64><<<grid, block, 0, s>>>(p, w, c);
    else
      attn_kernel<Bf16Path<128>, 128><<<grid, block, 0, s>>>(p, w, c);
  }
  return hipGetLastError();
}

hipError_t launch_combine(const DevPlan& p, const Workspace& w,
                          const AttnCall& c, hipStream_t s) {
  if (p.n_tiles == 0) return hipSuccess;
  dim3 grid(p.n_tiles, p.hq), block(256);
  if (c.fp32) {
    if (c.d == 64)
      combine_kernel<64, true><<<grid, block, 0, s>>>(p, w, c);
    else
      combine_kernel<128, true><<<grid, block, 0, s>>>(p, w, c);
  } else {
    if (c.d == 64)
      combine_kernel<64, false><<<grid, block, 0, s>>>(p, w, c);
    else
      combine_kernel<128, false><<<grid, block, 0, s>>>(p, w, c);
  }
  return hipGetLastError();
}

}  // namespace evisel
