// Adaptive top-p block retention for gfx950 (appendix "Detailed Sparse
// Prefilling": mean-key block representative, block affinity over the
// history H_i, softmax over H_i, smallest subset whose probability reaches
// tau_p).
//
// pool_kernel    kbar_j = mean of block j's keys per kv head, an fp32 sum in
//                token order divided by the block length. For bf16 inputs
//                kbar is kept as two bf16 values, hi = RNE(kbar) and
//                lo = RNE(kbar - hi), so the affinity can run on bf16 MFMA
//                while kbar keeps about 16 significant bits; both arrays are
//                d-chunk-major ([kv head][d / 8][block][8]), so the 32
//                blocks of one MFMA operand load are contiguous.
// select_kernel  one work-group per (query block, query head), launched
//                longest history first (see the kernel). The block's
//                rows share their history (local blocks 0 .. nh-1 of the
//                video). Each pass's query rows are staged in LDS once per
//                work-group (bf16). Affinities g = q . kbar * scale *
//                log2(e) come from 32x32x16 bf16 MFMA, hi and lo accumulated
//                into one fp32 tile (fp32 inputs: 32x32x2 f32 MFMA), and are
//                staged in LDS,
//                each row owned by TPR consecutive lanes (TPR/4 quads). Per
//                row: e_j = exp2(g_j - max), Z = sum e_j, threshold
//                tau * Z. The retained set is {j : e_j >= t*} for the
//                largest t* whose tail mass F(t*) = sum_{e_j >= t*} e_j still
//                reaches the threshold. t* is found by bisection over the
//                bit patterns of the non-negative fp32 e_j (ordered like the
//                values), stopping once a single candidate value is left;
//                after four passes over all entries, each lane copies the
//                few entries still inside the bracket to its LDS slice and
//                the remaining passes read only those. When several e_j
//                equal t*, they are retained in ascending block order until
//                the threshold is reached. Every sum runs in a fixed order
//                and the lanes of a row see identical reductions, so the
//                result is bitwise reproducible.
// seg_fill_kernel  -inf into the per-(row, frame) partial masses before a
//                top-p attention pass (tiles that no row of a work item
//                retained are skipped and write nothing).
#include <algorithm>

#include "kernels.h"

namespace evisel {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kSelThreads = 256;
constexpr int kTile64 = 64;
constexpr size_t kSelLdsTwoPerCu = 80 * 1024;
constexpr size_t kSelLdsMax = 160 * 1024;

__device__ __forceinline__ float neg_inf() { return -__builtin_inff(); }

template <bool F32, int D>
__global__ __launch_bounds__(D) void pool_kernel(const DevPlan pl,
                                                 const void* __restrict__ k,
                                                 void* __restrict__ kbar) {
  const int b = blockIdx.x, kvh = blockIdx.y, c = threadIdx.x;
  const BlockDesc bd = pl.blocks[b];
  if (bd.region == kSys) return;
  const size_t rs = (size_t)pl.hkv * D;
  const size_t base = ((size_t)bd.start * pl.hkv + kvh) * D + c;
  // a whole 64-token block's loads in flight (one round trip), then their
  // sum in token order
  float s = 0.f;
  for (int r0 = 0; r0 < bd.len; r0 += kTile64) {
    float x[kTile64];
#pragma unroll
    for (int i = 0; i < kTile64; ++i) {
      const int r = min(r0 + i, bd.len - 1);
      x[i] = F32 ? ((const float*)k)[base + r * rs]
                 : (float)((const __bf16*)k)[base + r * rs];
    }
#pragma unroll
    for (int i = 0; i < kTile64; ++i)
      if (r0 + i < bd.len) s += x[i];
  }
  const float m = s / (float)bd.len;
  if (F32) {
    ((float*)kbar)[((size_t)kvh * pl.nb + b) * D + c] = m;
  } else {
    // d-chunk-major: the 8-element chunk c / 8 of every block is
    // contiguous, so a 32-block MFMA operand load reads 512 bytes in a row
    const size_t o = (((size_t)kvh * (D / 8) + c / 8) * pl.nb + b) * 8 + (c & 7);
    const __bf16 hi = (__bf16)m;
    const __bf16 lo = (__bf16)(m - (float)hi);
    ((__bf16*)kbar)[o] = hi;
    ((__bf16*)kbar)[(size_t)pl.hkv * pl.nb * D + o] = lo;
  }
}

// Reductions over the TPR lanes of a row (TPR = 4, 8 or 16 consecutive
// lanes). Each step combines a lane with a partner that holds the same
// partial as the lane's own mirror image, so every lane of the group ends
// with the same bits (fp addition is commutative).
template <int CTRL>
__device__ __forceinline__ int dpp(int x) {
  return __builtin_amdgcn_update_dpp(0, x, CTRL, 0xF, 0xF, true);
}
template <int CTRL>
__device__ __forceinline__ float dppf(float x) {
  return __builtin_bit_cast(float, dpp<CTRL>(__builtin_bit_cast(int, x)));
}
constexpr int kQuadSwap1 = 0xB1;      // quad_perm [1, 0, 3, 2]
constexpr int kQuadSwap2 = 0x4E;      // quad_perm [2, 3, 0, 1]
constexpr int kHalfMirror = 0x141;    // lane i <-> 7 - i within 8
constexpr int kRowMirror = 0x140;     // lane i <-> 15 - i within 16

template <int TPR>
__device__ __forceinline__ float grp_sum(float x) {
  x += dppf<kQuadSwap1>(x);
  x += dppf<kQuadSwap2>(x);
  if (TPR >= 8) x += dppf<kHalfMirror>(x);
  if (TPR >= 16) x += dppf<kRowMirror>(x);
  return x;
}
template <int TPR>
__device__ __forceinline__ int grp_sumi(int x) {
  x += dpp<kQuadSwap1>(x);
  x += dpp<kQuadSwap2>(x);
  if (TPR >= 8) x += dpp<kHalfMirror>(x);
  if (TPR >= 16) x += dpp<kRowMirror>(x);
  return x;
}
template <int TPR>
__device__ __forceinline__ float grp_max(float x) {
  x = fmaxf(x, dppf<kQuadSwap1>(x));
  x = fmaxf(x, dppf<kQuadSwap2>(x));
  if (TPR >= 8) x = fmaxf(x, dppf<kHalfMirror>(x));
  if (TPR >= 16) x = fmaxf(x, dppf<kRowMirror>(x));
  return x;
}
template <int TPR>
__device__ __forceinline__ unsigned grp_minu(unsigned x) {
  x = min(x, (unsigned)dpp<kQuadSwap1>((int)x));
  x = min(x, (unsigned)dpp<kQuadSwap2>((int)x));
  if (TPR >= 8) x = min(x, (unsigned)dpp<kHalfMirror>((int)x));
  if (TPR >= 16) x = min(x, (unsigned)dpp<kRowMirror>((int)x));
  return x;
}
template <int TPR>
__device__ __forceinline__ unsigned grp_maxu(unsigned x) {
  x = max(x, (unsigned)dpp<kQuadSwap1>((int)x));
  x = max(x, (unsigned)dpp<kQuadSwap2>((int)x));
  if (TPR >= 8) x = max(x, (unsigned)dpp<kHalfMirror>((int)x));
  if (TPR >= 16) x = max(x, (unsigned)dpp<kRowMirror>((int)x));
  return x;
}

// Values per thread and LDS row stride (in floats) for a history of nh
// blocks; both multiples of 4 so rows can be read as 16-byte vectors.
__host__ __device__ inline int sel_per_thread(int nh, int tpr) {
  return ((nh + tpr - 1) / tpr + 3) & ~3;
}
__host__ __device__ inline int sel_stride(int nh, int tpr) {
  return tpr * sel_per_thread(nh, tpr) + 4;
}
// LDS floats ahead of the per-row bit words: a pass's affinities
// [rows][stride] for the longest history, which also hold the pass's query
// rows ([rows][d + 8] bf16) while they are read into registers.
__host__ __device__ inline int sel_region0(int nh_max, int tpr, int d) {
  const int rpw = kSelThreads / tpr;
  const int ev = rpw * sel_stride(nh_max, tpr), qs = rpw * (d + 8) / 2;
  return ev > qs ? ev : qs;
}
inline size_t sel_lds_bytes(int nh_max, int tpr, int W, int d) {
  return (size_t)(sel_region0(nh_max, tpr, d) + 64 * W) * 4;
}

// Retention of one row whose TPR lanes hold e-candidates g_j (log2 units) in
// LDS, entries [j0, j0 + cnt) of the row's history at my[0 .. cnt). Sets the
// retained history bits in wrow (LDS, OR). retain_row_regs keeps the lane's
// L <= RV values in registers (RV = kRegVals, or kRegValsLong for the long
// form), retain_row_lds streams them from LDS.
// Both find the same cut except where a tail sum F lies within its fp32
// rounding of the threshold (they associate the sums differently).
//
// The bisection keeps F(lo) >= thr > F(hi), and clo - chi counts the
// entries inside [lo, hi) (the register variant takes that count only when
// it copies them). Each lane keeps a, its partial sum of the entries at or
// above hi; the lanes' partials of F(mid) are summed over the row in a
// fixed tree. The LDS variant takes a lane's partial as a plus its entries
// in [mid, hi) in index order. The register variant runs four passes over
// all its entries, each partial the sum of the lane's entries >= mid in
// index order, then copies the few entries still inside [lo, hi), in order,
// into the lane's LDS slice and runs the remaining passes over that list,
// each partial a plus the list entries >= mid, with a frozen at the copy
// (the list holds nothing at or above that hi, and entries below lo lie
// below every later mid). Every entry test is then one compare.
constexpr int kRegVals = 36;
constexpr int kRegValsLong = 72;   // the long form, 16 lanes per row
// Passes over every entry before the copy: a full pass costs three VALU
// instructions per entry, a pass over the copied list four and a half per
// entry of the wave's longest list, so narrowing the lists first pays up to
// four passes on rows of a few hundred near-uniform block affinities.
constexpr int kFullPasses = 4;

// Bits [j0, j0 + n) of a row from a lane's mask (n <= 64, j0 % 4 == 0).
__device__ __forceinline__ void or_bits(uint32_t* wrow, int j0,
                                        unsigned long long m) {
  if (!m) return;
  const int w0 = j0 >> 5, off = j0 & 31;
  const unsigned long long lo = m << off;
  const unsigned long long hi = off ? m >> (64 - off) : 0ull;
  if ((unsigned)lo) atomicOr(wrow + w0, (unsigned)lo);
  if ((unsigned)(lo >> 32)) atomicOr(wrow + w0 + 1, (unsigned)(lo >> 32));
  if ((unsigned)hi) atomicOr(wrow + w0 + 2, (unsigned)hi);
}
// The same from NW 32-bit words (bit i of the lane's mask in word i / 32).
template <int NW>
__device__ __forceinline__ void or_bits_w(uint32_t* wrow, int j0,
                                          const unsigned (&m)[NW]) {
  const int w0 = j0 >> 5, off = j0 & 31;
#pragma unroll
  for (int k = 0; k <= NW; ++k) {
    const unsigned cur = k < NW ? m[k] << off : 0u;
    const unsigned prev = k > 0 && off ? m[k - 1] >> (32 - off) : 0u;
    if (cur | prev) atomicOr(wrow + w0 + k, cur | prev);
  }
}

// One bisection step from the lane's partial f = a + (its entries in
// [mid, hi)) and their count k.
template <int TPR>
__device__ __forceinline__ void bisect_step(float f, int k, unsigned mid,
                                            float thr, unsigned& lo,
                                            unsigned& hi, int& clo, int& chi,
                                            float& fhi, float& a) {
  const float F = grp_sum<TPR>(f);
  const int K = chi + grp_sumi<TPR>(k);          // entries >= mid
  if (F >= thr) {
    lo = mid;
    clo = K;
  } else {
    hi = mid;
    chi = K;
    fhi = F;
    a = f;
  }
}

// Ties at lo (several entries with the bit pattern lo and F(lo + 1) < thr):
// how many of them to take, in ascending block order, and how many of them
// lie in this lane's lower-numbered neighbours.
template <int TPR>
__device__ __forceinline__ void tie_share(int mine, float fhi, float thr,
                                          unsigned lo, int nt, int lane,
                                          int part, int& take, int& rank) {
  const float et = __uint_as_float(lo);
  float cum = fhi;
  take = 0;
  while (take < nt && cum < thr) {
    cum += et;
    ++take;
  }
  rank = 0;
  for (int q2 = 0; q2 < TPR; ++q2) {
    const int o = __shfl(mine, lane - part + q2);
    rank += q2 < part ? o : 0;
  }
}

template <int TPR, int RV>
__device__ __forceinline__ void retain_row_regs(float* my, int L, int nh,
                                                int j0, float tau, int lane,
                                                int part, uint32_t* wrow) {
  constexpr int NCK = RV / 4;
  constexpr int NW = (RV + 31) / 32;   // mask words
  const int nck = L >> 2;                         // uniform per work-group
  // Entries past the history hold -inf (the affinity pass writes the row
  // up to TPR * L), so their e is +0; the cut t* found below is never 0 (F
  // at any key up to the smallest positive e is the whole sum Z >= tau Z),
  // so zeros are never retained or counted as ties, and no validity mask
  // is needed.
  float v[RV];
#pragma unroll
  for (int c = 0; c < NCK; ++c) {
    f32x4 t = {};
    if (c < nck) t = *(const f32x4*)(my + 4 * c);
#pragma unroll
    for (int e = 0; e < 4; ++e) v[4 * c + e] = t[e];
  }
  // (chunks c >= nck hold no entries: skipped, and +0 from here on)
  float mx = neg_inf();
#pragma unroll
  for (int c = 0; c < NCK; ++c)
    if (c < nck)
#pragma unroll
      for (int e = 0; e < 4; ++e) mx = fmaxf(mx, v[4 * c + e]);
  mx = grp_max<TPR>(mx);
  float z = 0.f;
  unsigned kmin = 0xFFFFFFFFu;
#pragma unroll
  for (int c = 0; c < NCK; ++c) {
    if (c < nck) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float x = __builtin_amdgcn_exp2f(v[4 * c + e] - mx);
        v[4 * c + e] = x;
        z += x;
        kmin = min(kmin, __float_as_uint(x) - 1u);  // +0 wraps to the top
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) v[4 * c + e] = 0.f;
    }
  }
  z = grp_sum<TPR>(z);
  kmin = grp_minu<TPR>(kmin) + 1u;
  const float thr = tau * z;
  // the row's largest e is exp2(0) = 1 exactly
  unsigned lo = kmin, hi = __float_as_uint(1.f) + 1u;
  int clo = nh, chi = 0;
  float fhi = 0.f, a = 0.f;
  // The full passes count nothing: a bracket that already holds a single
  // entry only narrows around it, which keeps the same retained set. The
  // count of entries inside the bracket is taken when they are copied.
  for (int it = 0; it < kFullPasses && hi - lo > 1u; ++it) {
    const unsigned mid = lo + ((hi - lo) >> 1);
    float f = 0.f;   // all of the lane's entries >= mid
#pragma unroll
    for (int c = 0; c < NCK; ++c) {
      if (c < nck) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const bool in = __float_as_uint(v[4 * c + e]) >= mid;
          f += in ? v[4 * c + e] : 0.f;
        }
      }
    }
    const float F = grp_sum<TPR>(f);
    if (F >= thr) {
      lo = mid;
    } else {
      hi = mid;
      fhi = F;
      a = f;
    }
  }
  if (hi - lo <= 1u) {
    // [lo, hi) = {lo}: its entries (every lane of the row sees the count)
    int mine = 0;
#pragma unroll
    for (int c = 0; c < NCK; ++c)
      if (c < nck)
#pragma unroll
        for (int e = 0; e < 4; ++e) mine += __float_as_uint(v[4 * c + e]) == lo;
    clo = grp_sumi<TPR>(mine);
  } else {
    // the lane's entries in [lo, hi), in index order, to my[0 .. n), then
    // zeros up to a multiple of 4 (n <= L, a multiple of 4; +0 lies below
    // every lo). Each store lands at or below the entry's own slot.
    const unsigned span = hi - lo;
    int n = 0;
#pragma unroll
    for (int c = 0; c < NCK; ++c) {
      if (c < nck) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          my[n] = v[4 * c + e];
          n += __float_as_uint(v[4 * c + e]) - lo < span;
        }
      }
    }
    const int n4 = (n + 3) & ~3;
    for (int i = n; i < n4; ++i) my[i] = 0.f;
    // from here a lane's partial is a (frozen) plus its list entries >= mid;
    // clo and chi count the list entries >= lo and >= hi
    clo = grp_sumi<TPR>(n);
    chi = 0;
    while (hi - lo > 1u && clo - chi > 1) {
      const unsigned mid = lo + ((hi - lo) >> 1);
      float f = a;
      int k = 0;
      for (int i = 0; i < n4; i += 4) {
        const f32x4 t = *(const f32x4*)(my + i);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const bool in = __float_as_uint(t[e]) >= mid;
          f += in ? t[e] : 0.f;
          k += in;
        }
      }
      const float F = grp_sum<TPR>(f);
      const int K = grp_sumi<TPR>(k);
      if (F >= thr) {
        lo = mid;
        clo = K;
      } else {
        hi = mid;
        chi = K;
        fhi = F;
      }
    }
  }
  unsigned mw[NW];
#pragma unroll
  for (int k = 0; k < NW; ++k) mw[k] = 0u;
  if (clo - chi <= 1) {
    // no tie: the entries >= lo
#pragma unroll
    for (int c = 0; c < NCK; ++c) {
      if (c < nck) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int i = 4 * c + e;
          const bool sel = __float_as_uint(v[i]) >= lo;
          mw[i >> 5] |= sel ? 1u << (i & 31) : 0u;
        }
      }
    }
  } else {
    int mine = 0;
#pragma unroll
    for (int i = 0; i < RV; ++i) mine += __float_as_uint(v[i]) == lo;
    int take, rank;
    tie_share<TPR>(mine, fhi, thr, lo, clo - chi, lane, part, take, rank);
#pragma unroll
    for (int i = 0; i < RV; ++i) {
      const unsigned kb = __float_as_uint(v[i]);
      bool sel = kb > lo;
      if (kb == lo) sel = rank++ < take;
      mw[i >> 5] |= sel ? 1u << (i & 31) : 0u;
    }
  }
  or_bits_w<NW>(wrow, j0, mw);
}

template <int TPR>
__device__ __forceinline__ void retain_row_lds(float* my, int L, int cnt,
                                               int nh, int j0, float tau,
                                               int lane, int part,
                                               uint32_t* wrow) {
  float mx = neg_inf();
  for (int i = 0; i < L; i += 4) {
    const f32x4 t = *(const f32x4*)(my + i);
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (i + e < cnt) mx = fmaxf(mx, t[e]);
  }
  mx = grp_max<TPR>(mx);
  float z = 0.f;
  unsigned kmin = 0xFFFFFFFFu, kmax = 0u;
  for (int i = 0; i < L; i += 4) {
    f32x4 t = *(const f32x4*)(my + i);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float x = i + e < cnt ? __builtin_amdgcn_exp2f(t[e] - mx) : 0.f;
      t[e] = x;
      z += x;
      const unsigned kb = __float_as_uint(x);
      kmin = min(kmin, kb - 1u);
      kmax = max(kmax, kb);
    }
    *(f32x4*)(my + i) = t;
  }
  z = grp_sum<TPR>(z);
  kmin = grp_minu<TPR>(kmin) + 1u;
  kmax = grp_maxu<TPR>(kmax);
  const float thr = tau * z;
  unsigned lo = kmin, hi = kmax + 1u;
  int clo = nh, chi = 0;
  float fhi = 0.f, a = 0.f;
  while (hi - lo > 1u && clo - chi > 1) {
    const unsigned mid = lo + ((hi - lo) >> 1), span = hi - mid;
    float f = a;
    int k = 0;
#pragma unroll 2
    for (int i = 0; i < L; i += 4) {
      const f32x4 t = *(const f32x4*)(my + i);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bool in = __float_as_uint(t[e]) - mid < span;
        f += in ? t[e] : 0.f;
        k += in;
      }
    }
    bisect_step<TPR>(f, k, mid, thr, lo, hi, clo, chi, fhi, a);
  }
  const bool tie = clo - chi > 1;
  int take = 0, rank = 0;
  if (tie) {
    int mine = 0;
    for (int i = 0; i < cnt; ++i) mine += __float_as_uint(my[i]) == lo;
    tie_share<TPR>(mine, fhi, thr, lo, clo - chi, lane, part, take, rank);
  }
  // 32 entries at a time (j0 % 4 == 0, so a run covers at most 2 words)
  for (int i0 = 0; i0 < cnt; i0 += 32) {
    unsigned long long m = 0ull;
    for (int i = i0; i < min(cnt, i0 + 32); ++i) {
      const unsigned kb = __float_as_uint(my[i]);
      bool sel = kb >= lo;
      if (tie && kb == lo) sel = rank++ < take;
      m |= (unsigned long long)sel << (i - i0);
    }
    or_bits(wrow, j0 + i0, m);
  }
}

// One 32x32 affinity tile's column share of a lane (row er of ev): columns
// 32 t + 8 (r / 4) + 4 g + r % 4 for r < 16. A tile wholly inside the
// history (the usual case, uniform over the wave) stores them unchecked.
__device__ __forceinline__ void store_affinities(const f32x16& acc, float sc,
                                                 float* er, int t, int g,
                                                 int nh, int ncols, bool rv) {
  if (!rv) return;
  float* const e0 = er + 32 * t + 4 * g;
  if (32 * t + 32 <= nh) {
#pragma unroll
    for (int r = 0; r < 16; ++r) e0[8 * (r >> 2) + (r & 3)] = acc[r] * sc;
  } else {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int j = 32 * t + 8 * (r >> 2) + 4 * g + (r & 3);
      if (j < ncols) e0[8 * (r >> 2) + (r & 3)] = j < nh ? acc[r] * sc
                                                        : neg_inf();
    }
  }
}

// Affinities g = q . kbar * scale * log2(e) of rows r0 + rl (rl < rows) of
// query block qb, head h, against its history blocks j < nh (global block
// first + j), written to ev[rl * stride + j]; columns nh <= j < ncols
// (ncols <= stride) get -inf. A wave takes the 32-row group rg and every
// wpg-th 32-column tile from ph: S^T = Kbar Q^T on bf16 MFMA with kbar =
// hi + lo accumulated into one fp32 tile (fp32: 32x32x2 MFMA).
template <bool F32, int D>
__device__ __forceinline__ void affinity_tiles(
    const DevPlan& pl, const void* kbar, const void* q, float scale_log2,
    const BlockDesc& qb, int h, int kvh, int first, int nh, int ncols,
    int r0, int rows, int rg, int ph, int wpg, float* ev, int stride,
    int lane, const __bf16* qs = nullptr) {
  const int l32 = lane & 31, g = lane >> 5;
  const int ntile = (ncols + 31) / 32;
  const int rl = rg * 32 + l32;
  const bool rv = rl < rows && r0 + rl < qb.len;
  // rows past the block read the block's first row; their affinities are
  // never stored
  const size_t qoff = ((size_t)(qb.start + (rv ? r0 + rl : 0)) * pl.hq + h) * D;
  if (!F32) {
    bf16x8 qf[D / 16];
    if (qs) {
      // rows staged in LDS by the whole work-group ([rows][D + 8]); every
      // wave has its operands before the first affinity overwrites them
      const __bf16* qr = qs + min(rl, rows - 1) * (D + 8) + 8 * g;
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk)
        qf[kk] = *(const bf16x8*)(qr + 16 * kk);
      __syncthreads();
    } else {
      const __bf16* qg = (const __bf16*)q + qoff + 8 * g;
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk)
        qf[kk] = *(const bf16x8*)(qg + 16 * kk);
    }
    // chunk 2 kk + g of block first + jb (d-chunk-major layout)
    const __bf16* kh0 = (const __bf16*)kbar +
                        (((size_t)kvh * (D / 8) + g) * pl.nb + first) * 8;
    const size_t lo_off = (size_t)pl.hkv * pl.nb * D;
    const size_t kk_step = (size_t)2 * pl.nb * 8;
    for (int t = ph; t < ntile; t += wpg) {
      const int jb = min(32 * t + l32, nh - 1);
      const __bf16* kh = kh0 + (size_t)jb * 8;
      // the tile's operand loads in two halves of D / 32 chunks each
      f32x16 acc = {};
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        constexpr int HK = D / 32;
        bf16x8 ah[HK], al[HK];
#pragma unroll
        for (int u = 0; u < HK; ++u) {
          const int kk = hf * HK + u;
          ah[u] = *(const bf16x8*)(kh + kk * kk_step);
          al[u] = *(const bf16x8*)(kh + lo_off + kk * kk_step);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < HK; ++u) {
          const int kk = hf * HK + u;
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah[u], qf[kk], acc, 0,
                                                        0, 0);
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al[u], qf[kk], acc, 0,
                                                        0, 0);
        }
      }
      store_affinities(acc, scale_log2, ev + rl * stride, t, g, nh, ncols, rv);
    }
  } else {
    float qf[D / 2];
    const float* qs = (const float*)q + qoff + g * (D / 2);
#pragma unroll
    for (int u = 0; u < D / 8; ++u) {
      f32x4 z = {};
      const f32x4 v = rv ? *(const f32x4*)(qs + 4 * u) : z;
#pragma unroll
      for (int e = 0; e < 4; ++e) qf[4 * u + e] = v[e];
    }
    const float* k0 =
        (const float*)kbar + ((size_t)kvh * pl.nb + first) * D + g * (D / 2);
    for (int t = ph; t < ntile; t += wpg) {
      const int jb = min(32 * t + l32, nh - 1);
      const float* kr = k0 + (size_t)jb * D;
      f32x16 acc = {};
#pragma unroll
      for (int u = 0; u < D / 8; ++u) {
        const f32x4 a = *(const f32x4*)(kr + 4 * u);
#pragma unroll
        for (int e = 0; e < 4; ++e)
          acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[e], qf[4 * u + e], acc,
                                                     0, 0, 0);
      }
      store_affinities(acc, scale_log2, ev + rl * stride, t, g, nh, ncols, rv);
    }
  }
}

// Four waves per SIMD (at most 128 registers): the per-row bisection is a
// chain of dependent VALU steps and reductions, and more resident waves hide
// its latency better than the registers an unconstrained allocation keeps.
// RV: a lane's values held in registers. The long form (RV > kRegVals,
// histories of up to 16 RV blocks at 16 lanes per row) needs about 80 KB of
// LDS per work-group, which already limits a CU to two of them, so it takes
// up to 256 registers at two waves per SIMD.
template <bool F32, int D, int TPR, int RV>
__global__ __launch_bounds__(kSelThreads) __attribute__((amdgpu_waves_per_eu(
    RV > kRegVals ? 2 : 4, RV > kRegVals ? 2 : 4))) void select_kernel(
    const DevPlan pl, const Workspace ws, const SelCall sc) {
  constexpr int RPW = kSelThreads / TPR;          // rows per pass
  constexpr int NRG = RPW >= 32 ? RPW / 32 : 1;   // 32-row MFMA groups
  constexpr int WPG = 4 / NRG;                    // waves per row group
  extern __shared__ __attribute__((aligned(16))) float dyn[];
  // one-dimensional grid, heads fastest, query blocks from the last: in a
  // video the history grows with the block index, so the longest
  // work-groups start first and the shortest fill the tail, and all heads
  // of one block (which read whole token rows of q between them) run
  // together
  const int qbid = pl.nb - 1 - (int)blockIdx.x / pl.hq;
  const int h = (int)blockIdx.x % pl.hq;
  const BlockDesc qb = pl.blocks[qbid];
  const int nh = pl.blk_local[qbid];              // |H|; -1 for system rows
  const int W = pl.W;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  uint32_t* const rb = sc.rbits + ((size_t)h * pl.nb + qbid) * W * 64;
  uint32_t* const ub = sc.ubits + ((size_t)h * pl.nb + qbid) * W;
  if (nh <= 0) {                                  // empty history
    for (int i = tid; i < W * 64; i += kSelThreads) rb[i] = 0u;
    for (int i = tid; i < W; i += kSelThreads) ub[i] = 0u;
    return;
  }
  const int L = sel_per_thread(nh, TPR);
  const int stride = sel_stride(nh, TPR);
  float* const ev = dyn;                                  // [RPW][stride]
  uint32_t* const wb =                                    // [64][W]
      (uint32_t*)(dyn + sel_region0(max(pl.hmax, 1), TPR, D));
  for (int i = tid; i < 64 * W; i += kSelThreads) wb[i] = 0u;

  const int kvh = h / (pl.hq / pl.hkv);
  const int first = qbid - nh;                    // global id of local 0
  const int rg = wave % NRG, ph = wave / NRG;

  for (int r0 = 0; r0 < qb.len; r0 += RPW) {
    // ---- affinities of rows r0 .. r0 + RPW - 1 against the history ----
    __bf16* qs = nullptr;
    if (!F32) {
      // the pass's query rows to LDS in whole 16-byte chunks (rows past
      // the block repeat its last row; their affinities are never stored)
      qs = (__bf16*)dyn;
      constexpr int CPR = D / 8;
      constexpr int NST = (RPW * CPR + kSelThreads - 1) / kSelThreads;
      bf16x8 st[NST];
#pragma unroll
      for (int u = 0; u < NST; ++u) {
        const int i = min(tid + u * kSelThreads, RPW * CPR - 1);
        const int row = i / CPR, c = i - row * CPR;
        const int tok = qb.start + min(r0 + row, qb.len - 1);
        st[u] = *(const bf16x8*)((const __bf16*)sc.q +
                                 ((size_t)tok * pl.hq + h) * D + 8 * c);
      }
#pragma unroll
      for (int u = 0; u < NST; ++u) {
        const int i = tid + u * kSelThreads;
        if (i < RPW * CPR) {
          const int row = i / CPR, c = i - row * CPR;
          *(bf16x8*)(qs + row * (D + 8) + 8 * c) = st[u];
        }
      }
      __syncthreads();
    }
    affinity_tiles<F32, D>(pl, ws.kbar, sc.q, sc.scale_log2, qb, h, kvh, first,
                           nh, TPR * L, r0, RPW, rg, ph, WPG, ev, stride, lane,
                           qs);
    __syncthreads();

    // ---- retention of each row (TPR lanes per row) ----
    {
      const int rr = tid / TPR, part = tid % TPR;
      const int row = r0 + rr;
      if (row < qb.len) {                         // uniform over the group
        const int j0 = part * L;
        const int cnt = max(0, min(L, nh - j0));  // real entries
        float* const my = ev + rr * stride + j0;
        uint32_t* const wrow = wb + row * W;
        if (L <= RV)
          retain_row_regs<TPR, RV>(my, L, nh, j0, sc.tau, lane, part, wrow);
        else
          retain_row_lds<TPR>(my, L, cnt, nh, j0, sc.tau, lane, part, wrow);
      }
    }
    __syncthreads();
  }

  // ---- per-row bits [W][64] and the union over the block's rows ----
  for (int i = tid; i < 64 * W; i += kSelThreads) {
    const int w = i >> 6, r = i & 63;
    rb[i] = wb[r * W + w];
  }
  for (int w = tid; w < W; w += kSelThreads) {
    unsigned u = 0u;
    for (int r = 0; r < 64; ++r) u |= wb[r * W + w];
    ub[w] = u;
  }
}

// ---------------------------------------------------------------------------
// Coarse query-frame evidence (appendix, coarse-map equation): for a query
// token i, the tokens of each retained history block j share the block
// affinity g_ij, the tokens of E_i (the video's system prefix and the causal
// prefix of i's own block) keep their exact logits, and the row is
// normalised. A retained block therefore carries the mass
// len_j 2^(g_ij - M) / Z with Z = sum_{m in E_i} 2^(s_im - M) +
// sum_{j in S_i} len_j 2^(g_ij - M) (log2 units). coarse_kernel takes one
// query-token block, one head and one pass of 16 rows; the 16 lanes of a
// row walk its history share. The per-block masses of the pass's rows are
// summed in row order into cpart; coarse_reduce_kernel adds a video's
// blocks and passes in order and spreads each block's mass evenly over its
// frames (frames never cross blocks).
constexpr int kCoarseTPR = 16;
constexpr int kCoarseRows = kSelThreads / kCoarseTPR;   // rows per pass
constexpr int kCoarsePasses = kTile64 / kCoarseRows;

__device__ __forceinline__ float pair_max_(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x),
                                            __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum_(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x),
                                            __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Log2 max and sum of row r0 + l32's exact logits over the E_i tiles e =
// ph, ph + 4, ... (system-prefix blocks, then the row's own block).
template <bool F32, int D>
__device__ __forceinline__ void exact_part(
    const DevPlan& pl, const SelCall& sc, const BlockDesc& qb, int qbid,
    int h, int kvh, int sys0, int nsys, int r0, int ph, int lane, float& mw,
    float& lw) {
  const int l32 = lane & 31, g = lane >> 5;
  const bool rv = l32 < kCoarseRows && r0 + l32 < qb.len;
  const int qtok = qb.start + r0 + l32;
  const size_t qoff = ((size_t)(rv ? qtok : qb.start) * pl.hq + h) * D;
  mw = -__builtin_inff();
  lw = 0.f;
  for (int e = ph; e <= nsys; e += 4) {
    const int kbid = e < nsys ? sys0 + e : qbid;
    const BlockDesc kb = pl.blocks[kbid];
    f32x16 s[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int key = min(32 * c + l32, kb.len - 1);
      const size_t koff = ((size_t)(kb.start + key) * pl.hkv + kvh) * D;
      if (!F32) {
        const __bf16* ks = (const __bf16*)sc.k + koff + 8 * g;
        const __bf16* qs = (const __bf16*)sc.q + qoff + 8 * g;
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk)
          s[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              *(const bf16x8*)(ks + 16 * kk), *(const bf16x8*)(qs + 16 * kk),
              s[c], 0, 0, 0);
      } else {
        const float* ks = (const float*)sc.k + koff + g * (D / 2);
        const float* qs = (const float*)sc.q + qoff + g * (D / 2);
#pragma unroll
        for (int u = 0; u < D / 2; ++u)
          s[c] = __builtin_amdgcn_mfma_f32_32x32x2f32(ks[u], qs[u], s[c], 0, 0,
                                                      0);
      }
    }
    float mt = -__builtin_inff();
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = 32 * c + 8 * (r >> 2) + 4 * g + (r & 3);
        const bool ok = rv && key < kb.len && kb.start + key <= qtok;
        s[c][r] = ok ? s[c][r] * sc.scale_log2 : -__builtin_inff();
        mt = fmaxf(mt, s[c][r]);
      }
    mt = pair_max_(mt);
    const float mn = fmaxf(mw, mt);
    if (mn == -__builtin_inff()) continue;
    float t = 0.f;
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) t += __builtin_amdgcn_exp2f(s[c][r] - mn);
    t = pair_sum_(t);
    lw = (mw == -__builtin_inff() ? 0.f : lw * __builtin_amdgcn_exp2f(mw - mn))
         + t;
    mw = mn;
  }
}

template <bool F32, int D>
__global__ __launch_bounds__(kSelThreads) void coarse_kernel(
    const DevPlan pl, const Workspace ws, const SelCall sc,
    float* __restrict__ cpart) {
  constexpr int TPR = kCoarseTPR, RPW = kCoarseRows;
  extern __shared__ __attribute__((aligned(16))) float dyn[];
  const int tile = blockIdx.x, h = blockIdx.y, pass = blockIdx.z;
  const TextTile tt = pl.tiles[tile];
  const int qbid = tt.qblock;
  const BlockDesc qb = pl.blocks[qbid];
  const int r0 = pass * RPW;
  const int nh = pl.blk_local[qbid];
  const int Wb = pl.W * 32;
  float* const dst = cpart + (((size_t)tile * kCoarsePasses + pass) * pl.hq +
                              h) * Wb;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  if (r0 >= qb.len || nh <= 0) {
    for (int j = tid; j < Wb; j += kSelThreads) dst[j] = 0.f;
    return;
  }
  const int L = sel_per_thread(nh, TPR), stride = sel_stride(nh, TPR);
  float* const ev = dyn;                      // [RPW][stride]
  float* const emx = dyn + RPW * stride;      // [4 waves][32 rows]
  float* const esm = emx + 4 * 32;
  const int kvh = h / (pl.hq / pl.hkv);
  const int first = qbid - nh;                // first visual block
  const SeqDesc sq = pl.seqs[tt.seq];
  const int nsys = (sq.vis0 - sq.tok0 + kTile64 - 1) / kTile64;
  affinity_tiles<F32, D>(pl, ws.kbar, sc.q, sc.scale_log2, qb, h, kvh, first,
                         nh, nh, r0, RPW, 0, wave, 4, ev, stride, lane);
  float mw, lw;
  exact_part<F32, D>(pl, sc, qb, qbid, h, kvh, first - nsys, nsys, r0, wave,
                     lane, mw, lw);
  if ((lane >> 5) == 0) {
    emx[wave * 32 + lane] = mw;
    esm[wave * 32 + lane] = lw;
  }
  __syncthreads();
  const int rr = tid / TPR, part = tid % TPR;
  const int row = r0 + rr;
  if (row < qb.len) {                         // uniform over the group
    float mE = -__builtin_inff(), lE = 0.f;   // waves' parts, in order
    for (int w = 0; w < 4; ++w) {
      const float m = emx[w * 32 + rr], l = esm[w * 32 + rr];
      if (m == -__builtin_inff()) continue;
      const float mn = fmaxf(mE, m);
      lE = (mE == -__builtin_inff() ? 0.f
                                    : lE * __builtin_amdgcn_exp2f(mE - mn)) +
           l * __builtin_amdgcn_exp2f(m - mn);
      mE = mn;
    }
    const uint32_t* rbw =
        ws.rbits + ((size_t)h * pl.nb + qbid) * pl.W * 64 + row;
    const int j0 = part * L;
    const int cnt = max(0, min(L, nh - j0));
    float* const my = ev + rr * stride + j0;
    float mx = -__builtin_inff();
    for (int i = 0; i < cnt; ++i) {
      const int j = j0 + i;
      const bool kept = (rbw[(size_t)(j >> 5) * 64] >> (j & 31)) & 1u;
      const float a = kept ? my[i] + __builtin_amdgcn_logf(
                                         (float)pl.blocks[first + j].len)
                           : -__builtin_inff();
      my[i] = a;
      mx = fmaxf(mx, a);
    }
    const float M = fmaxf(grp_max<TPR>(mx), mE);
    float z = 0.f;
    for (int i = 0; i < cnt; ++i) {
      const float w = __builtin_amdgcn_exp2f(my[i] - M);
      my[i] = w;
      z += w;
    }
    z = grp_sum<TPR>(z) + lE * __builtin_amdgcn_exp2f(mE - M);
    const float inv = 1.f / z;
    for (int i = 0; i < cnt; ++i) my[i] *= inv;
  }
  __syncthreads();
  for (int j = tid; j < Wb; j += kSelThreads) {
    float t = 0.f;
    if (j < nh)
      for (int r = 0; r < RPW && r0 + r < qb.len; ++r) t += ev[r * stride + j];
    dst[j] = t;
  }
}

// out[h][f] = sum over the video's query blocks and passes (in order) of
// the mass of f's block, times the share of the block's tokens in frame f.
__global__ __launch_bounds__(256) void coarse_reduce_kernel(
    const DevPlan pl, const float* __restrict__ cpart,
    float* __restrict__ out) {
  const int f = blockIdx.x * 256 + threadIdx.x, h = blockIdx.y;
  if (f >= pl.T) return;
  const SeqDesc sq = pl.seqs[pl.frame_seq[f]];
  const int Wb = pl.W * 32;
  float t = 0.f;
  if (sq.n_tiles > 0) {
    const int qb0 = pl.tiles[sq.tile0].qblock;
    const int first = qb0 - pl.blk_local[qb0];
    const int j = (int)(((int64_t)(f - sq.frame0) * pl.Nv) / kTile64);
    for (int ti = sq.tile0; ti < sq.tile0 + sq.n_tiles; ++ti)
      for (int ps = 0; ps < kCoarsePasses; ++ps)
        t += cpart[(((size_t)ti * kCoarsePasses + ps) * pl.hq + h) * Wb + j];
    t *= (float)pl.Nv / (float)pl.blocks[first + j].len;
  }
  out[(size_t)h * pl.T + f] = t;
}

__global__ void seg_fill_kernel(float* __restrict__ p, size_t n) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += stride)
    p[i] = neg_inf();
}

template <bool F32, int D, int TPR, int RV = kRegVals>
hipError_t launch_sel(const DevPlan& p, const Workspace& w, const SelCall& c,
                      size_t lds, hipStream_t s) {
  auto* fn = select_kernel<F32, D, TPR, RV>;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute(
        (const void*)fn, hipFuncAttributeMaxDynamicSharedMemorySize,
        (int)lds);
    if (e != hipSuccess) return e;
  }
  fn<<<dim3(p.nb * p.hq), dim3(kSelThreads), lds, s>>>(p, w, c);
  return hipGetLastError();
}

template <bool F32, int D>
hipError_t launch_sel_d(const DevPlan& p, const Workspace& w,
                        const SelCall& c, int nh_max, hipStream_t s) {
  // fewest lanes per row whose share of the longest history fits in
  // registers (and whose LDS lets two work-groups share a CU); else 16 lanes
  // per row with the long register form; else the LDS-streaming variant
  // with the widest rows that fit
  const int tprs[3] = {4, 8, 16};
  int pick = -1;
  for (int i = 0; i < 3 && pick < 0; ++i)
    if (sel_per_thread(nh_max, tprs[i]) <= kRegVals &&
        sel_lds_bytes(nh_max, tprs[i], p.W, D) <= kSelLdsTwoPerCu)
      pick = i;
  if (pick < 0 && sel_per_thread(nh_max, 16) <= kRegValsLong &&
      sel_lds_bytes(nh_max, 16, p.W, D) <= kSelLdsTwoPerCu)
    return launch_sel<F32, D, 16, kRegValsLong>(
        p, w, c, sel_lds_bytes(nh_max, 16, p.W, D), s);
  for (int i = 0; i < 3 && pick < 0; ++i)
    if (sel_lds_bytes(nh_max, tprs[i], p.W, D) <= kSelLdsTwoPerCu) pick = i;
  for (int i = 0; i < 3 && pick < 0; ++i)
    if (sel_lds_bytes(nh_max, tprs[i], p.W, D) <= kSelLdsMax) pick = i;
  if (pick < 0) return hipErrorInvalidValue;
  const size_t lds = sel_lds_bytes(nh_max, tprs[pick], p.W, D);
  if (pick == 0) return launch_sel<F32, D, 4>(p, w, c, lds, s);
  if (pick == 1) return launch_sel<F32, D, 8>(p, w, c, lds, s);
  return launch_sel<F32, D, 16>(p, w, c, lds, s);
}

}  // namespace

size_t select_lds_need(int nh_max, int W) {
  return sel_lds_bytes(nh_max, 16, W, 128);
}

hipError_t launch_select(const DevPlan& p, const Workspace& w,
                         const SelCall& c, hipStream_t s) {
  if (c.fp32) {
    if (c.d == 64)
      pool_kernel<true, 64><<<dim3(p.nb, p.hkv), dim3(64), 0, s>>>(p, c.k,
                                                                   w.kbar);
    else
      pool_kernel<true, 128><<<dim3(p.nb, p.hkv), dim3(128), 0, s>>>(p, c.k,
                                                                     w.kbar);
  } else {
    if (c.d == 64)
      pool_kernel<false, 64><<<dim3(p.nb, p.hkv), dim3(64), 0, s>>>(p, c.k,
                                                                    w.kbar);
    else
      pool_kernel<false, 128><<<dim3(p.nb, p.hkv), dim3(128), 0, s>>>(
          p, c.k, w.kbar);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int nh_max = std::max(p.hmax, 1);
  if (c.fp32)
    return c.d == 64 ? launch_sel_d<true, 64>(p, w, c, nh_max, s)
                     : launch_sel_d<true, 128>(p, w, c, nh_max, s);
  return c.d == 64 ? launch_sel_d<false, 64>(p, w, c, nh_max, s)
                   : launch_sel_d<false, 128>(p, w, c, nh_max, s);
}

size_t coarse_part_floats(int n_tiles, int hq, int W) {
  return (size_t)n_tiles * kCoarsePasses * hq * W * 32;
}

hipError_t launch_coarse(const DevPlan& p, const Workspace& w,
                         const SelCall& c, float* cpart, float* out,
                         hipStream_t s) {
  if (p.n_tiles > 0) {
    const int nh_max = std::max(p.hmax, 1);
    const size_t lds = (size_t)kCoarseRows *
                           sel_stride(nh_max, kCoarseTPR) * 4 + 2 * 4 * 32 * 4;
    dim3 grid(p.n_tiles, p.hq, kCoarsePasses), block(kSelThreads);
    auto go = [&](auto fn) -> hipError_t {
      if (lds > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute(
            (const void*)fn, hipFuncAttributeMaxDynamicSharedMemorySize,
            (int)lds);
        if (e != hipSuccess) return e;
      }
      fn<<<grid, block, lds, s>>>(p, w, c, cpart);
      return hipGetLastError();
    };
    hipError_t e;
    if (c.fp32)
      e = c.d == 64 ? go(coarse_kernel<true, 64>) : go(coarse_kernel<true, 128>);
    else
      e = c.d == 64 ? go(coarse_kernel<false, 64>)
                    : go(coarse_kernel<false, 128>);
    if (e != hipSuccess) return e;
  }
  coarse_reduce_kernel<<<dim3((p.T + 255) / 256, p.hq), dim3(256), 0, s>>>(
      p, cpart, out);
  return hipGetLastError();
}

hipError_t launch_seg_fill(const DevPlan& p, const Workspace& w,
                           hipStream_t s) {
  const size_t n = (size_t)p.hq * p.segtot;
  if (n == 0) return hipSuccess;
  const int blocks = (int)std::min<size_t>((n + 255) / 256, 4096);
  seg_fill_kernel<<<dim3(blocks), dim3(256), 0, s>>>(w.seg, n);
  return hipGetLastError();
}

}  // namespace evisel
