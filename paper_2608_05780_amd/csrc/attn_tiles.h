// Tile machinery shared by the attention kernels (attn.hip, attn_pipe.hip):
// LDS swizzles, the direct global -> LDS tile loader and the bf16 / fp32
// MFMA operand paths of one 64-key tile.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

#define EV_LDS __attribute__((address_space(3)))

namespace evisel {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kTile = 64;
constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr float kLn2 = 0.69314718055994530942f;
constexpr float kRescaleSlack = 8.0f;  // log2 units
// Probabilities taken against a stale reference may reach 2^kFastSlack
// before the reference is moved (fp32 accumulators and the bf16 P keep
// their relative precision at any such scale).
constexpr float kFastSlack = 64.0f;
constexpr float kFastBound = 18446744073709551616.0f;   // 2^kFastSlack

__device__ __forceinline__ float neg_inf() { return -__builtin_inff(); }
__device__ __forceinline__ float exp2_(float x) {
  return __builtin_amdgcn_exp2f(x);
}
__device__ __forceinline__ float log2_(float x) {
  return __builtin_amdgcn_logf(x);
}
// v_permlane32_swap(x, x) returns (x[lane], x[lane ^ 32]) in some order on
// every lane, so the pair's sum and max need no LDS round trip.
__device__ __forceinline__ float pair_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x),
                                            __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float pair_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x),
                                            __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// 16-byte chunk swizzles of a 64-row LDS tile: physical chunk = logical
// chunk ^ swz(row), RC chunks per row. They keep the operand reads free of
// bank conflicts whether the LDS serves 128 or 256 bytes per pass:
//   K (ds_read_b128, lane = key): 16 consecutive keys hit 16 distinct
//     chunk positions (8 when a row has only 8 chunks);
//   V (ds_read_b64_tr_b16): the 4 rows a 16-lane group addresses take the
//     XOR masks 0, 6, 10, 12, whose bits 1-2 and bits 2-3 are both distinct,
//     so 2-chunk (128 B) and 4-chunk (256 B) row slices never collide.
enum Swz { kSwzK = 0, kSwzV = 1, kSwzNone = 2 };
template <int SWZ, int RC>
__device__ __forceinline__ int swz(int row) {
  if (SWZ == kSwzK) return row & (RC >= 16 ? 15 : 7);
  if (SWZ == kSwzV) return ((0xCA60 >> (4 * (row & 3))) & 15) & (RC - 1);
  return 0;
}

// One 16-byte-per-lane global -> LDS load: lane l's 16 bytes from
// gbase + voff land at LDS byte address lds + 16 l. Issued as inline
// assembly so that the compiler does not treat later LDS reads as possibly
// racing with it (it would otherwise wait for every outstanding load,
// including the next tile's, before the transposed V reads); every caller
// waits for vmcnt(0) and a barrier before reading the destination. The LDS
// address is an input operand bound to m0 (the register the instruction
// takes it from), so the compiler writes m0 itself and knows it holds that
// value; it passes through readfirstlane because it is wave-uniform and m0
// is a scalar register. The s_nop 4 gives the instruction five wait states
// after whatever precedes it: a vector-memory instruction that reads an SGPR
// written by a VALU instruction (v_readlane_b32, which the compiler uses to
// restore spilled SGPRs such as gbase) needs five, and the compiler inserts
// them only for memory instructions it knows about, not for inline assembly.
// The same nop covers the one wait state between the m0 write and its use.
__device__ __forceinline__ void lds_dma16(uint32_t lds, const char* gbase,
                                          uint32_t voff) {
  asm volatile("s_nop 4\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(gbase),
                 "{m0}"(__builtin_amdgcn_readfirstlane(lds))
               : "memory");
}

// Loads of one 64-key tile of a [S][H][D] tensor into LDS: every thread
// fetches N = 64*RC/256 chunks of 16 bytes and a wavefront's load fills 64
// consecutive 16-byte LDS slots. The (row, chunk) a lane fetches is fixed,
// so its byte offset from the tile's first row is computed once; per tile
// the address is a wave-uniform base plus that offset. Rows past klen
// re-read row klen-1 (finite values; they get zero probability).
template <typename T, int D, int SWZ>
struct TileLoader {
  static constexpr int RC = D * (int)sizeof(T) / 16;
  static constexpr int N = kTile * RC / kThreads;
  static constexpr int RSTEP = 64 / RC;   // row step between loads i, i+1
  uint32_t off[N];    // byte offset of this lane's chunk for a full tile
  int row0;           // row of load 0 (load i fetches row row0 + i*RSTEP)
  uint32_t rowbytes;  // bytes between consecutive tokens (hkv * D * sizeof T)

  __device__ void init(int hkv, int wave, int lane) {
    rowbytes = (uint32_t)hkv * D * sizeof(T);
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int slot = (wave * N + i) * 64 + lane;
      const int r = slot / RC;
      const int ch = (slot % RC) ^ swz<SWZ, RC>(r);
      if (i == 0) row0 = r;
      off[i] = (uint32_t)r * rowbytes + (uint32_t)ch * 16;
    }
  }

  __device__ void issue(EV_LDS char* buf, const T* src, int kstart, int klen,
                        int kvh, int wave) const {
    const char* base =
        (const char*)src + ((size_t)kstart * rowbytes + (size_t)kvh * D *
                                                            sizeof(T));
    const uint32_t lds0 =
        (uint32_t)(uintptr_t)buf + (uint32_t)(wave * N * 1024);
    if (klen == kTile) {
#pragma unroll
      for (int i = 0; i < N; ++i) lds_dma16(lds0 + i * 1024, base, off[i]);
    } else {
#pragma unroll
      for (int i = 0; i < N; ++i) {
        const int r = row0 + i * RSTEP;
        const uint32_t over =
            r >= klen ? (uint32_t)(r - (klen - 1)) * rowbytes : 0u;
        lds_dma16(lds0 + i * 1024, base, off[i] - over);
      }
    }
  }
};

// ---------------------------------------------------------------------------
// bf16 operands.
template <int D>
struct Bf16Path {
  using T = __bf16;
  static constexpr int RC = D / 8;   // 16-byte chunks per row
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

  // S^T[key][q] for the two 32-key halves of the tile: lane (key, g) reads
  // logical chunk 2kk + g of K row key.
  __device__ static void qk(f32x16 (&s)[2], const EV_LDS char* kt,
                            const QFrag& qf, int l32, int g) {
    bf16x8 kf[D / 16][2];
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk)
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const int key = 32 * c + l32;
        const int ch = (2 * kk + g) ^ swz<kSwzK, RC>(key);
        kf[kk][c] = *(const EV_LDS bf16x8*)(kt + (key * RC + ch) * 16);
      }
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk)
#pragma unroll
      for (int c = 0; c < 2; ++c)
        s[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kk][c], qf.x[kk],
                                                        s[c], 0, 0, 0);
    // eight operand reads ahead, then two MFMAs per two further reads
    __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
#pragma unroll
    for (int i = 0; i < D / 16 - 4; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
  }

  // O^T[d][q] += V^T[d][key] P^T[key][q]. The B operand of k-step (c, s)
  // is the lane's own s[c][8s .. 8s+7], i.e. keys 32c + 16s + 8(e/4) +
  // 4g + e%4 for e = 0..7. The A operand for d-tile mt: two transpose reads
  // in which lane j of each 16-lane group addresses V row
  // 32c + 16s + 4g + j/4 (+8 for the second) at column
  // 32mt + 16((lane/16) % 2) + 4(j % 4); lane i then holds V[those 4 keys]
  // at column 32mt + lane % 32.
  // Per-lane part of the transpose-read address of d-tile mt: the lane's
  // row offset 4g + j/4 and its swizzled chunk. The chunk of d-tile mt is
  // (4mt + x) ^ sw with x < 4, i.e. (4mt ^ (sw & ~3)) | (x ^ (sw & 3)), so
  // the k-step part (32c + 16s rows) is a constant added to these.
  static constexpr int NMT = D / 32;
  struct PvOff {
    int v[NMT];
  };
  __device__ static void pv_offsets(PvOff& po, int lane) {
    const int j = lane & 15, q16 = lane >> 4, g = lane >> 5;
    const int sw = swz<kSwzV, RC>(j >> 2);   // row % 4 == j / 4 below
    const int x = 2 * (q16 & 1) + ((j & 3) >> 1);
#pragma unroll
    for (int mt = 0; mt < NMT; ++mt) {
      const int ch = ((4 * mt) ^ (sw & ~3)) | (x ^ (sw & 3));
      po.v[mt] = ((4 * g + (j >> 2)) * RC + ch) * 16 + 8 * (j & 1);
    }
  }
  __device__ static void pv(f32x16 (&o)[D / 32], const EV_LDS char* vt,
                            const f32x16 (&p)[2], const PvOff& po) {
    bf16x8 va[4][NMT];
    bf16x8 pb[4];
#pragma unroll
    for (int cs = 0; cs < 4; ++cs) {
      const int c = cs >> 1, s = cs & 1;
      const f32x8 pf = s == 0 ? __builtin_shufflevector(p[c], p[c], 0, 1, 2, 3,
                                                        4, 5, 6, 7)
                              : __builtin_shufflevector(p[c], p[c], 8, 9, 10,
                                                        11, 12, 13, 14, 15);
      pb[cs] = __builtin_convertvector(pf, bf16x8);
#pragma unroll
      for (int mt = 0; mt < NMT; ++mt) {
        const EV_LDS char* a0 = vt + po.v[mt] + (32 * c + 16 * s) * RC * 16;
        const EV_LDS char* a1 = a0 + 8 * RC * 16;   // row + 8
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (EV_LDS i16x4*)a0);
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (EV_LDS i16x4*)a1);
        const i16x4 lohi[2] = {lo, hi};
        va[cs][mt] = __builtin_bit_cast(bf16x8, lohi);
      }
    }
#pragma unroll
    for (int cs = 0; cs < 4; ++cs)
#pragma unroll
      for (int mt = 0; mt < NMT; ++mt)
        o[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[cs][mt], pb[cs],
                                                        o[mt], 0, 0, 0);
    // eight transpose reads (four operands) ahead, then one MFMA per two
    // further reads
    __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
#pragma unroll
    for (int i = 0; i < 4 * NMT - 4; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
  }

  __device__ static void store_o(void* out, int qpos, int h, int hq, int d0,
                                 f32x4 v) {
    bf16x4 b = __builtin_convertvector(v, bf16x4);
    *(bf16x4*)((__bf16*)out + ((size_t)qpos * hq + h) * D + d0) = b;
  }
  // Q and O move through LDS in the K-tile layout (rows of RC swizzled
  // 16-byte chunks), so that every global access is a whole row: 16 lanes
  // cover one row of one head. Q arrives by the same direct global -> LDS
  // loads as the key tiles.
  static constexpr bool kStaged = true;
  static constexpr int kPer = kTile * RC / kThreads;   // chunks per thread

  // The B operand of row `row` from a staged Q tile (as load_q).
  __device__ static void load_q_lds(QFrag& qf, const EV_LDS char* src,
                                    int row, int g) {
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      const int ch = (2 * kk + g) ^ swz<kSwzK, RC>(row);
      qf.x[kk] = *(const EV_LDS bf16x8*)(src + (row * RC + ch) * 16);
    }
  }
  // The lane's O^T values (times inv) of row `row` into a staged O tile:
  // o[mt][4 r4 .. 4 r4 + 3] are d = 32 mt + 8 r4 + 4 g .. + 3.
  __device__ static void o_to_lds(EV_LDS char* dst, const f32x16 (&o)[D / 32],
                                  float inv, int row, int g) {
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const f32x4 v = {o[mt][4 * r4] * inv, o[mt][4 * r4 + 1] * inv,
                         o[mt][4 * r4 + 2] * inv, o[mt][4 * r4 + 3] * inv};
        const int ch = (4 * mt + r4) ^ swz<kSwzK, RC>(row);
        *(EV_LDS bf16x4*)(dst + (row * RC + ch) * 16 + 8 * g) =
            __builtin_convertvector(v, bf16x4);
      }
  }
  // Rows [start, start+len) of head h from a staged O tile to out, as
  // non-temporal stores: O is not read again here, and streaming it keeps
  // the key/value tiles that other work-groups re-read in L2.
  __device__ static void o_from_lds(void* out, const EV_LDS char* src,
                                    int start, int len, int h, int hq,
                                    int tid) {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int slot = i * kThreads + tid, row = slot / RC, ch = slot % RC;
      if (row < len) {
        typedef int i32x4 __attribute__((ext_vector_type(4)));
        const i32x4 v = *(const EV_LDS i32x4*)(src + (row * RC +
                                                (ch ^ swz<kSwzK, RC>(row))) * 16);
        __builtin_nontemporal_store(
            v, (i32x4*)((__bf16*)out + ((size_t)(start + row) * hq + h) * D +
                        ch * 8));
      }
    }
  }
};

// ---------------------------------------------------------------------------
// fp32 operands (32x32x2 f32 MFMA). The contraction over d pairs element t
// of lane half g with d = g*D/2 + t, so every lane reads contiguous runs.
// V needs no transpose: each lane contributes one value per k-step.
template <int D>
struct F32Path {
  using T = float;
  static constexpr int RC = D / 4;
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
      for (int jj = 0; jj < 4; ++jj) qf.x[4 * u + jj] = t[jj];
    }
  }

  __device__ static void qk(f32x16 (&s)[2], const EV_LDS char* kt,
                            const QFrag& qf, int l32, int g) {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int key = 32 * c + l32;
#pragma unroll
      for (int u = 0; u < D / 8; ++u) {
        const int ch = (g * D / 8 + u) ^ swz<kSwzK, RC>(key);
        const f32x4 kf = *(const EV_LDS f32x4*)(kt + (key * RC + ch) * 16);
#pragma unroll
        for (int jj = 0; jj < 4; ++jj)
          s[c] = __builtin_amdgcn_mfma_f32_32x32x2f32(kf[jj], qf.x[4 * u + jj],
                                                      s[c], 0, 0, 0);
      }
    }
  }

  struct PvOff {
    int lane;
  };
  __device__ static void pv_offsets(PvOff& po, int lane) { po.lane = lane; }
  __device__ static void pv(f32x16 (&o)[D / 32], const EV_LDS char* vt,
                            const f32x16 (&p)[2], const PvOff& po) {
    const int lane = po.lane;
    const int l32 = lane & 31, g = lane >> 5;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = 32 * c + 8 * (r >> 2) + 4 * g + (r & 3);
#pragma unroll
        for (int mt = 0; mt < D / 32; ++mt)
          o[mt] = __builtin_amdgcn_mfma_f32_32x32x2f32(
              *(const EV_LDS float*)(vt + key * RC * 16 + (32 * mt + l32) * 4),
              p[c][r], o[mt], 0, 0, 0);
      }
    }
  }

  __device__ static void store_o(void* out, int qpos, int h, int hq, int d0,
                                 f32x4 v) {
    *(f32x4*)((float*)out + ((size_t)qpos * hq + h) * D + d0) = v;
  }
  static constexpr bool kStaged = false;
  __device__ static void load_q_lds(QFrag&, const EV_LDS char*, int, int) {}
  __device__ static void o_to_lds(EV_LDS char*, const f32x16 (&)[D / 32],
                                  float, int, int) {}
  __device__ static void o_from_lds(void*, const EV_LDS char*, int, int, int,
                                    int, int) {}
};


}  // namespace
}  // namespace evisel
