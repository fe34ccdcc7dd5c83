// Device helpers shared by the translation units of the gfx950 kernels
// (convolution forward and input gradient per storage type, weight
// gradient, pooling and row kernels): MFMA fragments, tile loaders, the
// instruction interleave of a K step, the XCD-aware tile order and the
// index arithmetic of band windows.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>

#include "kernels.hpp"

namespace lrcnn {

// Launch timing of the matrix-core kernels (test hook; kernels.hip):
// begin() registers a launch and returns its index (-1 when profiling is
// off); the launch carries the index's start and stop events.
namespace prof {
extern bool on;
// (bytes: the launch's algorithmic HBM bytes; es: storage element size,
// which selects the matrix-core peak of its roofline time)
int begin(const std::string &name, double flops, hipStream_t s, double bytes = 0.0,
          int es = 0);
hipEvent_t start(int i);
hipEvent_t stop(int i);
}  // namespace prof

// Launch of a kernel that may be profiled: with profiling on (pr >= 0) the
// start and stop events are attached to the dispatch itself
// (hipExtLaunchKernelGGL), so their interval is the kernel's execution
// and not the queue time around it; otherwise a plain launch.
template <typename F, typename... Args>
inline void launch_timed(F kernel, dim3 grid, hipStream_t s, int pr, Args... args) {
  if (pr >= 0)
    hipExtLaunchKernelGGL(kernel, grid, dim3(256), 0, s, prof::start(pr), prof::stop(pr), 0,
                          args...);
  else
    hipLaunchKernelGGL(kernel, grid, dim3(256), 0, s, args...);
}

// Convolution launchers, one translation unit per storage type and
// direction (conv_*.hip).
int launch_conv_f32_fwd(const ConvArgs &a, hipStream_t s);
int launch_conv_f32_dgrad(const ConvArgs &a, hipStream_t s);
int launch_conv_bf16_fwd(const ConvArgs &a, hipStream_t s);
int launch_conv_bf16_dgrad(const ConvArgs &a, hipStream_t s);

typedef uint16_t bf16;
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ float ldf(const float *p) { return *p; }
__device__ __forceinline__ float ldf(const bf16 *p) {
  return __uint_as_float((uint32_t)(*p) << 16);
}
// float32 -> bfloat16, round to nearest, ties to even (NaN stays NaN):
// the gfx950 conversion instruction (v_cvt_pk_bf16_f32), which gives the
// same bits as the integer rounding u + 0x7fff + ((u >> 16) & 1) for every
// non-NaN float32 input, denormals included (checked over all 2^32 bit
// patterns on the device).
__device__ __forceinline__ bf16 f2bf(float f) {
  return __builtin_bit_cast(bf16, (__bf16)f);
}
__device__ __forceinline__ void stf(float *p, float v) { *p = v; }
__device__ __forceinline__ void stf(bf16 *p, float v) { *p = f2bf(v); }

__device__ __forceinline__ int fdiv(int a, int b) {
  return a >= 0 ? a / b : -((-a + b - 1) / b);
}

// Tile geometry: a K tile row is KR 16-byte vectors (64 or 128 bytes) of one
// pixel or one weight row, staged in LDS with one extra vector of pitch.
#ifndef LRCNN_SWZ
#define LRCNN_SWZ 1
#endif
// forward convolution operands copied from global memory straight into LDS
#ifndef LRCNN_LDS_DMA
#define LRCNN_LDS_DMA 1
#endif
// input-gradient operands (stride 1, bfloat16) copied the same way
#ifndef LRCNN_DG_DMA
#define LRCNN_DG_DMA 1
#endif
// LDS stages of the direct-copy ring (3 or 4)
#ifndef LRCNN_DMA_ST
#define LRCNN_DMA_ST 3
#endif
template <typename T, int KR = 4>
struct Cfg {
  static constexpr int E = 16 / (int)sizeof(T);  // elements per 16 bytes
  static constexpr int BK = KR * E;               // K elements per tile row
  static constexpr int LDK = LRCNN_SWZ ? BK : BK + E;  // LDS pitch in elements
};
// Row-major LDS tiles with LRCNN_SWZ: no padding; the 16-byte vector v of
// row r is stored at slot v ^ ((r >> 2) & 3) (4 vectors per row), which
// keeps the 16-lane phases of 16-byte reads (16 consecutive rows, one
// vector) and writes (4 rows x 4 vectors) on distinct banks. With KR = 8
// vectors per row the slot is v ^ ((r >> 1) & 7): the 8 rows of one parity
// among 16 consecutive rows then take 8 distinct slots, and the two
// parities sit in the two 32-bank halves.
template <int KR>
__device__ __forceinline__ int swz(int row, int vec) {
  if (!LRCNN_SWZ) return vec;
  return KR == 8 ? (vec ^ ((row >> 1) & 7)) : (vec ^ ((row >> 2) & 3));
}

constexpr int BM = 128;

// k-major LDS tiles ([k][row], W elements per k row). float32: pitch W + 4
// (fragments read single words, a column of 32 rows per read). bfloat16:
// pitch W, no padding; the 64-byte chunk c of k row k is stored at chunk
// c ^ sw(k). A transposing fragment read (below) takes 64 bytes from each
// of four consecutive k rows in one 256-byte pass over the 64 banks; sw
// places those four on distinct 16-bank groups, for any W that is a
// multiple of 32 (bank group of chunk c of row k: (k W / 32 + c) mod 4).
// A 16-byte vector stays inside its chunk, and 16 consecutive vectors of a
// row (or of two rows when W = 64) still cover 64 distinct banks.
template <typename T, int W>
struct KM {
  static constexpr bool SW = sizeof(T) == 2;
  static constexpr int P = SW ? W : W + 4;  // pitch in elements
  static_assert(!SW || W % 32 == 0, "k-major bfloat16 tile width");
  __device__ static __forceinline__ int sw(int k) {
    constexpr int C = W / 32;
    return C >= 4 ? (k & 3) : C == 2 ? ((k >> 1) & 1) : 0;
  }
  __device__ static __forceinline__ int off(int k, int col) {
    return SW ? k * W + (col ^ (sw(k) << 5)) : k * P + col;
  }
};

// ------------------------------------------------------------------ MFMA
// Operand fragments of one 128 x BN tile step. Wave w owns rows
// [wm, wm+64) and columns [wn, wn+BN/2); lane l feeds row/column (l & 31) of
// each 32x32 block and the K slice [S*(l>>5), S*(l>>5)+S), S = BK/2, of the
// tile row. A and B use the same slice order, so every MFMA adds products of
// matching K indices; the order in which K is summed is the same for every
// output element and every band.
// AKM / BKM select the LDS layout of an operand: 0 = [row][k] (pitch
// LDK), fragments read as 16-byte vectors; 1 = [k][row] (layout KM),
// fragments read as 4-byte words (float32) or with transposing reads
// (bfloat16). k-major staging lets operands whose global layout is K-outer
// (the input gradient's weights, both weight-gradient operands) be stored
// with 16-byte writes.
// TA / TB: rows of the A tile and columns of the B tile in LDS (the row
// width of a k-major operand); NB = BN / 64 column blocks per wave.
template <typename T, int BN, int KR, int AKM = 0, int BKM = 0, int TA = BM, int TB = BN>
struct Frag;

template <int BN, int KR, int AKM, int BKM, int TA, int TB>
struct Frag<float, BN, KR, AKM, BKM, TA, TB> {
  static constexpr int LDK = Cfg<float, KR>::LDK, NB = BN / 64, NV = KR / 2;
  static constexpr int S = 4 * NV;            // K elements per lane group
  static constexpr int PA = KM<float, TA>::P, PB = KM<float, TB>::P;
  // instructions per tile step: MFMAs and LDS reads of one fragment load
  static constexpr int NMFMA = S * 2 * NB;
  static constexpr int NDSR = (AKM ? 2 * S : 2 * NV) + (BKM ? NB * S : NB * NV);
  float a[2][S], b[NB][S];
  __device__ __forceinline__ void load(const float *As, const float *Bs, int wm, int wn,
                                       int lane) {
    const int r = lane & 31, g = lane >> 5;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      if (AKM) {
#pragma unroll
        for (int s = 0; s < S; ++s) a[i][s] = As[(S * g + s) * PA + wm + 32 * i + r];
      } else {
        const int row = wm + 32 * i + r;
        const float4 *p = (const float4 *)(As + row * LDK);
#pragma unroll
        for (int q = 0; q < NV; ++q) {
          const float4 t = p[swz<KR>(row, NV * g + q)];
          a[i][4 * q] = t.x, a[i][4 * q + 1] = t.y, a[i][4 * q + 2] = t.z, a[i][4 * q + 3] = t.w;
        }
      }
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      if (BKM) {
#pragma unroll
        for (int s = 0; s < S; ++s) b[j][s] = Bs[(S * g + s) * PB + wn + 32 * j + r];
      } else {
        const int row = wn + 32 * j + r;
        const float4 *p = (const float4 *)(Bs + row * LDK);
#pragma unroll
        for (int q = 0; q < NV; ++q) {
          const float4 t = p[swz<KR>(row, NV * g + q)];
          b[j][4 * q] = t.x, b[j][4 * q + 1] = t.y, b[j][4 * q + 2] = t.z, b[j][4 * q + 3] = t.w;
        }
      }
    }
  }
  __device__ __forceinline__ void mma(f32x16 (&acc)[2][NB]) const {
#pragma unroll
    for (int s = 0; s < S; ++s)
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i][s], b[j][s], acc[i][j], 0, 0, 0);
  }
};

// bfloat16: one MFMA slice s (16 K values) gives lane half g = l >> 5 the
// K values 8*NV*g + 8*s + [0, 8) of row / column l & 31 of its 32x32 block
// (NV = KR / 2 slices per K tile row).
// [row][k] operands are read as one 16-byte vector per slice. k-major
// operands ([k][row], layout KM) are read with two transposing LDS
// reads (ds_read_b64_tr_b16): within each 16-lane group, lane i receives
// element i mod 4 of the 8-byte runs addressed by lanes 4*k' + i/4,
// k' = 0..3, so lane 16*G + 4*k' + q addresses K row
// 8*NV*(G >> 1) + 8*s + 4*t + k' at column 16*(G & 1) + 4*q (t = 0, 1 for
// the two reads), which hands every lane the same K values as the
// [row][k] read. Both layouts therefore sum K in the same order.
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
template <int W, int NV>
__device__ __forceinline__ bf16x8 ld_tr8(const bf16 *T, int base, int s, int lane) {
  const int G = lane >> 4, sl = lane & 15;
  const int k = 8 * NV * (G >> 1) + 8 * s + (sl >> 2);
  const int col = base + 16 * (G & 1) + 4 * (sl & 3);
  const bf16 *p0 = T + KM<bf16, W>::off(k, col), *p1 = T + KM<bf16, W>::off(k + 4, col);
  const bf16x4 r0 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
      (lds_bf16x4 *)((__attribute__((address_space(3))) char *)(char *)p0));
  const bf16x4 r1 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
      (lds_bf16x4 *)((__attribute__((address_space(3))) char *)(char *)p1));
  return __builtin_shufflevector(r0, r1, 0, 1, 2, 3, 4, 5, 6, 7);
}

template <int BN, int KR, int AKM, int BKM, int TA, int TB>
struct Frag<bf16, BN, KR, AKM, BKM, TA, TB> {
  static constexpr int LDK = Cfg<bf16, KR>::LDK, NB = BN / 64, NV = KR / 2;
  static constexpr int NMFMA = NV * 2 * NB;
  static constexpr int NDSR = (AKM ? 4 * NV : 2 * NV) + (BKM ? 2 * NB * NV : NB * NV);
  bf16x8 a[2][NV], b[NB][NV];
  __device__ __forceinline__ void load(const bf16 *As, const bf16 *Bs, int wm, int wn,
                                       int lane) {
    const int r = lane & 31, g = lane >> 5;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      if (AKM) {
#pragma unroll
        for (int q = 0; q < NV; ++q) a[i][q] = ld_tr8<TA, NV>(As, wm + 32 * i, q, lane);
      } else {
        const int row = wm + 32 * i + r;
        const bf16x8 *p = (const bf16x8 *)(As + row * LDK);
#pragma unroll
        for (int q = 0; q < NV; ++q) a[i][q] = p[swz<KR>(row, NV * g + q)];
      }
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      if (BKM) {
#pragma unroll
        for (int q = 0; q < NV; ++q) b[j][q] = ld_tr8<TB, NV>(Bs, wn + 32 * j, q, lane);
      } else {
        const int row = wn + 32 * j + r;
        const bf16x8 *p = (const bf16x8 *)(Bs + row * LDK);
#pragma unroll
        for (int q = 0; q < NV; ++q) b[j][q] = p[swz<KR>(row, NV * g + q)];
      }
    }
  }
  __device__ __forceinline__ void mma(f32x16 (&acc)[2][NB]) const {
#pragma unroll
    for (int s = 0; s < NV; ++s)
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i][s], b[j][s], acc[i][j],
                                                              0, 0, 0);
  }
};


// Row of the 32x32 accumulator block held in register v of lane l.
__device__ __forceinline__ int acc_row(int v, int lane) {
  return 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
}

// Load E consecutive elements (16 bytes) or zeros; `lim` = elements of the
// vector that exist (scalar path for channel counts not a multiple of E).
template <typename T, bool VEC>
__device__ __forceinline__ uint4 load16(const T *p, bool ok, int lim) {
  if (VEC) {
    return ok ? *(const uint4 *)p : make_uint4(0, 0, 0, 0);
  } else {
    union {
      uint4 u;
      T e[Cfg<T>::E];
    } r;
    r.u = make_uint4(0, 0, 0, 0);
    if (ok) {
#pragma unroll
      for (int e = 0; e < Cfg<T>::E; ++e)
        if (e < lim) r.e[e] = p[e];
    }
    return r.u;
  }
}

// Branch-free 16-byte load: an element outside the operand reads a
// 16-byte block of zeros instead, so the loads of a tile step stay in one
// basic block and can be scheduled among the MFMAs. The block is a mutable
// global that nothing writes, so the compiler cannot fold its value and
// turn the load back into a conditional one.
static __device__ __align__(16) uint4 g_zero16[1] = {};
__device__ __forceinline__ uint4 load16z(const void *base, long long off_bytes, bool ok) {
  const uint4 *q = ok ? (const uint4 *)((const char *)base + off_bytes) : &g_zero16[0];
  return *q;
}
// 16 bytes at p (or, if !ok, the zero block at `zero`, whose address the
// caller holds in registers) copied from global memory straight into LDS
// (global_load_lds_dwordx4): lane l of the wave writes bytes
// [16 l, 16 l + 16) after the wave-uniform LDS byte address `lds` (in M0).
// The copy is counted by vmcnt like any global load; no registers hold the
// data. It is issued as inline assembly so that the compiler does not
// track it: its waitcnt pass cannot tell one LDS stage from another and
// would wait for every copy before each LDS read. The caller orders the
// copies with explicit vmcnt waits and barriers; the "memory" clobber keeps
// the compiler from moving LDS accesses across it.
__device__ __forceinline__ void load16_lds_a(const void *p, bool ok, uint32_t lds,
                                             const void *zero) {
  const void *q = ok ? p : zero;
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off"
               :
               : "s"(__builtin_amdgcn_readfirstlane(lds)), "v"(q)
               : "memory", "m0");
}
// 16 bytes at p if ok, else the zero block at `zero`, read as a global
// memory load (the selected pointer is generic to the compiler)
__device__ __forceinline__ uint4 load16_sel(const void *p, bool ok, const void *zero) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(1))) const u32x4 g_u32x4;
  const u32x4 v = *(g_u32x4 *)(ok ? p : zero);
  return make_uint4(v.x, v.y, v.z, v.w);
}
// s_waitcnt with only the vector-memory counter limited to N (gfx9
// encoding: vmcnt in bits 3:0 and 15:14; expcnt and lgkmcnt at their
// maxima, i.e. not waited for).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Instruction schedule of one steady-state tile step: the MFMAs of the
// current fragments are interleaved with the LDS reads of the next
// fragments, the LDS writes of tile t+2 and the global loads (with their
// address arithmetic) of tile t+3, so the matrix pipe is not left idle
// while the wave issues memory work.
template <int NMF, int DSR, int DSW, int VMR>
__device__ __forceinline__ void interleave_step() {
  constexpr int Q = NMF / 4 > 0 ? NMF / 4 : 1;
  constexpr int R1 = (DSR + Q - 1) / Q, W1 = (DSW + Q - 1) / Q, V1 = (VMR + Q - 1) / Q;
#pragma unroll
  for (int i = 0; i < Q; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, R1, 0);  // LDS read
  }
#pragma unroll
  for (int i = 0; i < Q; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x200, W1, 0);  // LDS write
  }
#pragma unroll
  for (int i = 0; i < Q; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, 8, 0);   // VALU
    __builtin_amdgcn_sched_group_barrier(0x020, V1, 0);  // global load
  }
#pragma unroll
  for (int i = 0; i < NMF - 3 * Q; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
  }
}

// XCD-aware tile order. Workgroups are dispatched to the 8 XCDs round-robin
// (workgroup w runs on XCD w mod 8), and each XCD has its own L2. The
// workgroup's linear id is remapped so that every XCD receives one
// contiguous run of the tile order, in which neighbouring tiles share
// operand rows; without it each XCD would fetch nearly all of both
// operands into its L2.
struct TileId {
  int x, y, z;
};
__device__ __forceinline__ TileId xcd_tile(bool y_fastest) {
  const int gx = gridDim.x, gy = gridDim.y;
  const int total = gx * gy * gridDim.z;
  const int w = blockIdx.x + gx * (blockIdx.y + gy * blockIdx.z);
  const int q = total >> 3, r = total & 7, c = w & 7, k = w >> 3;
  const int id = c < r ? c * (q + 1) + k : r * (q + 1) + (c - r) * q + k;
  TileId t;
  if (y_fastest) {
    t.y = id % gy;
    const int rest = id / gy;
    t.x = rest % gx;
    t.z = rest / gx;
  } else {
    t.x = id % gx;
    const int rest = id / gx;
    t.y = rest % gy;
    t.z = rest / gy;
  }
  return t;
}

// ------------------------------------------------------- shared helpers
static unsigned grid_for(long long total) {
  long long g = (total + 255) / 256;
  if (g > 65536) g = 65536;
  return (unsigned)(g < 1 ? 1 : g);
}

__device__ __forceinline__ long long view_off(const View &v, int b, int row,
                                              int inner) {
  return b * v.bs + (long long)(row - v.row0) * v.W * v.C + inner;
}

__device__ __forceinline__ void ld4(const float *p, float (&v)[4]) {
  const float4 q = *(const float4 *)p;
  v[0] = q.x, v[1] = q.y, v[2] = q.z, v[3] = q.w;
}
__device__ __forceinline__ void ld4(const bf16 *p, float (&v)[4]) {
  const uint2 q = *(const uint2 *)p;
  v[0] = __uint_as_float(q.x << 16), v[1] = __uint_as_float(q.x & 0xffff0000u);
  v[2] = __uint_as_float(q.y << 16), v[3] = __uint_as_float(q.y & 0xffff0000u);
}
__device__ __forceinline__ void st4(float *p, const float (&v)[4]) {
  *(float4 *)p = make_float4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ void st4(bf16 *p, const float (&v)[4]) {
  uint2 q;
  q.x = (uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16);
  q.y = (uint32_t)f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16);
  *(uint2 *)p = q;
}
template <typename T, int V>
__device__ __forceinline__ void ldv(const T *p, float (&v)[4]) {
  if (V == 4) ld4(p, v);
  else v[0] = ldf(p);
}
template <typename T, int V>
__device__ __forceinline__ void stv(T *p, const float (&v)[4]) {
  if (V == 4) st4(p, v);
  else stf(p, v[0]);
}

// Decompose a flat index over B x rows x (W*C/V) into (b, row, inner):
// by multiply-shift division when every index fits in 32 bits, else by
// 64-bit division.
struct RowIter {
  long long inner, total;
  int R, r0;
  int fast;
  FastDiv fin, fr;
  __device__ __forceinline__ void at(long long idx, int V, int &b, int &y, int &in) const {
    if (fast) {
      uint32_t t, i, q, yy;
      fdiv_qr((uint32_t)idx, fin, t, i);
      fdiv_qr(t, fr, q, yy);
      in = (int)i * V;
      y = r0 + (int)yy;
      b = (int)q;
      return;
    }
    const long long i = idx % inner;
    const long long t = idx / inner;
    in = (int)(i * V);
    y = r0 + (int)(t % R);
    b = (int)(t / R);
  }
};
static RowIter row_iter(int B, int r0, int r1, int W, int C, int V) {
  RowIter it;
  it.inner = (long long)W * C / V;
  it.R = r1 - r0;
  it.r0 = r0;
  it.total = (long long)B * it.R * it.inner;
  it.fast = it.total < (1ll << 32) && it.R > 0 && it.inner > 0;
  if (it.fast) {
    it.fin = fast_div((uint32_t)it.inner);
    it.fr = fast_div((uint32_t)it.R);
  }
  return it;
}
#define GRID_STRIDE(idx, total)                                                   \
  for (long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x; idx < total; \
       idx += (long long)gridDim.x * blockDim.x)

// Base value an input-gradient element is added to: the error window's
// current value, or, when the launch initializes the window, the carried
// error (rows >= cinit_t) or zero. `inner` = x * C + c.
__device__ __forceinline__ const float *err_base(int init, const View &cinit, int cinit_t, int b,
                                                 int y, long long inner, const float *cur) {
  if (!init) return cur;
  if (cinit.p && y >= cinit_t)
    return (const float *)cinit.p + view_off(cinit, b, y, (int)inner);
  return nullptr;
}
__device__ __forceinline__ const float *dgrad_base(const ConvArgs &a, int b, int y,
                                                   long long inner, const float *cur) {
  return err_base(a.dst_init, a.cinit, a.cinit_t, b, y, inner, cur);
}

// Store V error values o of pixel (b, y, x), channels n.. of C, at d in
// the error window, or, when the launch completes the producer's error
// (eo.fact), as the producer's error operand (ReLU mask, affine scale,
// storage dtype; the same arithmetic as the activation backward) or its
// float32 carry to the previous band.
template <typename T, int V>
__device__ __forceinline__ void err_out(const ErrOut &eo, int C, int b, int y, int x, int n,
                                        float (&o)[4], float *d) {
  if (!eo.fact) {
    stv<float, V>(d, o);
    return;
  }
  const int inner = x * C + n;
  if (y < eo.fa) {
    stv<float, V>((float *)eo.carry.p + view_off(eo.carry, b, y, inner), o);
    return;
  }
  if (eo.relu) {
    float zz[4];
    ldv<T, V>((const T *)eo.z.p + view_off(eo.z, b, y, inner), zz);
#pragma unroll
    for (int e = 0; e < V; ++e)
      if (!(zz[e] > 0.f)) o[e] = 0.f;
  }
  if (eo.scale) {
#pragma unroll
    for (int e = 0; e < V; ++e) o[e] *= eo.scale[n + e];
  }
  stv<T, V>((T *)eo.dc.p + view_off(eo.dc, b, y, inner), o);
}
template <typename T, int V>
__device__ __forceinline__ void dgrad_out(const ConvArgs &a, int b, int y, int x, int n,
                                          float (&o)[4], float *d) {
  err_out<T, V>(a.eo, a.N, b, y, x, n, o, d);
}

}  // namespace lrcnn
