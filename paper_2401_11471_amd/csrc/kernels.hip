// gfx950 (CDNA4) kernels for row-centric CNN training.
//
// Convolutions run as implicit GEMMs on the matrix cores:
//   forward      (Eq. (1)):  M = B*rows*W_out pixels, N = C_out,
//                            K = kh*kw*C_in (tap-major, channel-minor)
//   input grad   (Get_error of Algorithm 1): the same kernel in gather form,
//                            M = producer pixels, N = C_in, K = kh*kw*C_out
//   weight grad  (g^l += Gradient, Eq. (2)): M = C_out, N = kh*kw*C_in,
//                            K = B*rows*W_out pixels, split over workgroups
//                            with a fixed-order reduction (deterministic)
// Operands are NHWC, so one 64-byte K slice of a pixel or a weight row is
// contiguous: tiles are fetched with 16-byte loads and staged in LDS as
// [row][k] with an 80-byte pitch; every lane then reads its K slice with
// 16-byte LDS reads. float32 uses v_mfma_f32_32x32x2_f32, bfloat16 uses
// v_mfma_f32_32x32x16_bf16 with float32 accumulation. A K loop runs over
// (tap, 64-byte channel chunk); rows of a band's window outside the image
// read as zero (semi-closed padding), rows inside are real data.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <map>
#include <string>
#include <vector>

#include "kernels.hpp"

namespace lrcnn {

// ------------------------------------------------------------- profiling
// Optional per-launch timing of the matrix-core kernels: two events on the
// launch stream around each launch, aggregated per kernel instantiation
// together with the launch's algorithmic FLOPs (what the convolution needs,
// not what the tiles compute).
namespace prof {
struct Rec {
  std::string name;
  hipEvent_t a, b;
  double flops;
};
static bool on = false;
static std::vector<Rec> recs;
static std::vector<hipEvent_t> pool;
static size_t used = 0;

static hipEvent_t take() {
  if (used == pool.size()) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    pool.push_back(e);
  }
  return pool[used++];
}
static int begin(const std::string &name, double flops, hipStream_t s) {
  if (!on) return -1;
  hipEvent_t a = take(), b = take();
  if (!a || !b) return -1;
  hipEventRecord(a, s);
  recs.push_back(Rec{name, a, b, flops});
  return (int)recs.size() - 1;
}
static void end(int i, hipStream_t s) {
  if (i >= 0) hipEventRecord(recs[i].b, s);
}
struct Agg {
  int64_t launches = 0;
  double ms = 0, flops = 0;
};
static std::vector<std::pair<std::string, Agg>> table;
}  // namespace prof

void profile_enable(int enable) {
  prof::on = enable != 0;
  if (prof::on) {
    prof::recs.clear();
    prof::used = 0;
    prof::table.clear();
  }
}

// Aggregate the recorded launches (the caller has synchronised the streams).
int profile_collect() {
  std::map<std::string, prof::Agg> m;
  for (auto &r : prof::recs) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) return -1;
    auto &g = m[r.name];
    g.launches += 1;
    g.ms += ms;
    g.flops += r.flops;
  }
  prof::table.assign(m.begin(), m.end());
  return (int)prof::table.size();
}

int profile_entry(int i, const char **name, int64_t *launches, double *ms, double *flops) {
  if (i < 0 || i >= (int)prof::table.size()) return -1;
  *name = prof::table[i].first.c_str();
  *launches = prof::table[i].second.launches;
  *ms = prof::table[i].second.ms;
  *flops = prof::table[i].second.flops;
  return 0;
}

typedef uint16_t bf16;
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ float ldf(const float *p) { return *p; }
__device__ __forceinline__ float ldf(const bf16 *p) {
  return __uint_as_float((uint32_t)(*p) << 16);
}
// float32 -> bfloat16, round to nearest, ties to even (NaN kept quiet).
__device__ __forceinline__ bf16 f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu))
    return (bf16)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16)(u >> 16);
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
// row r is stored at slot v ^ ((r >> 2) & 3), which keeps the 16-lane
// phases of 16-byte reads (16 consecutive rows, one vector) and writes (4
// rows x 4 vectors) on distinct banks. Needs 4 vectors per row.
__device__ __forceinline__ int swz(int row, int vec) {
  return LRCNN_SWZ ? (vec ^ ((row >> 2) & 3)) : vec;
}

constexpr int BM = 128;

// ------------------------------------------------------------------ MFMA
// Operand fragments of one 128 x BN tile step. Wave w owns rows
// [wm, wm+64) and columns [wn, wn+BN/2); lane l feeds row/column (l & 31) of
// each 32x32 block and the K slice [S*(l>>5), S*(l>>5)+S), S = BK/2, of the
// tile row. A and B use the same slice order, so every MFMA adds products of
// matching K indices; the order in which K is summed is the same for every
// output element and every band.
// AKM / BKM select the LDS layout of an operand: 0 = [row][k] (pitch
// LDK), fragments read as 16-byte vectors; 1 = [k][row] (pitch rows + 4),
// fragments read as 4-byte words. k-major staging lets operands whose global
// layout is K-outer (the input gradient's weights, both weight-gradient
// operands) be stored with 16-byte writes; it is used for float32, where
// one element feeds one MFMA.
// TA / TB: rows of the A tile and columns of the B tile in LDS (the pitch
// of a k-major operand); NB = BN / 64 column blocks per wave.
template <typename T, int BN, int KR, int AKM = 0, int BKM = 0, int TA = BM, int TB = BN>
struct Frag;

template <int BN, int KR, int AKM, int BKM, int TA, int TB>
struct Frag<float, BN, KR, AKM, BKM, TA, TB> {
  static constexpr int LDK = Cfg<float, KR>::LDK, NB = BN / 64, NV = KR / 2;
  static constexpr int S = 4 * NV;            // K elements per lane group
  static constexpr int PA = TA + 4, PB = TB + 4;
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
          const float4 t = p[swz(row, NV * g + q)];
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
          const float4 t = p[swz(row, NV * g + q)];
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
// K values 16*g + 8*s + [0, 8) of row / column l & 31 of its 32x32 block.
// [row][k] operands are read as one 16-byte vector per slice. k-major
// operands ([k][row], pitch rows + 8) are read with two transposing LDS
// reads (ds_read_b64_tr_b16): within each 16-lane group, lane i receives
// element i mod 4 of the 8-byte runs addressed by lanes 4*k' + i/4,
// k' = 0..3, so lane 16*G + 4*k' + q addresses K row
// 16*(G >> 1) + 8*s + 4*t + k' at column 16*(G & 1) + 4*q (t = 0, 1 for the
// two reads), which hands every lane the same K values as the [row][k]
// read. Both layouts therefore sum K in the same order.
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
__device__ __forceinline__ bf16x8 ld_tr8(const bf16 *T, int pitch, int base, int s, int lane) {
  const int G = lane >> 4, sl = lane & 15;
  const int k = 16 * (G >> 1) + 8 * s + (sl >> 2);
  const int col = base + 16 * (G & 1) + 4 * (sl & 3);
  const bf16 *p0 = T + k * pitch + col, *p1 = T + (k + 4) * pitch + col;
  const bf16x4 r0 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
      (lds_bf16x4 *)((__attribute__((address_space(3))) char *)(char *)p0));
  const bf16x4 r1 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
      (lds_bf16x4 *)((__attribute__((address_space(3))) char *)(char *)p1));
  return __builtin_shufflevector(r0, r1, 0, 1, 2, 3, 4, 5, 6, 7);
}

template <int BN, int KR, int AKM, int BKM, int TA, int TB>
struct Frag<bf16, BN, KR, AKM, BKM, TA, TB> {
  static constexpr int LDK = Cfg<bf16, KR>::LDK, NB = BN / 64, NV = KR / 2;
  static constexpr int PA = TA + 8, PB = TB + 8;
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
        for (int q = 0; q < NV; ++q) a[i][q] = ld_tr8(As, PA, wm + 32 * i, q, lane);
      } else {
        const int row = wm + 32 * i + r;
        const bf16x8 *p = (const bf16x8 *)(As + row * LDK);
#pragma unroll
        for (int q = 0; q < NV; ++q) a[i][q] = p[swz(row, NV * g + q)];
      }
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      if (BKM) {
#pragma unroll
        for (int q = 0; q < NV; ++q) b[j][q] = ld_tr8(Bs, PB, wn + 32 * j, q, lane);
      } else {
        const int row = wn + 32 * j + r;
        const bf16x8 *p = (const bf16x8 *)(Bs + row * LDK);
#pragma unroll
        for (int q = 0; q < NV; ++q) b[j][q] = p[swz(row, NV * g + q)];
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
__device__ __align__(16) uint4 g_zero16[1] = {};
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

// ------------------------------------------- conv forward / input grad
// ONE: a single tap (1x1 kernel, or a phase with one tap): each A row's
// validity and address are fixed for the launch, so a K step only adds the
// channel offset.
template <typename T, int BN, int KR, bool DGRAD, bool VEC, bool S1, bool ONE = false>
// bfloat16: three workgroups per CU (the register budget is set for it;
// the swizzled LDS tiles fit three); float32 keeps the registers of two
__global__ __launch_bounds__(256, sizeof(T) == 2 ? 3 : 2) void conv_gemm_kernel(ConvArgs a) {
  using CF = Cfg<T, KR>;
  constexpr int E = CF::E, BK = CF::BK, LDK = CF::LDK;
  constexpr int NB = BN / 64;
  constexpr int NA = KR / 2;             // A rows loaded per thread
  constexpr int NBL = BN * KR / 256;     // B vectors loaded per thread
  constexpr int RS = 256 / KR;           // row stride between a thread's loads
  // forward with 16-byte rows: both operands copied straight from global
  // memory into their LDS stage (no registers, no LDS writes by the wave).
  // The K vector of a thread's tile rows is then chosen so that its
  // swizzled LDS slot is lane & 3: each wave's rows fill 1 KiB of LDS in
  // lane order, the layout of a direct copy.
  constexpr bool LANE_SLOT = KR == 4 && LRCNN_SWZ;
  constexpr bool DMA = LRCNN_LDS_DMA && LANE_SLOT && !DGRAD && VEC;
  // LDS stages. Register staging: while tile t is multiplied, the
  // fragments of t+1 are read, tile t+2 is written and tile t+3 is fetched
  // from global memory. Direct copies: tiles t+2 .. t+ST-1 are in flight.
  constexpr int ST = DMA ? LRCNN_DMA_ST : 3;
  // input gradient: weights staged k-major (16-byte stores)
  constexpr int BKM = DGRAD ? 1 : 0;
  constexpr int PB = BN + E;
  constexpr int BSZ = BKM ? BK * PB : BN * LDK;
  // LDS: the operand ring during the K loop; the forward epilogue then
  // reuses it to stage the output tile ([BM][BN + E] in the storage dtype)
  constexpr int CP = BN + E;
  constexpr size_t RING = sizeof(T) * ST * ((size_t)BM * LDK + BSZ);
  // (input gradient: float32 tile [BM][BN + 4], added to the error window);
  // a tile larger than the ring is staged in two halves of 64 rows
  constexpr size_t CROW = DGRAD ? sizeof(float) * (BN + 4) : sizeof(T) * CP;
  constexpr int HR = CROW * BM > RING ? BM / 2 : BM;
  constexpr size_t CTILE = CROW * HR;
  __shared__ __align__(16) char smem[RING > CTILE ? RING : CTILE];
  T (*As)[BM * LDK] = reinterpret_cast<T (*)[BM * LDK]>(smem);
  T (*Bs)[BSZ] = reinterpret_cast<T (*)[BSZ]>(smem + sizeof(T) * ST * BM * LDK);
  // (wave index read from lane 0 so the compiler keeps it, and the LDS
  // addresses derived from it, in scalar registers)
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int R = a.y1 - a.y0;
  const int M = a.B * R * a.Wd;
  // pixel stride of a phase of a strided input gradient (else 1)
  const int ps = DGRAD && a.pst > 1 ? a.pst : 1;
  // output-channel tiles fastest: a run of consecutive pixel tiles per XCD
  const TileId tl = xcd_tile(true);
  const int m0 = tl.x * BM, n0 = tl.y * BN;
  const int taps = a.kh * a.kw;
  const int CB = (a.KC + BK - 1) / BK;
  const bool tpk = !VEC && !DGRAD && a.tpack;
  const int KT = tpk ? (taps + KR - 1) / KR : taps * CB;
  // K vector of this thread's tile rows: (l & 3) ^ ((l >> 4) & 3) for lane
  // l puts it in LDS slot l & 3 (the swizzle is an XOR with (row >> 2) & 3)
  const int kv = LANE_SLOT ? ((tid & 3) ^ ((tid >> 4) & 3)) : tid % KR;
  const int wrow = wave * (64 / KR);  // first tile row of this wave's pass
  const T *src = (const T *)a.src.p;
  const T *w = (const T *)a.w;
  const long long srow = (long long)a.src.W * a.src.C;

  // pixels of this thread's A rows
  int ay[NA], ax[NA];
  long long abase[NA];
  bool am[NA];
#pragma unroll
  for (int i = 0; i < NA; ++i) {
    int m = m0 + tid / KR + RS * i;
    am[i] = m < M;
    int mm = am[i] ? m : 0;
    uint32_t t, x, b, y;
    fdiv_qr((uint32_t)mm, a.fw, t, x);
    fdiv_qr(t, a.fr, b, y);
    ax[i] = a.px0 + ps * (int)x;
    ay[i] = a.y0 + ps * (int)y;
    abase[i] = (long long)b * a.src.bs - (long long)a.src.row0 * srow;
  }
  // source row / column of each A row before the tap offset, and its
  // address there: a K step then adds one uniform offset per tap and
  // channel block (input gradient: subtracts the tap)
  int by[NA], bx[NA];
  long long rbase[NA];
#pragma unroll
  for (int i = 0; i < NA; ++i) {
    // (a phase: consumer row (y + ph) / s - i for its i-th tap, exactly)
    by[i] = DGRAD ? (ps > 1 ? (ay[i] + a.ph) / ps : ay[i] + a.ph) : ay[i] * a.sh - a.ph;
    bx[i] = DGRAD ? (ps > 1 ? (ax[i] + a.pw) / ps : ax[i] + a.pw) : ax[i] * a.sw - a.pw;
    rbase[i] = abase[i] + (long long)by[i] * srow + (long long)bx[i] * a.src.C;
  }
  bool rowok[NA];
#pragma unroll
  for (int i = 0; i < NA; ++i)
    rowok[i] = ONE && am[i] & (bx[i] >= 0) & (by[i] >= a.sy0) & (by[i] < a.sy1) & (bx[i] < a.Ws);
  // Forward direct copies (the launcher sends only kernels of up to 64
  // taps here): the taps under which an A row reads inside the source
  // window, as bits tap = ti * kw + tj (rows ti in [sy0 - by, sy1 - by),
  // columns tj in [-bx, Ws - bx)), and the address of the row's first
  // element at tap 0; a K step then tests one bit and adds one uniform
  // offset.
  // (input gradient, stride 1 or a stride phase: the same test with the
  // taps mirrored, sy = by - ti and sx = bx - tj, operands staged through
  // registers)
  constexpr bool TMASK = DMA && !ONE;
  constexpr bool RMASK = DGRAD && S1 && VEC && !ONE;
  constexpr bool MASK = TMASK || RMASK;
  uint64_t tmask[MASK ? NA : 1];
  const char *rp[DMA || RMASK ? NA : 1];
  if (DMA || RMASK) {
#pragma unroll
    for (int i = 0; i < NA; ++i) rp[i] = (const char *)src + (rbase[i] + kv * E) * (long long)sizeof(T);
  }
  if (MASK) {
#pragma unroll
    for (int i = 0; i < NA; ++i)
      tmask[i] = am[i] ? tap_window_mask(by[i], bx[i], a.kh, a.kw, a.sy0, a.sy1, a.Ws, DGRAD)
                       : 0ull;
  }
  // B operand. Forward: B[k][n] = W[n][tap][k], contiguous along k, stored
  // as 16-byte rows. Input gradient: B[k][n] = W[k][tap][n] (k = output
  // channel of the consumer), contiguous along n, so each 16-byte load
  // holds E columns of one k and is written to LDS transposed.
  constexpr int BV = BN / E;           // 16-byte vectors per k (input grad)
  constexpr int BKS = 256 / BV;        // k rows per pass (input grad)
  int bn[NBL];
  bool bvld[NBL];
#pragma unroll
  for (int j = 0; j < NBL; ++j) {
    bn[j] = DGRAD ? n0 + (tid % BV) * E : n0 + tid / KR + RS * j;
    bvld[j] = bn[j] < a.N;
  }
  const int bk0 = tid / BV;
  // taps of the weight tensor (a phase reads a subset of the full kernel)
  const int wtaps = ps > 1 ? a.taps_full : taps;
  long long bbase[NBL];
#pragma unroll
  for (int j = 0; j < NBL; ++j)
    bbase[j] = DGRAD ? (long long)(bk0 + BKS * j) * wtaps * a.N + bn[j]
                     : (long long)bn[j] * taps * a.KC + kv * E;
  const char *wp[DMA || RMASK ? NBL : 1];
  if (DMA || RMASK) {
#pragma unroll
    for (int j = 0; j < NBL; ++j) wp[j] = (const char *)w + bbase[j] * (long long)sizeof(T);
  }
  // LDS byte addresses of the stages (uniform)
  const uint32_t lds_a = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)smem;
  constexpr uint32_t ASB = sizeof(T) * BM * LDK, BSB = sizeof(T) * BSZ;
  const uint32_t lds_b = lds_a + ST * ASB;

  // K iterations of this workgroup (split-K over the tile's z), walked as
  // (tap, channel block) without divisions in the loop
  const int kbeg = tl.z * a.kts;
  const int kend = min(KT, kbeg + a.kts);
  int tap = kbeg / CB, cbi = kbeg - (kbeg / CB) * CB;
  int ti = tap / a.kw, tj = tap - (tap / a.kw) * a.kw;
  int kpk = kbeg;  // tap-packed forward: current K iteration
  // tap-mask loaders: byte offsets of the current (tap, channel block) in
  // the source (+-(ti * row pitch + tj * C) + cb) and in the weights
  // (forward: tap * KC + cb along a weight row; input gradient: cb *
  // taps * N + wtap * N down a column, wtap the tap of the full kernel),
  // advanced by uniform deltas: next channel block, next tap, next kernel
  // row
  constexpr long long ES = sizeof(T);
  constexpr long long SG = DGRAD ? -1 : 1;
  long long ub = (SG * ((long long)ti * srow + (long long)tj * a.src.C) + cbi * BK) * ES;
  const long long d_step = BK * ES, d_tap = (SG * a.src.C - (long long)(CB - 1) * BK) * ES;
  const long long d_row =
      (SG * (srow - (long long)(a.kw - 1) * a.src.C) - (long long)(CB - 1) * BK) * ES;
  const long long wst = DGRAD ? (long long)wtaps * a.N : 1;  // per channel
  const long long wtp = DGRAD ? a.N : a.KC;                 // per tap
  const int dwt = ps > 1 ? ps : 1;                          // next tap in a row
  const int dwr = ps > 1 ? ps * a.kw_full - ps * (a.kw - 1) : 1;  // next kernel row
  const int wtap0 = ps > 1 ? (a.ty0 + ps * ti) * a.kw_full + a.tx0 + ps * tj : tap;
  long long wb = ((long long)cbi * BK * wst + (long long)wtap0 * wtp) * ES;
  const long long dw_step = BK * wst * ES;
  const long long dw_tap = (-(long long)(CB - 1) * BK * wst + (long long)dwt * wtp) * ES;
  const long long dw_row = (-(long long)(CB - 1) * BK * wst + (long long)dwr * wtp) * ES;
  // the advance as masked adds (a conditional 64-bit choice compiles to
  // branches): + step, + (tap - step) on a new tap, + (row - tap) on a new
  // kernel row
  const long long dd_tap = d_tap - d_step, dd_row = d_row - d_tap;
  const long long ddw_tap = dw_tap - dw_step, ddw_row = dw_row - dw_tap;
  // the zero block's address, made opaque so that it is computed once and
  // not rebuilt in the loop
  const void *zblk = &g_zero16[0];
  asm volatile("" : "+s"(zblk));

  uint4 ra[NA], rb[NBL];
  // bounds tests use non-short-circuit '&' so that no test becomes a branch
  // (st: the LDS stage a direct copy writes)
  auto gload = [&](int st) {
    if (tpk) {
      // vector kv of a tile row holds channels [0, KC) of tap kpk*KR + kv
      const int tp = kpk * KR + kv;
      const bool tok = tp < taps;
      uint32_t ti_, tj_;
      fdiv_qr((uint32_t)(tok ? tp : 0), a.fkw, ti_, tj_);
#pragma unroll
      for (int i = 0; i < NA; ++i) {
        const int sy = by[i] + (int)ti_, sx = bx[i] + (int)tj_;
        const bool ok = tok & am[i] & (sx >= 0) & (sy >= a.sy0) & (sy < a.sy1) & (sx < a.Ws);
        const long long off = rbase[i] + (long long)ti_ * srow + (long long)tj_ * a.src.C;
        ra[i] = load16<T, false>(ok ? src + off : src, ok, a.KC);
      }
#pragma unroll
      for (int j = 0; j < NBL; ++j) {
        const bool ok = bvld[j] & tok;
        const long long off = bbase[j] - kv * E + (long long)tp * a.KC;
        rb[j] = load16<T, false>(ok ? w + off : w, ok, a.KC);
      }
      ++kpk;
      return;
    }
    const int cb = cbi * BK;
    const int c0 = cb + kv * E;
    const bool cok = c0 < a.KC;
    const int lim = a.KC - c0;
    const long long tofs = (long long)ti * srow + (long long)tj * a.src.C;  // uniform
    if (DMA && ONE) {
      // one tap: the row's validity is fixed, K steps through channel blocks
      const long long co = (long long)cb * sizeof(T);
#pragma unroll
      for (int i = 0; i < NA; ++i)
        load16_lds_a(rp[i] + co, rowok[i] & cok,
                     lds_a + st * ASB + (wrow + RS * i) * LDK * (uint32_t)sizeof(T), zblk);
#pragma unroll
      for (int j = 0; j < NBL; ++j)
        load16_lds_a(wp[j] + co, bvld[j] & cok,
                     lds_b + st * BSB + (wrow + RS * j) * LDK * (uint32_t)sizeof(T), zblk);
      ++cbi;
      return;
    }
    if (RMASK) {
#pragma unroll
      for (int i = 0; i < NA; ++i) {
        const bool ok = ((uint32_t)(tmask[i] >> tap) & 1u) & cok;
        ra[i] = load16_sel(rp[i] + ub, ok, zblk);
      }
#pragma unroll
      for (int j = 0; j < NBL; ++j) {
        const bool ok = bvld[j] & (cb + bk0 + BKS * j < a.KC);
        rb[j] = load16_sel(wp[j] + wb, ok, zblk);
      }
    } else if (TMASK) {
#pragma unroll
      for (int i = 0; i < NA; ++i)
        load16_lds_a(rp[i] + ub, ((uint32_t)(tmask[i] >> tap) & 1u) & cok,
                     lds_a + st * ASB + (wrow + RS * i) * LDK * (uint32_t)sizeof(T), zblk);
#pragma unroll
      for (int j = 0; j < NBL; ++j)
        load16_lds_a(wp[j] + wb, bvld[j] & cok,
                     lds_b + st * BSB + (wrow + RS * j) * LDK * (uint32_t)sizeof(T), zblk);
    } else {
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      int sy, sx;
      bool ok;
      long long off;
      if (ONE) {
        ra[i] = load16z(src, (rbase[i] + c0) * (long long)sizeof(T), rowok[i] & cok);
        continue;
      }
      if (DGRAD && !S1) {
        const int ty = by[i] - ti, tx = bx[i] - tj;
        sy = ty / a.sh;
        sx = tx / a.sw;
        ok = (ty >= 0) & (tx >= 0) & (sy * a.sh == ty) & (sx * a.sw == tx);
        off = abase[i] + sy * srow + (long long)sx * a.src.C + c0;
      } else {
        sy = DGRAD ? by[i] - ti : by[i] + ti;
        sx = DGRAD ? bx[i] - tj : bx[i] + tj;
        ok = sx >= 0;
        off = (DGRAD ? rbase[i] - tofs : rbase[i] + tofs) + c0;
      }
      ok = ok & am[i] & cok & (sy >= a.sy0) & (sy < a.sy1) & (sx < a.Ws);
      if (VEC) {
        ra[i] = load16z(src, off * (long long)sizeof(T), ok);
      } else {
        const T *p = src;
        if (ok) p = src + off;
        ra[i] = load16<T, VEC>(p, ok, lim);
      }
    }
#pragma unroll
    for (int j = 0; j < NBL; ++j) {
      bool ok;
      long long off;
      int blim;
      if (DGRAD) {
        const int o = cb + bk0 + BKS * j;
        ok = bvld[j] & (o < a.KC);
        const int wtap = ps > 1 ? (a.ty0 + ps * ti) * a.kw_full + a.tx0 + ps * tj : tap;
        off = bbase[j] + ((long long)cb * wtaps + wtap) * a.N;
        blim = a.N - bn[j];
      } else {
        ok = bvld[j] & cok;
        off = bbase[j] + (long long)tap * a.KC + cb;
        blim = lim;
      }
      if (VEC) {
        rb[j] = load16z(w, off * (long long)sizeof(T), ok);
      } else {
        const T *p = ok ? w + off : w;
        rb[j] = load16<T, VEC>(p, ok, blim);
      }
    }
    }
    // advance to the next (tap, channel block) without branches
    const bool wrap = ++cbi == CB;
    cbi = wrap ? 0 : cbi;
    tap += wrap ? 1 : 0;
    tj += wrap ? 1 : 0;
    const bool nrow = tj == a.kw;
    tj = nrow ? 0 : tj;
    ti += nrow ? 1 : 0;
    if (MASK) {
      const long long mw = -(long long)wrap, mr = -(long long)nrow;
      ub += d_step + (dd_tap & mw) + (dd_row & mr);
      wb += dw_step + (ddw_tap & mw) + (ddw_row & mr);
    }
  };

  f32x16 acc[2][NB];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const int wm = (wave & 1) * 64, wn = (wave >> 1) * (BN / 2);
  auto store = [&](int st) {
#pragma unroll
    for (int i = 0; i < NA; ++i)
      *(uint4 *)(&As[st][(tid / KR + RS * i) * LDK + swz(tid / KR + RS * i, kv) * E]) = ra[i];
#pragma unroll
    for (int j = 0; j < NBL; ++j) {
      if (BKM) {
        *(uint4 *)(&Bs[st][(bk0 + BKS * j) * PB + (tid % BV) * E]) = rb[j];
      } else if (DGRAD) {
        union {
          uint4 u;
          T e[E];
        } t;
        t.u = rb[j];
#pragma unroll
        for (int e = 0; e < E; ++e)
          Bs[st][((tid % BV) * E + e) * LDK + bk0 + BKS * j] = t.e[e];
      } else {
        *(uint4 *)(&Bs[st][(tid / KR + RS * j) * LDK + swz(tid / KR + RS * j, kv) * E]) = rb[j];
      }
    }
  };
  const int n = kend - kbeg;
  using FR = Frag<T, BN, KR, 0, BKM>;
  FR f0, f1;
  int t = 0;
  if constexpr (DMA) {
    // Tile t+ST is copied into the stage of tile t once every wave has read
    // tile t; a step waits only for tile t+1, so a copy has ST-1 steps to
    // arrive. LD: copies per thread per tile; wait_tiles(k) leaves the
    // copies of the k most recent tiles in flight.
    constexpr int LD = NA + NBL;
    auto wait_tiles = [](int k) {
      if (ST > 3 && k >= 2) wait_vmcnt<(ST > 3 ? 2 : 0) * LD>();
      else if (k == 1) wait_vmcnt<LD>();
      else wait_vmcnt<0>();
    };
#pragma unroll
    for (int i = 0; i < ST; ++i)
      if (i < n) gload(i);
    wait_tiles(min(n, ST) - 1);
    __syncthreads();
    if (n > 0) f0.load(As[0], Bs[0], wm, wn, lane);
    int sc = 0;  // stage of tile t
    auto dstep = [&](int t, FR &cur, FR &nxt) {
      const int s1 = sc == ST - 1 ? 0 : sc + 1;
      if (t + 1 < n) {
        wait_tiles(min(n - 1, t + ST - 1) - t - 1);
        __syncthreads();
        nxt.load(As[s1], Bs[s1], wm, wn, lane);
        if (t + ST < n) gload(sc);
      }
      cur.mma(acc);
      sc = s1;
    };
    auto dstep_full = [&](FR &cur, FR &nxt) {
      const int s1 = sc == ST - 1 ? 0 : sc + 1;
      wait_vmcnt<(ST - 2) * LD>();
      __syncthreads();
      nxt.load(As[s1], Bs[s1], wm, wn, lane);
      gload(sc);
      cur.mma(acc);
      interleave_step<FR::NMFMA, FR::NDSR, 0, LD>();
      sc = s1;
    };
    for (; t + ST + 1 < n; t += 2) {
      dstep_full(f0, f1);
      dstep_full(f1, f0);
    }
    for (; t + 1 < n; t += 2) {
      dstep(t, f0, f1);
      dstep(t + 1, f1, f0);
    }
    if (t < n) dstep(t, f0, f1);
    // the stages are reused by the epilogue
    __syncthreads();
  } else {
  if (n > 0) {
    gload(0);
    store(0);
  }
  if (n > 1) {
    gload(0);
    store(1);
  }
  if (n > 2) gload(0);
  __syncthreads();
  if (n > 0) f0.load(As[0], Bs[0], wm, wn, lane);
  int s1 = 1, s2 = 2;  // stages of tiles t+1 and t+2
  auto step = [&](int t, FR &cur, FR &nxt) {
    if (t + 1 < n) nxt.load(As[s1], Bs[s1], wm, wn, lane);
    if (t + 2 < n) {
      store(s2);
      if (t + 3 < n) gload(0);
    }
    cur.mma(acc);
    s1 = s2;
    s2 = s2 == ST - 1 ? 0 : s2 + 1;
    __syncthreads();
  };
  // steady state: every part of the step exists, so the step is one
  // straight-line block with an explicit instruction interleave
  constexpr int NDSW = NA + ((DGRAD && !BKM) ? NBL * E : NBL);
  auto step_full = [&](FR &cur, FR &nxt) {
    nxt.load(As[s1], Bs[s1], wm, wn, lane);
    store(s2);
    gload(0);
    cur.mma(acc);
    interleave_step<FR::NMFMA, FR::NDSR, NDSW, NA + NBL>();
    s1 = s2;
    s2 = s2 == ST - 1 ? 0 : s2 + 1;
    __syncthreads();
  };
  for (; t + 4 < n; t += 2) {
    step_full(f0, f1);
    step_full(f1, f0);
  }
  for (; t + 1 < n; t += 2) {
    step(t, f0, f1);
    step(t + 1, f1, f0);
  }
  if (t < n) step(t, f0, f1);
  }

  if (gridDim.z > 1) {
    // split-K: raw partial sums, reduced in split order by the epilogue kernel
    float *part = a.part + (long long)tl.z * M * a.N;
    const int col = lane & 31;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int m = m0 + wm + 32 * i + acc_row(v, lane);
        if (m >= M) continue;
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          const int n = n0 + wn + 32 * j + col;
          if (n < a.N) part[(long long)m * a.N + n] = acc[i][j][v];
        }
      }
    return;
  }

  // epilogue
  const int col = lane & 31;
  const long long drow = (long long)a.dst.W * a.N;
  if (!DGRAD && (a.N % E) == 0) {
    // forward: affine, ReLU (and the optional mask) in registers, the tile
    // staged in LDS, then whole 16-byte row chunks stored per thread
    T *Ct = reinterpret_cast<T *>(smem);
    constexpr int CPR = BN / E;     // 16-byte chunks per tile row
    constexpr int RPP = 256 / CPR;  // tile rows per pass
    const int cc = tid % CPR;
    const int n = n0 + cc * E;
    for (int h0 = 0; h0 < BM; h0 += HR) {
    if (h0) __syncthreads();
    if (wm >= h0 && wm < h0 + HR) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int r = wm - h0 + 32 * i + acc_row(v, lane);
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          const int cl = wn + 32 * j + col;
          const int nn = n0 + cl;
          float val = acc[i][j][v];
          if (nn < a.N) {
            if (a.scale) val = val * a.scale[nn] + a.shift[nn];
            if (a.relu) val = val > 0.f ? val : 0.f;
          }
          stf(&Ct[r * CP + cl], val);
        }
      }
    }
    __syncthreads();
    for (int r = h0 + tid / CPR; r < h0 + HR; r += RPP) {
      const int m = m0 + r;
      if (m >= M || n >= a.N) continue;
      uint32_t t_, x_, b_, y_;
      fdiv_qr((uint32_t)m, a.fw, t_, x_);
      fdiv_qr(t_, a.fr, b_, y_);
      const int x = a.px0 + ps * (int)x_, y = a.y0 + ps * (int)y_, b = (int)b_;
      const long long off = b * a.dst.bs + (y - a.dst.row0) * drow + (long long)x * a.N + n;
      uint4 q = *(const uint4 *)&Ct[(r - h0) * CP + cc * E];
      if (a.res.p) {
        // fused residual add: the stored conv value plus the add's other
        // input, then the add's ReLU
        union {
          uint4 u;
          T e[E];
        } cv, rv;
        cv.u = q;
        rv.u = *(const uint4 *)((const T *)a.res.p + b * a.res.bs + (y - a.res.row0) * drow +
                                (long long)x * a.N + n);
#pragma unroll
        for (int e = 0; e < E; ++e) {
          float v = ldf(&cv.e[e]) + ldf(&rv.e[e]);
          if (a.res_relu) v = v > 0.f ? v : 0.f;
          stf(&cv.e[e], v);
        }
        q = cv.u;
      }
      *(uint4 *)((T *)a.dst.p + off) = q;
      if (a.mask) {
        union {
          uint4 u;
          T e[E];
        } w;
        w.u = q;
        uint8_t *mk = a.mask + (((long long)b * a.mask_h + y) * a.Wd + x) * a.N + n;
#pragma unroll
        for (int e = 0; e < E; ++e) mk[e] = ldf(&w.e[e]) > 0.f ? 1 : 0;
      }
    }
    }
    return;
  }
  if (DGRAD && (a.N % 4) == 0) {
    // input gradient: the float32 tile staged in LDS, then 16-byte
    // read-add-write of the error window
    constexpr int FP = BN + 4;
    float *Ct = reinterpret_cast<float *>(smem);
    constexpr int CPR = BN / 4;
    constexpr int RPP = 256 / CPR;
    const int cc = tid % CPR;
    const int n = n0 + cc * 4;
    for (int h0 = 0; h0 < BM; h0 += HR) {
    if (h0) __syncthreads();
    if (wm >= h0 && wm < h0 + HR) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int r = wm - h0 + 32 * i + acc_row(v, lane);
#pragma unroll
        for (int j = 0; j < NB; ++j) Ct[r * FP + wn + 32 * j + col] = acc[i][j][v];
      }
    }
    __syncthreads();
    for (int r = h0 + tid / CPR; r < h0 + HR; r += RPP) {
      const int m = m0 + r;
      if (m >= M || n >= a.N) continue;
      uint32_t t_, x_, b_, y_;
      fdiv_qr((uint32_t)m, a.fw, t_, x_);
      fdiv_qr(t_, a.fr, b_, y_);
      const int x = a.px0 + ps * (int)x_, y = a.y0 + ps * (int)y_, b = (int)b_;
      float4 *d = (float4 *)((float *)a.dst.p + b * a.dst.bs + (y - a.dst.row0) * drow +
                             (long long)x * a.N + n);
      const float4 q = *(const float4 *)&Ct[(r - h0) * FP + cc * 4];
      const float *bp = dgrad_base(a, b, y, (long long)x * a.N + n, (const float *)d);
      float4 o = bp ? *(const float4 *)bp : make_float4(0.f, 0.f, 0.f, 0.f);
      float ov[4] = {o.x + q.x, o.y + q.y, o.z + q.z, o.w + q.w};
      dgrad_out<T, 4>(a, b, y, x, n, ov, (float *)d);
    }
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int m = m0 + wm + 32 * i + acc_row(v, lane);
      if (m >= M) continue;
      uint32_t t_, x_, b_, y_;
      fdiv_qr((uint32_t)m, a.fw, t_, x_);
      fdiv_qr(t_, a.fr, b_, y_);
      const int x = a.px0 + ps * (int)x_, y = a.y0 + ps * (int)y_, b = (int)b_;
      const long long off = b * a.dst.bs + (y - a.dst.row0) * drow + (long long)x * a.N;
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const int n = n0 + wn + 32 * j + col;
        if (n >= a.N) continue;
        float val = acc[i][j][v];
        if (DGRAD) {
          float *d = (float *)a.dst.p + off + n;
          const float *bp = dgrad_base(a, b, y, (long long)x * a.N + n, d);
          float ov[4] = {(bp ? *bp : 0.f) + val, 0.f, 0.f, 0.f};
          dgrad_out<T, 1>(a, b, y, x, n, ov, d);
        } else {
          if (a.scale) val = val * a.scale[n] + a.shift[n];
          if (a.relu) val = val > 0.f ? val : 0.f;
          stf((T *)a.dst.p + off + n, val);
          if (a.mask)
            a.mask[(((long long)b * a.mask_h + y) * a.Wd + x) * a.N + n] =
                val > 0.f ? 1 : 0;
        }
      }
    }
  }
}

// Sum the split-K partials of every output element in split order, then
// apply the forward epilogue (affine, ReLU, store, mask) or add the input
// gradient into the error window.
// Sum the split-K partials of every output element in a fixed order
// (G groups of threads each add the splits z = g, g + G, ...; the G group
// sums are then added in order), then apply the forward epilogue (affine,
// ReLU, store, mask) or add the input gradient into the error window.
template <typename T, bool DGRAD, int V>
__global__ __launch_bounds__(256) void conv_split_epilogue(ConvArgs a, int splits, int G) {
  __shared__ float red[256 * 4];
  const int R = a.y1 - a.y0;
  const long long M = (long long)a.B * R * a.Wd;
  const long long MN = M * a.N;
  const long long drow = (long long)a.dst.W * a.N;
  const int ps = DGRAD && a.pst > 1 ? a.pst : 1;
  const int epb = 256 / G;  // vectors per block
  const int g = threadIdx.x / epb, e = threadIdx.x - g * epb;
  const long long idx = ((long long)blockIdx.x * epb + e) * V;
  float val[4] = {0.f, 0.f, 0.f, 0.f};
  if (idx < MN) {
    for (int z = g; z < splits; z += G) {
      float q[4];
      ldv<float, V>(a.part + z * MN + idx, q);
#pragma unroll
      for (int k = 0; k < V; ++k) val[k] += q[k];
    }
  }
#pragma unroll
  for (int k = 0; k < V; ++k) red[(g * epb + e) * 4 + k] = val[k];
  __syncthreads();
  if (g != 0 || idx >= MN) return;
#pragma unroll
  for (int k = 0; k < V; ++k) val[k] = 0.f;
  for (int gg = 0; gg < G; ++gg)
#pragma unroll
    for (int k = 0; k < V; ++k) val[k] += red[(gg * epb + e) * 4 + k];
  // M * N < 2^32 for every split launch (the launcher checks)
  uint32_t m_, n_, t_, x_, b_, y_;
  fdiv_qr((uint32_t)idx, a.fn, m_, n_);
  fdiv_qr(m_, a.fw, t_, x_);
  fdiv_qr(t_, a.fr, b_, y_);
  const int n = (int)n_, x = a.px0 + ps * (int)x_, y = a.y0 + ps * (int)y_, b = (int)b_;
  const long long off = b * a.dst.bs + (y - a.dst.row0) * drow + (long long)x * a.N + n;
  if (DGRAD) {
    float *d = (float *)a.dst.p + off;
    const float *bp = dgrad_base(a, b, y, (long long)x * a.N + n, d);
    float q[4] = {0.f, 0.f, 0.f, 0.f};
    if (bp) ldv<float, V>(bp, q);
#pragma unroll
    for (int k = 0; k < V; ++k) q[k] += val[k];
    dgrad_out<T, V>(a, b, y, x, n, q, d);
  } else {
    float rv[4];
    if (a.res.p)
      ldv<T, V>((const T *)a.res.p + b * a.res.bs + (y - a.res.row0) * drow +
                    (long long)x * a.N + n, rv);
#pragma unroll
    for (int k = 0; k < V; ++k) {
      if (a.scale) val[k] = val[k] * a.scale[n + k] + a.shift[n + k];
      if (a.relu) val[k] = val[k] > 0.f ? val[k] : 0.f;
      if (a.res.p) {
        // fused residual add on the value as stored, then the add's ReLU
        T t;
        stf(&t, val[k]);
        val[k] = ldf(&t) + rv[k];
        if (a.res_relu) val[k] = val[k] > 0.f ? val[k] : 0.f;
      }
      if (a.mask)
        a.mask[(((long long)b * a.mask_h + y) * a.Wd + x) * a.N + n + k] = val[k] > 0.f ? 1 : 0;
    }
    stv<T, V>((T *)a.dst.p + off, val);
  }
}


#ifndef LRCNN_CONV_KR
#define LRCNN_CONV_KR 4
#endif

template <typename T, bool DGRAD>
static int conv_launch(const ConvArgs &a0, hipStream_t s) {
  constexpr int KR = LRCNN_CONV_KR;
  using CF = Cfg<T, KR>;
  ConvArgs a = a0;
  const int M = a.B * (a.y1 - a.y0) * a.Wd;
  if (M <= 0 || a.N <= 0) return 0;
  // (the 16-byte loaders test taps against a 64-bit mask: larger kernels
  // take the element-wise loader)
  const bool vec = (a.KC % CF::E) == 0 && (!DGRAD || (a.N % CF::E) == 0) &&
                   a.kh * a.kw <= 64 && a.kw < 64;
  a.tpack = !vec && conv_tap_packed(a.KC, (int)sizeof(T), DGRAD);
  a.fkw = fast_div((uint32_t)a.kw);
  const int KT = a.tpack ? (a.kh * a.kw + KR - 1) / KR : a.kh * a.kw * ((a.KC + CF::BK - 1) / CF::BK);
  const ConvTiles ct = conv_tiles(M, a.N, KT, a.part ? a.part_bytes : 0, (int)sizeof(T));
  const int bn = ct.bn;
  const int splits = ct.splits;
  // a fused residual add needs the vector epilogues of the forward
  if (a.res.p && (DGRAD || (a.N % CF::E) != 0)) return (int)hipErrorInvalidValue;
  // split partial sums must fit the buffer (the schedule never exceeds it)
  if (splits > 1 && (!a.part || (size_t)splits * (size_t)M * (size_t)a.N * 4 > a.part_bytes))
    return (int)hipErrorInvalidValue;
  if (splits > 1 && (long long)M * a.N >= (1ll << 32)) return (int)hipErrorInvalidValue;
  a.fw = fast_div((uint32_t)a.Wd);
  a.fr = fast_div((uint32_t)(a.y1 - a.y0));
  a.fn = fast_div((uint32_t)a.N);
  a.kts = (KT + splits - 1) / splits;
  dim3 grid((M + BM - 1) / BM, (a.N + bn - 1) / bn, splits);
  int pr = -1;
  if (prof::on) {
    // algorithmic FLOPs: forward 2*M*N*K; input gradient 2 * consumer pixels
    // * C_out * taps * C_in (taps that a stride skips are not counted)
    const double taps = (double)a.kh * a.kw;
    const double fl = DGRAD && a.pst <= 1 ? 2.0 * a.B * (a.sy1 - a.sy0) * a.Ws * a.KC * taps * a.N
                                          : 2.0 * M * a.N * taps * a.KC;
    std::string nm = std::string("conv_gemm_kernel<") + (sizeof(T) == 4 ? "float" : "bf16") +
                     ", " + std::to_string(bn) + (DGRAD ? ", dgrad" : ", fwd") +
                     (vec ? ", vec>" : ", scalar>");
    pr = prof::begin(nm, fl, s);
  }
  // the input gradient of a strided convolution divides by the stride
  // (a phase of it is dense)
  const bool s1 = !DGRAD || (a.sh == 1 && a.sw == 1) || a.pst > 1;
  const bool one = vec && s1 && a.kh == 1 && a.kw == 1;
  if (bn == 64) {
    if (!s1) {
      if (vec) conv_gemm_kernel<T, 64, KR, DGRAD, true, false><<<grid, 256, 0, s>>>(a);
      else conv_gemm_kernel<T, 64, KR, DGRAD, false, false><<<grid, 256, 0, s>>>(a);
    } else if (one) {
      conv_gemm_kernel<T, 64, KR, DGRAD, true, true, true><<<grid, 256, 0, s>>>(a);
    } else if (vec) {
      conv_gemm_kernel<T, 64, KR, DGRAD, true, true><<<grid, 256, 0, s>>>(a);
    } else {
      conv_gemm_kernel<T, 64, KR, DGRAD, false, true><<<grid, 256, 0, s>>>(a);
    }
  } else {
    if (!s1) {
      if (vec) conv_gemm_kernel<T, 128, KR, DGRAD, true, false><<<grid, 256, 0, s>>>(a);
      else conv_gemm_kernel<T, 128, KR, DGRAD, false, false><<<grid, 256, 0, s>>>(a);
    } else if (one) {
      conv_gemm_kernel<T, 128, KR, DGRAD, true, true, true><<<grid, 256, 0, s>>>(a);
    } else if (vec) {
      conv_gemm_kernel<T, 128, KR, DGRAD, true, true><<<grid, 256, 0, s>>>(a);
    } else {
      conv_gemm_kernel<T, 128, KR, DGRAD, false, true><<<grid, 256, 0, s>>>(a);
    }
  }
  prof::end(pr, s);
  if (splits > 1) {
    int p2 = prof::begin("conv_split_epilogue", 0.0, s);
    const int G = splits >= 8 ? 8 : splits >= 4 ? 4 : 2;
    const long long vecs = a.N % 4 == 0 ? (long long)M * a.N / 4 : (long long)M * a.N;
    const unsigned blocks = (unsigned)((vecs + 256 / G - 1) / (256 / G));
    if (a.N % 4 == 0)
      conv_split_epilogue<T, DGRAD, 4><<<blocks, 256, 0, s>>>(a, splits, G);
    else
      conv_split_epilogue<T, DGRAD, 1><<<blocks, 256, 0, s>>>(a, splits, G);
    prof::end(p2, s);
  }
  return (int)hipGetLastError();
}

// Phases of the input gradient of a strided convolution. Producer pixel y
// receives tap i of the s-strided kernel only when (y + ph - i) is a
// multiple of s, i.e. i = (y + ph) mod s + s * i'. Grouping producer rows
// and columns by (y + ph) mod s gives s^2 dense problems, each with about
// 1/s^2 of the taps, instead of one launch in which the MFMAs also multiply
// the s^2 - 1 of every s^2 (pixel, tap) pairs that are zero. One dimension:
// the first pixel >= lo of residue r, the count of such pixels below hi,
// and the taps of the phase.
struct PhaseDim {
  int first, count, taps;
};
static PhaseDim phase_dim(int lo, int hi, int p, int k, int s, int r) {
  PhaseDim d;
  d.first = lo + (((r - (lo + p)) % s) + s) % s;
  d.count = d.first < hi ? (hi - d.first + s - 1) / s : 0;
  d.taps = r < k ? (k - r + s - 1) / s : 0;
  return d;
}

static thread_local int g_phases = 0;  // 0: by estimate, 1: always, 2: never
void set_dgrad_phases(int mode) { g_phases = mode; }

template <typename T, bool DGRAD>
static int conv_dispatch(const ConvArgs &a, hipStream_t s) {
  if (!DGRAD || (a.sh == 1 && a.sw == 1) || a.sh != a.sw || a.pst > 1 || g_phases == 2)
    return conv_launch<T, DGRAD>(a, s);
  const int M = a.B * (a.y1 - a.y0) * a.Wd;
  if (M <= 0 || a.N <= 0) return 0;
  // phases when their estimated durations (plus a launch each) beat the
  // single launch over all taps
  const int es = (int)sizeof(T);
  const size_t cap = a.part ? a.part_bytes : 0;
  const double one = conv_tiles(M, a.N, conv_k_iters(a.kh * a.kw, a.KC, es, true), cap, es).us;
  double ph = 0;
  for (int ry = 0; ry < a.sh; ++ry)
    for (int rx = 0; rx < a.sw; ++rx) {
      const PhaseDim py = phase_dim(a.y0, a.y1, a.ph, a.kh, a.sh, ry);
      const PhaseDim px = phase_dim(0, a.Wd, a.pw, a.kw, a.sw, rx);
      if (py.count == 0 || px.count == 0 || (py.taps * px.taps == 0 && !a.dst_init)) continue;
      ph += 5.0 + conv_tiles((long long)a.B * py.count * px.count, a.N,
                             conv_k_iters(py.taps * px.taps, a.KC, es, true), cap, es).us;
    }
  if (ph >= one && g_phases != 1) return conv_launch<T, DGRAD>(a, s);
  for (int ry = 0; ry < a.sh; ++ry)
    for (int rx = 0; rx < a.sw; ++rx) {
      const PhaseDim py = phase_dim(a.y0, a.y1, a.ph, a.kh, a.sh, ry);
      const PhaseDim px = phase_dim(0, a.Wd, a.pw, a.kw, a.sw, rx);
      // a phase without taps still writes its pixels when the launch
      // initializes the error window
      if (py.count == 0 || px.count == 0 || (py.taps * px.taps == 0 && !a.dst_init)) continue;
      ConvArgs b = a;
      b.pst = a.sh;
      b.y0 = py.first;
      b.y1 = py.first + py.count;
      b.px0 = px.first;
      b.Wd = px.count;
      b.ty0 = ry;
      b.tx0 = rx;
      b.kw_full = a.kw;
      b.taps_full = a.kh * a.kw;
      b.kh = py.taps * px.taps == 0 ? 0 : py.taps;
      b.kw = py.taps * px.taps == 0 ? 1 : px.taps;
      if (int e = conv_launch<T, DGRAD>(b, s)) return e;
    }
  return 0;
}

int launch_conv(int dt, int dgrad, const ConvArgs &a, void *stream) {
  hipStream_t s = (hipStream_t)stream;
  if (dt == DT_F32)
    return dgrad ? conv_dispatch<float, true>(a, s) : conv_dispatch<float, false>(a, s);
  return dgrad ? conv_dispatch<bf16, true>(a, s) : conv_dispatch<bf16, false>(a, s);
}


// ------------------------------------------------------------ weight grad
// A[m = co][k = pixel] = dc[pixel][co] and B[k = pixel][n = (tap, ci)] =
// input pixel under tap. Both are K-outer in memory, so both tiles are
// staged k-major ([k][row], 16-byte stores). The tile is WBM x 128: WBM =
// 128 (four waves of 64 x 64) or, for 64 output channels or fewer, WBM = 64
// (four waves of 64 x 32), so a narrow layer does not compute a half-empty
// tile.
#ifndef LRCNN_WG_OCC
#define LRCNN_WG_OCC 2
#endif
template <typename T, int WBM, bool AVEC, bool BVEC>
__global__ __launch_bounds__(256, LRCNN_WG_OCC) void wgrad_kernel(WgradArgs a, int kchunk,
                                                    float *dw) {
  constexpr int E = Cfg<T>::E, BK = Cfg<T>::BK;
  constexpr int BN = 128;
  constexpr int FBN = WBM == 128 ? 128 : 64;  // columns per wave: FBN / 2
  constexpr int NB = FBN / 64;
  constexpr int RV = BN / E;        // 16-byte vectors per B tile row
  constexpr int KS = 256 / RV;      // pixels of B loaded per pass
  constexpr int RVA = WBM / E;      // 16-byte vectors per A tile row
  constexpr int KSA = 256 / RVA;    // pixels of A loaded per pass
  constexpr int NPA = BK / KSA;     // A passes per tile
  constexpr int PA = WBM + E, PB = BN + E;
  constexpr int ASZ = BK * PA, BSZ = BK * PB;
  constexpr int ST = 3;
  __shared__ __align__(16) T As[ST][ASZ];
  __shared__ __align__(16) T Bs[ST][BSZ];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int R = a.y1 - a.y0;
  const int K = a.B * R * a.Wv;
  const int taps = a.kh * a.kw;
  const int N = taps * a.Ci;
  // one split's pixel range per run of workgroups on an XCD
  const TileId tl = xcd_tile(false);
  const int m0 = tl.x * WBM, n0 = tl.y * BN;
  const int kbeg = tl.z * kchunk;
  const int kend = min(K, kbeg + kchunk);
  const int rv = tid % RV, kk0 = tid / RV;
  const int rva = tid % RVA, kka0 = tid / RVA;
  const T *dc = (const T *)a.dc;
  const T *src = (const T *)a.src.p;
  const long long srow = (long long)a.src.W * a.src.C;

  // this thread's B columns n0 + rv*E + e: (tap, channel) of each element
  const int nb0 = n0 + rv * E;
  const int tapv = nb0 / a.Ci, cv = nb0 - (nb0 / a.Ci) * a.Ci;
  const int tiv = tapv / a.kw, tjv = tapv - (tapv / a.kw) * a.kw;
  const int ov = m0 + rva * E;

  union V16 {
    uint4 u;
    T e[E];
  };
  V16 ra[NPA], rb[2];
  int k0 = kbeg;
  const bool ovok = ov < a.Co, nbok = nb0 < N;
  // channel counts that are not a multiple of E (the first layer): the
  // (tap, channel) of each of this thread's E columns, fixed for the launch
  int cti[BVEC ? 1 : E], ctj[BVEC ? 1 : E], cc[BVEC ? 1 : E];
  bool cok[BVEC ? 1 : E];
  if (!BVEC) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int n = nb0 + e;
      const int tap = n / a.Ci;
      cc[e] = n - tap * a.Ci;
      cti[e] = tap / a.kw;
      ctj[e] = tap - cti[e] * a.kw;
      cok[e] = n < N;
    }
  }
  const T *zero_e = (const T *)&g_zero16[0];
  // bounds tests use non-short-circuit '&' so that no test becomes a branch
  auto gload = [&]() {
#pragma unroll
    for (int i = 0; i < NPA; ++i) {
      // A: E output channels of pixel p
      const int p = k0 + kka0 + KSA * i;
      const bool pk = p < kend;
      if (AVEC) {
        ra[i].u = load16z(dc, ((long long)p * a.Co + ov) * (long long)sizeof(T), pk & ovok);
      } else {
#pragma unroll
        for (int e = 0; e < E; ++e)
          ra[i].e[e] = (pk && ov + e < a.Co) ? dc[(long long)p * a.Co + ov + e] : (T)0;
      }
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      // B: E input values of pixel p under the column's tap
      const int p = k0 + kk0 + KS * i;
      const bool pk = p < kend;
      uint32_t t, x, yy, b;
      fdiv_qr((uint32_t)(pk ? p : 0), a.fw, t, x);
      fdiv_qr(t, a.fr, b, yy);
      const int y = a.y0 + (int)yy;
      if (BVEC) {
        const int sy = y * a.sh - a.ph + tiv, sx = x * a.sw - a.pw + tjv;
        const bool ok = pk & nbok & (sy >= 0) & (sy < a.Hs) & (sx >= 0) & (sx < a.Ws);
        const long long off =
            b * a.src.bs + (sy - a.src.row0) * srow + (long long)sx * a.src.C + cv;
        rb[i].u = load16z(src, off * (long long)sizeof(T), ok);
      } else {
        const long long bbase = b * a.src.bs - a.src.row0 * srow;
        const int sy0 = y * a.sh - a.ph, sx0 = x * a.sw - a.pw;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const int sy = sy0 + cti[e], sx = sx0 + ctj[e];
          const bool ok =
              pk & cok[e] & (sy >= 0) & (sy < a.Hs) & (sx >= 0) & (sx < a.Ws);
          const T *q = ok ? src + bbase + sy * srow + (long long)sx * a.src.C + cc[e] : zero_e;
          rb[i].e[e] = *q;
        }
      }
    }
    k0 += BK;
  };
  auto store = [&](int st) {
#pragma unroll
    for (int i = 0; i < NPA; ++i)
      *(uint4 *)(&As[st][(kka0 + KSA * i) * PA + rva * E]) = ra[i].u;
#pragma unroll
    for (int i = 0; i < 2; ++i)
      *(uint4 *)(&Bs[st][(kk0 + KS * i) * PB + rv * E]) = rb[i].u;
  };

  f32x16 acc[2][NB];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const int wm = WBM == 128 ? (wave & 1) * 64 : 0;
  const int wn = WBM == 128 ? (wave >> 1) * 64 : wave * 32;
  const int n = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;
  if (n > 0) {
    gload();
    store(0);
  }
  if (n > 1) {
    gload();
    store(1);
  }
  if (n > 2) gload();
  __syncthreads();
  using FR = Frag<T, FBN, 4, 1, 1, WBM, BN>;
  FR f0, f1;
  if (n > 0) f0.load(As[0], Bs[0], wm, wn, lane);
  int s1 = 1, s2 = 2;
  auto step = [&](int t, FR &cur, FR &nxt) {
    if (t + 1 < n) nxt.load(As[s1], Bs[s1], wm, wn, lane);
    if (t + 2 < n) {
      store(s2);
      if (t + 3 < n) gload();
    }
    cur.mma(acc);
    s1 = s2;
    s2 = s2 == ST - 1 ? 0 : s2 + 1;
    __syncthreads();
  };
  auto step_full = [&](FR &cur, FR &nxt) {
    nxt.load(As[s1], Bs[s1], wm, wn, lane);
    store(s2);
    gload();
    cur.mma(acc);
    interleave_step<FR::NMFMA, FR::NDSR, NPA + 2, NPA + 2>();
    s1 = s2;
    s2 = s2 == ST - 1 ? 0 : s2 + 1;
    __syncthreads();
  };
  int t = 0;
  if (AVEC && BVEC) {
    for (; t + 4 < n; t += 2) {
      step_full(f0, f1);
      step_full(f1, f0);
    }
  }
  for (; t + 1 < n; t += 2) {
    step(t, f0, f1);
    step(t + 1, f1, f0);
  }
  if (t < n) step(t, f0, f1);

  const int col = lane & 31;
  float *out = gridDim.z == 1 ? dw : a.out + (long long)tl.z * a.Co * N;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int m = m0 + wm + 32 * i + acc_row(v, lane);
      if (m >= a.Co) continue;
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const int nn = n0 + wn + 32 * j + col;
        if (nn >= N) continue;
        float *d = out + (long long)m * N + nn;
        if (gridDim.z == 1) *d = a.overwrite ? acc[i][j][v] : *d + acc[i][j][v];
        else *d = acc[i][j][v];
      }
    }
}

// dW += (first band: dW =) sum over the split partial sums in a fixed order
// (deterministic):
// eight groups of threads each add the splits z = g, g + 8, ... of 32
// vectors of V elements, then the eight group sums are added in order.
template <int V>
__global__ __launch_bounds__(256) void wgrad_reduce_kernel(const float *part, float *dw,
                                                           long long mn, int splits,
                                                           int overwrite) {
  __shared__ float red[8][32 * 4];
  const int g = threadIdx.x >> 5, e = threadIdx.x & 31;
  const long long i = ((long long)blockIdx.x * 32 + e) * V;
  float acc[4] = {0.f, 0.f, 0.f, 0.f}, q[4];
  if (i < mn) {
    for (int z = g; z < splits; z += 8) {
      ldv<float, V>(part + z * mn + i, q);
#pragma unroll
      for (int k = 0; k < V; ++k) acc[k] += q[k];
    }
  }
#pragma unroll
  for (int k = 0; k < V; ++k) red[g][e * 4 + k] = acc[k];
  __syncthreads();
  if (g == 0 && i < mn) {
    float sum[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int gg = 0; gg < 8; ++gg)
#pragma unroll
      for (int k = 0; k < V; ++k) sum[k] += red[gg][e * 4 + k];
    if (overwrite) {
#pragma unroll
      for (int k = 0; k < V; ++k) q[k] = sum[k];
    } else {
      ldv<float, V>(dw + i, q);
#pragma unroll
      for (int k = 0; k < V; ++k) q[k] += sum[k];
    }
    stv<float, V>(dw + i, q);
  }
}

template <typename T>
static int wgrad_dispatch(const WgradArgs &a0, float *dw, hipStream_t s) {
  WgradArgs a = a0;
  const int K = a.B * (a.y1 - a.y0) * a.Wv;
  const int N = a.kh * a.kw * a.Ci;
  if (K <= 0) return 0;
  // pixel indices are split by multiply-shift division
  a.fw = fast_div((uint32_t)a.Wv);
  a.fr = fast_div((uint32_t)(a.y1 - a.y0));
  constexpr int BK = Cfg<T>::BK;
  const WgradTiles wt = wgrad_tiles(a.Co, N, K, a.out ? a.part_bytes : 0, (int)sizeof(T));
  int splits = wt.splits;
  const int KT = (K + BK - 1) / BK;
  const int kchunk = (KT + splits - 1) / splits * BK;
  splits = (K + kchunk - 1) / kchunk;
  if (splits > 1 && (!a.out || (size_t)splits * (size_t)a.Co * (size_t)N * 4 > a.part_bytes))
    return (int)hipErrorInvalidValue;
  const bool avec = (a.Co % Cfg<T>::E) == 0, bvec = (a.Ci % Cfg<T>::E) == 0;
  const int wbm = wt.rows;
  dim3 grid((a.Co + wbm - 1) / wbm, (N + 127) / 128, splits);
  int pr = -1;
  if (prof::on)
    pr = prof::begin(std::string("wgrad_kernel<") + (sizeof(T) == 4 ? "float" : "bf16") +
                         (avec && bvec ? ", vec>" : ", scalar>"),
                     2.0 * K * a.Co * N, s);
  if (wbm == 64) {
    if (avec && bvec) wgrad_kernel<T, 64, true, true><<<grid, 256, 0, s>>>(a, kchunk, dw);
    else if (avec) wgrad_kernel<T, 64, true, false><<<grid, 256, 0, s>>>(a, kchunk, dw);
    else wgrad_kernel<T, 64, false, false><<<grid, 256, 0, s>>>(a, kchunk, dw);
  } else {
    if (avec && bvec) wgrad_kernel<T, 128, true, true><<<grid, 256, 0, s>>>(a, kchunk, dw);
    else if (avec) wgrad_kernel<T, 128, true, false><<<grid, 256, 0, s>>>(a, kchunk, dw);
    else wgrad_kernel<T, 128, false, false><<<grid, 256, 0, s>>>(a, kchunk, dw);
  }
  prof::end(pr, s);
  if (splits > 1) {
    long long mn = (long long)a.Co * N;
    int p2 = prof::begin("wgrad_reduce_kernel", 0.0, s);
    if (mn % 4 == 0)
      wgrad_reduce_kernel<4><<<(unsigned)((mn / 4 + 31) / 32), 256, 0, s>>>(a.out, dw, mn,
                                                                            splits, a.overwrite);
    else
      wgrad_reduce_kernel<1><<<(unsigned)((mn + 31) / 32), 256, 0, s>>>(a.out, dw, mn, splits,
                                                                        a.overwrite);
    prof::end(p2, s);
  }
  return (int)hipGetLastError();
}

int launch_wgrad(int dt, const WgradArgs &a, float *dw, void *stream) {
  hipStream_t s = (hipStream_t)stream;
  return dt == DT_F32 ? wgrad_dispatch<float>(a, dw, s) : wgrad_dispatch<bf16>(a, dw, s);
}

// ------------------------------------------------------------- max-pool
template <typename T, int V>
__global__ void pool_fwd_kernel(PoolArgs a) {
  const int R = a.y1 - a.y0;
  const int CV = a.C / V;
  const long long total = (long long)a.B * R * a.Wd * CV;
  const long long srow = (long long)a.src.W * a.src.C;
  const long long drow = (long long)a.Wd * a.C;
  const bool fast = total < (1ll << 32);
  GRID_STRIDE(idx, total) {
    int c, x, yy, b;
    if (fast) {
      uint32_t t0, c0, t1, x0, b0, y0;
      fdiv_qr((uint32_t)idx, a.fcv, t0, c0);
      fdiv_qr(t0, a.fw, t1, x0);
      fdiv_qr(t1, a.fr, b0, y0);
      c = (int)c0 * V, x = (int)x0, yy = (int)y0, b = (int)b0;
    } else {
      c = (int)(idx % CV) * V;
      long long t = idx / CV;
      x = (int)(t % a.Wd);
      t /= a.Wd;
      yy = (int)(t % R);
      b = (int)(t / R);
    }
    const int y = a.y0 + yy;
    const T *src = (const T *)a.src.p + b * a.src.bs;
    float best[4];
    int bi[4] = {0, 0, 0, 0};
    for (int i = 0; i < a.kh; ++i) {
      const int sy = y * a.sh - a.ph + i;
      for (int j = 0; j < a.kw; ++j) {
        const int sx = x * a.sw - a.pw + j;
        float v[4];
        if (sy >= 0 && sy < a.Hs && sx >= 0 && sx < a.Ws) {
          ldv<T, V>(src + (sy - a.src.row0) * srow + (long long)sx * a.src.C + c, v);
        } else {
#pragma unroll
          for (int e = 0; e < V; ++e) v[e] = -__builtin_huge_valf();
        }
        const int tp = i * a.kw + j;
#pragma unroll
        for (int e = 0; e < V; ++e)
          if (tp == 0 || v[e] > best[e]) {
            best[e] = v[e];
            bi[e] = tp;
          }
      }
    }
    const long long o = b * a.dst.bs + (y - a.dst.row0) * drow + (long long)x * a.C + c;
    stv<T, V>((T *)a.dst.p + o, best);
    const long long flat = (((long long)b * R + yy) * a.Wd + x) * a.C + c;
    const long long mfl = (((long long)b * a.mask_h + y) * a.Wd + x) * a.C + c;
#pragma unroll
    for (int e = 0; e < V; ++e) {
      if (a.am) a.am[flat + e] = (uint8_t)bi[e];
      if (a.mask) a.mask[mfl + e] = (uint8_t)bi[e];
    }
  }
}


int launch_pool_fwd(int dt, const PoolArgs &a0, void *stream) {
  const long long total = (long long)a0.B * (a0.y1 - a0.y0) * a0.Wd * a0.C;
  if (total <= 0) return 0;
  hipStream_t s = (hipStream_t)stream;
  const bool v4 = a0.C % 4 == 0;
  PoolArgs a = a0;
  a.fcv = fast_div((uint32_t)(v4 ? a.C / 4 : a.C));
  a.fw = fast_div((uint32_t)a.Wd);
  a.fr = fast_div((uint32_t)(a.y1 - a.y0));
  const unsigned g = grid_for(v4 ? total / 4 : total);
  if (dt == DT_F32) {
    if (v4) pool_fwd_kernel<float, 4><<<g, 256, 0, s>>>(a);
    else pool_fwd_kernel<float, 1><<<g, 256, 0, s>>>(a);
  } else {
    if (v4) pool_fwd_kernel<bf16, 4><<<g, 256, 0, s>>>(a);
    else pool_fwd_kernel<bf16, 1><<<g, 256, 0, s>>>(a);
  }
  return (int)hipGetLastError();
}

template <typename T, int V>
__global__ void pool_bwd_kernel(PoolBwdArgs a) {
  const int Ru = a.ub - a.ua, R = a.y1 - a.y0;
  const int CV = a.C / V;
  const long long total = (long long)a.B * Ru * a.Wu * CV;
  const long long vrow = (long long)a.Wv * a.C, urow = (long long)a.Wu * a.C;
  const bool fast = total < (1ll << 32);
  GRID_STRIDE(idx, total) {
    int c, xi, yi, b;
    if (fast) {
      uint32_t t0, c0, t1, x0, b0, y0;
      fdiv_qr((uint32_t)idx, a.fcv, t0, c0);
      fdiv_qr(t0, a.fw, t1, x0);
      fdiv_qr(t1, a.fr, b0, y0);
      c = (int)c0 * V, xi = (int)x0, yi = a.ua + (int)y0, b = (int)b0;
    } else {
      c = (int)(idx % CV) * V;
      long long t = idx / CV;
      xi = (int)(t % a.Wu);
      t /= a.Wu;
      yi = a.ua + (int)(t % Ru);
      b = (int)(t / Ru);
    }
    // windows y with y*sh - ph <= yi < y*sh - ph + kh, inside [y0, y1)
    const int ylo = max(a.y0, fdiv(yi + a.ph - a.kh, a.sh) + 1);
    const int yhi = min(a.y1 - 1, fdiv(yi + a.ph, a.sh));
    const int xlo = max(0, fdiv(xi + a.pw - a.kw, a.sw) + 1);
    const int xhi = min(a.Wv - 1, fdiv(xi + a.pw, a.sw));
    float sum[4] = {0.f, 0.f, 0.f, 0.f};
    for (int y = ylo; y <= yhi; ++y)
      for (int x = xlo; x <= xhi; ++x) {
        const int tp = (yi - (y * a.sh - a.ph)) * a.kw + (xi - (x * a.sw - a.pw));
        const long long ai = (((long long)b * R + (y - a.y0)) * a.Wv + x) * a.C + c;
        float dv[4];
        ldv<float, V>((const float *)a.dv.p + b * a.dv.bs + (y - a.dv.row0) * vrow +
                          (long long)x * a.C + c, dv);
#pragma unroll
        for (int e = 0; e < V; ++e)
          if (a.am[ai + e] == tp) sum[e] += dv[e];
      }
    float *d = (float *)a.du.p + b * a.du.bs + (yi - a.du.row0) * urow + (long long)xi * a.C + c;
    const float *bp = err_base(a.dst_init, a.cinit, a.cinit_t, b, yi, (long long)xi * a.C + c, d);
    float q[4] = {0.f, 0.f, 0.f, 0.f};
    if (bp) ldv<float, V>(bp, q);
#pragma unroll
    for (int e = 0; e < V; ++e) q[e] += sum[e];
    err_out<T, V>(a.eo, a.C, b, yi, xi, c, q, d);
  }
}

int launch_pool_bwd(int dt, const PoolBwdArgs &a0, void *stream) {
  const long long total = (long long)a0.B * (a0.ub - a0.ua) * a0.Wu * a0.C;
  if (total <= 0) return 0;
  PoolBwdArgs a = a0;
  a.fcv = fast_div((uint32_t)(a.C % 4 == 0 ? a.C / 4 : a.C));
  a.fw = fast_div((uint32_t)a.Wu);
  a.fr = fast_div((uint32_t)(a.ub - a.ua));
  hipStream_t s = (hipStream_t)stream;
  const bool v4 = a.C % 4 == 0;
  const unsigned g = grid_for(v4 ? total / 4 : total);
  if (dt == DT_F32) {
    if (v4) pool_bwd_kernel<float, 4><<<g, 256, 0, s>>>(a);
    else pool_bwd_kernel<float, 1><<<g, 256, 0, s>>>(a);
  } else {
    if (v4) pool_bwd_kernel<bf16, 4><<<g, 256, 0, s>>>(a);
    else pool_bwd_kernel<bf16, 1><<<g, 256, 0, s>>>(a);
  }
  return (int)hipGetLastError();
}

// ------------------------------------------------------- elementwise rows
// Row-range kernels over band windows. When a row's W*C elements are a
// multiple of 4, every thread handles 4 consecutive elements with one
// 16-byte (float32) or 8-byte (bfloat16) access per tensor.
template <typename T, int V>
__global__ void add_fwd_kernel(View a, View bb, View z, int relu, uint8_t *mask,
                               int mask_h, RowIter it) {
  const long long rowlen = (long long)z.W * z.C;
  GRID_STRIDE(idx, it.total) {
    int b, y, in;
    it.at(idx, V, b, y, in);
    float u[4], w[4];
    ldv<T, V>((const T *)a.p + view_off(a, b, y, in), u);
    ldv<T, V>((const T *)bb.p + view_off(bb, b, y, in), w);
#pragma unroll
    for (int e = 0; e < V; ++e) {
      u[e] += w[e];
      if (relu) u[e] = u[e] > 0.f ? u[e] : 0.f;
      if (mask) mask[((long long)b * mask_h + y) * rowlen + in + e] = u[e] > 0.f ? 1 : 0;
    }
    stv<T, V>((T *)z.p + view_off(z, b, y, in), u);
  }
}

int launch_add_fwd(int dt, View a, View b, View z, int relu, uint8_t *mask,
                   int mask_h, int B, int y0, int y1, int W, int C, void *stream) {
  const int V = ((long long)W * C) % 4 == 0 ? 4 : 1;
  RowIter it = row_iter(B, y0, y1, W, C, V);
  if (it.total <= 0) return 0;
  hipStream_t s = (hipStream_t)stream;
  const unsigned g = grid_for(it.total);
  if (dt == DT_F32) {
    if (V == 4) add_fwd_kernel<float, 4><<<g, 256, 0, s>>>(a, b, z, relu, mask, mask_h, it);
    else add_fwd_kernel<float, 1><<<g, 256, 0, s>>>(a, b, z, relu, mask, mask_h, it);
  } else {
    if (V == 4) add_fwd_kernel<bf16, 4><<<g, 256, 0, s>>>(a, b, z, relu, mask, mask_h, it);
    else add_fwd_kernel<bf16, 1><<<g, 256, 0, s>>>(a, b, z, relu, mask, mask_h, it);
  }
  return (int)hipGetLastError();
}

// One input side of the residual add's backward: either accumulate the
// error into the input's float32 window (dc == nullptr), or, when the input
// is a conv without ReLU whose only consumer is this add, write that conv's
// error operand rnd(scale[c] * d) directly (contiguous own rows, the layout
// act_bwd_kernel writes), which makes its window and its act_bwd pass
// unnecessary.
template <typename T, int V>
__device__ __forceinline__ void add_bwd_side(const AddSide &sd, long long idx, int in, int b,
                                             int y, const float (&d)[4]) {
  if (sd.dc) {
    float e[4];
#pragma unroll
    for (int k = 0; k < V; ++k) e[k] = sd.scale ? d[k] * sd.scale[(in + k) % sd.C] : d[k];
    stv<T, V>((T *)sd.dc + idx * V, e);
  } else {
    float x[4] = {0.f, 0.f, 0.f, 0.f};
    float *p = (float *)sd.win.p + view_off(sd.win, b, y, in);
    const float *bp = err_base(sd.init, sd.cinit, sd.cinit_t, b, y, in, p);
    if (bp) ldv<float, V>(bp, x);
#pragma unroll
    for (int k = 0; k < V; ++k) x[k] += d[k];
    stv<float, V>(p, x);
  }
}

template <typename T, int V>
__global__ void add_bwd_kernel(View dz, View z, AddSide sa, AddSide sb, int relu, RowIter it) {
  GRID_STRIDE(idx, it.total) {
    int b, y, in;
    it.at(idx, V, b, y, in);
    float d[4], zz[4];
    ldv<float, V>((const float *)dz.p + view_off(dz, b, y, in), d);
    if (relu) {
      ldv<T, V>((const T *)z.p + view_off(z, b, y, in), zz);
#pragma unroll
      for (int e = 0; e < V; ++e)
        if (!(zz[e] > 0.f)) d[e] = 0.f;
    }
    add_bwd_side<T, V>(sa, idx, in, b, y, d);
    add_bwd_side<T, V>(sb, idx, in, b, y, d);
  }
}

int launch_add_bwd(int dt, View dz, View z, const AddSide &sa, const AddSide &sb, int relu,
                   int B, int y0, int y1, int W, int C, void *stream) {
  const int V = ((long long)W * C) % 4 == 0 ? 4 : 1;
  RowIter it = row_iter(B, y0, y1, W, C, V);
  if (it.total <= 0) return 0;
  hipStream_t s = (hipStream_t)stream;
  const unsigned g = grid_for(it.total);
  if (dt == DT_F32) {
    if (V == 4) add_bwd_kernel<float, 4><<<g, 256, 0, s>>>(dz, z, sa, sb, relu, it);
    else add_bwd_kernel<float, 1><<<g, 256, 0, s>>>(dz, z, sa, sb, relu, it);
  } else {
    if (V == 4) add_bwd_kernel<bf16, 4><<<g, 256, 0, s>>>(dz, z, sa, sb, relu, it);
    else add_bwd_kernel<bf16, 1><<<g, 256, 0, s>>>(dz, z, sa, sb, relu, it);
  }
  return (int)hipGetLastError();
}

// Error operand of a conv (dc = rnd(scale[c] * dz * [z > 0]) over the
// band's own rows, contiguous) and, in the same launch, the float32 copy of
// the rows [lo, a) of dz that are carried to the previous band.
template <typename T, int V>
__global__ void act_bwd_kernel(View dz, View z, const float *scale, int relu, T *dc,
                               int C, RowIter it, View cdst, RowIter cit) {
  GRID_STRIDE(idx, it.total + cit.total) {
    int b, y, in;
    float d[4], zz[4];
    if (idx >= it.total) {
      cit.at(idx - it.total, V, b, y, in);
      ldv<float, V>((const float *)dz.p + view_off(dz, b, y, in), d);
      stv<float, V>((float *)cdst.p + view_off(cdst, b, y, in), d);
      continue;
    }
    it.at(idx, V, b, y, in);
    ldv<float, V>((const float *)dz.p + view_off(dz, b, y, in), d);
    if (relu) {
      ldv<T, V>((const T *)z.p + view_off(z, b, y, in), zz);
#pragma unroll
      for (int e = 0; e < V; ++e)
        if (!(zz[e] > 0.f)) d[e] = 0.f;
    }
    if (scale) {
#pragma unroll
      for (int e = 0; e < V; ++e) d[e] *= scale[(in + e) % C];
    }
    stv<T, V>(dc + idx * V, d);
  }
}

int launch_act_bwd(int dt, View dz, View z, const float *scale, int relu,
                   void *dc, int B, int y0, int y1, int W, int C, void *stream,
                   const View *carry, int c0, int c1) {
  const int V = ((long long)W * C) % 4 == 0 ? 4 : 1;
  RowIter it = row_iter(B, y0, y1, W, C, V);
  RowIter cit = row_iter(B, c0, carry ? c1 : c0, W, C, V);
  const View cd = carry ? *carry : View{};
  if (it.total + cit.total <= 0) return 0;
  hipStream_t s = (hipStream_t)stream;
  const unsigned g = grid_for(it.total + cit.total);
  if (dt == DT_F32) {
    if (V == 4)
      act_bwd_kernel<float, 4><<<g, 256, 0, s>>>(dz, z, scale, relu, (float *)dc, C, it, cd, cit);
    else
      act_bwd_kernel<float, 1><<<g, 256, 0, s>>>(dz, z, scale, relu, (float *)dc, C, it, cd, cit);
  } else {
    if (V == 4)
      act_bwd_kernel<bf16, 4><<<g, 256, 0, s>>>(dz, z, scale, relu, (bf16 *)dc, C, it, cd, cit);
    else
      act_bwd_kernel<bf16, 1><<<g, 256, 0, s>>>(dz, z, scale, relu, (bf16 *)dc, C, it, cd, cit);
  }
  return (int)hipGetLastError();
}

template <typename TS, typename TD, int V>
__global__ void rows_copy_kernel(View src, View dst, int accumulate, RowIter it) {
  GRID_STRIDE(idx, it.total) {
    int b, y, in;
    it.at(idx, V, b, y, in);
    float v[4], d[4];
    ldv<TS, V>((const TS *)src.p + view_off(src, b, y, in), v);
    TD *pd = (TD *)dst.p + view_off(dst, b, y, in);
    if (accumulate) {
      ldv<TD, V>(pd, d);
#pragma unroll
      for (int e = 0; e < V; ++e) v[e] += d[e];
    }
    stv<TD, V>(pd, v);
  }
}

template <typename TS, typename TD>
static void rows_copy_go(View src, View dst, int acc, RowIter it, int V, hipStream_t s) {
  const unsigned g = grid_for(it.total);
  if (V == 4) rows_copy_kernel<TS, TD, 4><<<g, 256, 0, s>>>(src, dst, acc, it);
  else rows_copy_kernel<TS, TD, 1><<<g, 256, 0, s>>>(src, dst, acc, it);
}

int launch_rows_copy(int st, int dtt, View src, View dst, int accumulate, int B,
                     int r0, int r1, int W, int C, void *stream) {
  const int V = ((long long)W * C) % 4 == 0 ? 4 : 1;
  RowIter it = row_iter(B, r0, r1, W, C, V);
  if (it.total <= 0) return 0;
  hipStream_t s = (hipStream_t)stream;
  if (st == DT_F32 && dtt == DT_F32) rows_copy_go<float, float>(src, dst, accumulate, it, V, s);
  else if (st == DT_F32) rows_copy_go<float, bf16>(src, dst, accumulate, it, V, s);
  else if (dtt == DT_F32) rows_copy_go<bf16, float>(src, dst, accumulate, it, V, s);
  else rows_copy_go<bf16, bf16>(src, dst, accumulate, it, V, s);
  return (int)hipGetLastError();
}

struct CopyBatch {
  int n;
  CopySeg seg[kMaxCopySegs];
  RowIter it[kMaxCopySegs];
  long long start[kMaxCopySegs + 1];  // first flat vector index of each segment
};

template <typename T, int V>
__global__ void rows_copy_batch_kernel(CopyBatch cb) {
  GRID_STRIDE(idx, cb.start[cb.n]) {
    int s = 0;
    while (s + 1 < cb.n && idx >= cb.start[s + 1]) ++s;
    const CopySeg &g = cb.seg[s];
    int b, y, in;
    cb.it[s].at(idx - cb.start[s], V, b, y, in);
    float v[4];
    ldv<T, V>((const T *)g.src.p + view_off(g.src, b, y, in), v);
    stv<T, V>((T *)g.dst.p + view_off(g.dst, b, y, in), v);
  }
}

int launch_rows_copy_batch(int dt, const CopySeg *segs, int n, void *stream) {
  if (n <= 0) return 0;
  if (n > kMaxCopySegs) return (int)hipErrorInvalidValue;
  CopyBatch cb{};
  int V = 4;
  for (int i = 0; i < n; ++i)
    if (((long long)segs[i].W * segs[i].C) % 4 != 0) V = 1;
  cb.n = n;
  cb.start[0] = 0;
  for (int i = 0; i < n; ++i) {
    cb.seg[i] = segs[i];
    cb.it[i] = row_iter(segs[i].B, segs[i].r0, segs[i].r1, segs[i].W, segs[i].C, V);
    cb.start[i + 1] = cb.start[i] + (cb.it[i].total > 0 ? cb.it[i].total : 0);
  }
  if (cb.start[n] <= 0) return 0;
  hipStream_t s = (hipStream_t)stream;
  const unsigned g = grid_for(cb.start[n]);
  if (dt == DT_F32) {
    if (V == 4) rows_copy_batch_kernel<float, 4><<<g, 256, 0, s>>>(cb);
    else rows_copy_batch_kernel<float, 1><<<g, 256, 0, s>>>(cb);
  } else {
    if (V == 4) rows_copy_batch_kernel<bf16, 4><<<g, 256, 0, s>>>(cb);
    else rows_copy_batch_kernel<bf16, 1><<<g, 256, 0, s>>>(cb);
  }
  return (int)hipGetLastError();
}

// Rows of a float32 error window at the start of a band: rows below t are
// zero, rows from t on are the error carried from the next band.
template <int V>
__global__ void rows_init_kernel(View dst, View carry, int t, RowIter it) {
  GRID_STRIDE(idx, it.total) {
    int b, y, in;
    it.at(idx, V, b, y, in);
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    if (y >= t) ldv<float, V>((const float *)carry.p + view_off(carry, b, y, in), v);
    stv<float, V>((float *)dst.p + view_off(dst, b, y, in), v);
  }
}

int launch_rows_init(View dst, const View *carry, int t, int B, int r0, int r1, int W, int C,
                     void *stream) {
  const int V = ((long long)W * C) % 4 == 0 ? 4 : 1;
  RowIter it = row_iter(B, r0, r1, W, C, V);
  if (it.total <= 0) return 0;
  const View cv = carry ? *carry : View{};
  if (!carry) t = r1;
  hipStream_t s = (hipStream_t)stream;
  if (V == 4) rows_init_kernel<4><<<grid_for(it.total), 256, 0, s>>>(dst, cv, t, it);
  else rows_init_kernel<1><<<grid_for(it.total), 256, 0, s>>>(dst, cv, t, it);
  return (int)hipGetLastError();
}

template <int V>
__global__ void rows_zero_kernel(View dst, RowIter it) {
  const float z[4] = {0.f, 0.f, 0.f, 0.f};
  GRID_STRIDE(idx, it.total) {
    int b, y, in;
    it.at(idx, V, b, y, in);
    stv<float, V>((float *)dst.p + view_off(dst, b, y, in), z);
  }
}

int launch_rows_zero(View dst, int B, int r0, int r1, int W, int C, void *stream) {
  const int V = ((long long)W * C) % 4 == 0 ? 4 : 1;
  RowIter it = row_iter(B, r0, r1, W, C, V);
  if (it.total <= 0) return 0;
  hipStream_t s = (hipStream_t)stream;
  if (V == 4) rows_zero_kernel<4><<<grid_for(it.total), 256, 0, s>>>(dst, it);
  else rows_zero_kernel<1><<<grid_for(it.total), 256, 0, s>>>(dst, it);
  return (int)hipGetLastError();
}

// Rows [r0, r1) of a map with C channels into a view with Cp > C channels
// (storage dtype), the extra channels zero. Gives a first layer with few
// input channels whole 16-byte vectors per pixel for its weight gradient.
template <typename T>
__global__ void pad_channels_kernel(View src, View dst, int C, int Cp, RowIter it) {
  GRID_STRIDE(idx, it.total) {
    int b, y, in;
    it.at(idx, 1, b, y, in);
    const int x = in / Cp, c = in - x * Cp;
    T v = (T)0;
    if (c < C) v = ((const T *)src.p)[view_off(src, b, y, x * C + c)];
    ((T *)dst.p)[view_off(dst, b, y, in)] = v;
  }
}

int launch_pad_channels(int dt, View src, View dst, int C, int Cp, int B, int r0, int r1,
                        int W, void *stream) {
  RowIter it = row_iter(B, r0, r1, W, Cp, 1);
  if (it.total <= 0) return 0;
  hipStream_t s = (hipStream_t)stream;
  if (dt == DT_F32)
    pad_channels_kernel<float><<<grid_for(it.total), 256, 0, s>>>(src, dst, C, Cp, it);
  else
    pad_channels_kernel<bf16><<<grid_for(it.total), 256, 0, s>>>(src, dst, C, Cp, it);
  return (int)hipGetLastError();
}

// dW [rows][C] from a channel-padded float32 [rows][Cp] (n = rows * C).
__global__ void compact_dw_kernel(const float *pad, float *dw, int C, int Cp, long long n) {
  GRID_STRIDE(i, n) {
    const long long t = i / C;
    dw[i] = pad[t * Cp + (i - t * C)];
  }
}

int launch_compact_dw(const float *pad, float *dw, int C, int Cp, long long n, void *stream) {
  if (n <= 0) return 0;
  compact_dw_kernel<<<grid_for(n), 256, 0, (hipStream_t)stream>>>(pad, dw, C, Cp, n);
  return (int)hipGetLastError();
}

__global__ void zero_kernel(float *p, long long n) {
  GRID_STRIDE(i, n) p[i] = 0.f;
}

int launch_zero_f32(float *p, size_t n, void *stream) {
  if (n == 0) return 0;
  zero_kernel<<<grid_for((long long)n), 256, 0, (hipStream_t)stream>>>(p, (long long)n);
  return (int)hipGetLastError();
}

}  // namespace lrcnn
