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

template <typename T>
struct Cfg {
  static constexpr int E = 16 / (int)sizeof(T);  // elements per 16 bytes
  static constexpr int BK = 4 * E;                // K per tile row: 64 bytes
  static constexpr int LDK = BK + E;              // LDS pitch: 80 bytes
};

constexpr int BM = 128;

// ------------------------------------------------------------------ MFMA
// One 128 x BN tile step. Wave w owns rows [wm, wm+64) and columns
// [wn, wn+BN/2); lane l feeds row/column (l & 31) of each 32x32 block and
// the K slice [KPL*(l>>5), KPL*(l>>5)+KPL) of the 64-byte tile row. The
// same slice order is used for A and B, so every MFMA adds products of
// matching K indices.
template <int BN>
__device__ __forceinline__ void mma_tile(const float *As, const float *Bs,
                                         f32x16 (&acc)[2][BN / 64], int wm,
                                         int wn, int lane) {
  constexpr int LDK = Cfg<float>::LDK, NB = BN / 64;
  const int r = lane & 31, g = lane >> 5;
  float4 a[2][2], b[NB][2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const float4 *p = (const float4 *)(As + (wm + 32 * i + r) * LDK + 8 * g);
    a[i][0] = p[0];
    a[i][1] = p[1];
  }
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const float4 *p = (const float4 *)(Bs + (wn + 32 * j + r) * LDK + 8 * g);
    b[j][0] = p[0];
    b[j][1] = p[1];
  }
#pragma unroll
  for (int s = 0; s < 8; ++s) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      float av = (s & 3) == 0 ? a[i][s >> 2].x : (s & 3) == 1 ? a[i][s >> 2].y
               : (s & 3) == 2 ? a[i][s >> 2].z : a[i][s >> 2].w;
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        float bv = (s & 3) == 0 ? b[j][s >> 2].x : (s & 3) == 1 ? b[j][s >> 2].y
                 : (s & 3) == 2 ? b[j][s >> 2].z : b[j][s >> 2].w;
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, acc[i][j], 0, 0, 0);
      }
    }
  }
}

template <int BN>
__device__ __forceinline__ void mma_tile(const bf16 *As, const bf16 *Bs,
                                         f32x16 (&acc)[2][BN / 64], int wm,
                                         int wn, int lane) {
  constexpr int LDK = Cfg<bf16>::LDK, NB = BN / 64;
  const int r = lane & 31, g = lane >> 5;
  bf16x8 a[2][2], b[NB][2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const bf16x8 *p = (const bf16x8 *)(As + (wm + 32 * i + r) * LDK + 16 * g);
    a[i][0] = p[0];
    a[i][1] = p[1];
  }
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const bf16x8 *p = (const bf16x8 *)(Bs + (wn + 32 * j + r) * LDK + 16 * g);
    b[j][0] = p[0];
    b[j][1] = p[1];
  }
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i][s], b[j][s],
                                                            acc[i][j], 0, 0, 0);
}

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

// ------------------------------------------- conv forward / input grad
template <typename T, int BN, bool DGRAD, bool VEC>
__global__ __launch_bounds__(256) void conv_gemm_kernel(ConvArgs a) {
  constexpr int E = Cfg<T>::E, BK = Cfg<T>::BK, LDK = Cfg<T>::LDK;
  constexpr int NB = BN / 64;
  __shared__ __align__(16) T As[2][BM * LDK];
  __shared__ __align__(16) T Bs[2][BN * LDK];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int R = a.y1 - a.y0;
  const int M = a.B * R * a.Wd;
  const int m0 = blockIdx.x * BM, n0 = blockIdx.y * BN;
  const int taps = a.kh * a.kw;
  const int CB = (a.KC + BK - 1) / BK;
  const int KT = taps * CB;
  const int kv = tid & 3;
  const T *src = (const T *)a.src.p;
  const T *w = (const T *)a.w;
  const long long srow = (long long)a.src.W * a.src.C;

  int ab[2], ay[2], ax[2];
  bool am[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    int m = m0 + (tid >> 2) + 64 * i;
    am[i] = m < M;
    int mm = am[i] ? m : 0;
    ax[i] = mm % a.Wd;
    int t = mm / a.Wd;
    ay[i] = a.y0 + t % R;
    ab[i] = t / R;
  }
  // B operand. Forward: B[k][n] = W[n][tap][k], contiguous along k, stored
  // as 16-byte rows. Input gradient: B[k][n] = W[k][tap][n] (k = output
  // channel of the consumer), contiguous along n, so each 16-byte load
  // holds E columns of one k and is written to LDS transposed.
  constexpr int BV = BN / E;           // 16-byte vectors per k (input grad)
  constexpr int BKS = 256 / BV;        // k rows per pass (input grad)
  int bn[NB];
  bool bvld[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    bn[j] = DGRAD ? n0 + (tid % BV) * E : n0 + (tid >> 2) + 64 * j;
    bvld[j] = bn[j] < a.N;
  }
  const int bk0 = tid / BV;

  // K iterations of this workgroup (split-K over blockIdx.z)
  const int kbeg = blockIdx.z * a.kts;
  const int kend = min(KT, kbeg + a.kts);

  uint4 ra[2], rb[NB];
  auto gload = [&](int kt) {
    const int tap = kt / CB;
    const int cb = (kt - tap * CB) * BK;
    const int c0 = cb + kv * E;
    const int ti = tap / a.kw, tj = tap - ti * a.kw;
    const bool cok = c0 < a.KC;
    const int lim = a.KC - c0;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      int sy, sx;
      bool ok;
      if (DGRAD) {
        int ty = ay[i] + a.ph - ti, tx = ax[i] + a.pw - tj;
        ok = ty >= 0 && tx >= 0;
        sy = ty / a.sh;
        sx = tx / a.sw;
        ok = ok && sy * a.sh == ty && sx * a.sw == tx;
      } else {
        sy = ay[i] * a.sh - a.ph + ti;
        sx = ax[i] * a.sw - a.pw + tj;
        ok = sx >= 0;
      }
      ok = ok && am[i] && cok && sy >= a.sy0 && sy < a.sy1 && sx < a.Ws;
      const T *p = src;
      if (ok)
        p = src + ab[i] * a.src.bs + (sy - a.src.row0) * srow +
            (long long)sx * a.src.C + c0;
      ra[i] = load16<T, VEC>(p, ok, lim);
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      if (DGRAD) {
        const int o = cb + bk0 + BKS * j;
        const bool ok = bvld[j] && o < a.KC;
        const T *p = ok ? w + ((long long)o * taps + tap) * a.N + bn[j] : w;
        rb[j] = load16<T, VEC>(p, ok, a.N - bn[j]);
      } else {
        const bool ok = bvld[j] && cok;
        const T *p = ok ? w + ((long long)bn[j] * taps + tap) * a.KC + c0 : w;
        rb[j] = load16<T, VEC>(p, ok, lim);
      }
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
  if (kend > kbeg) gload(kbeg);
  for (int kt = kbeg; kt < kend; ++kt) {
    const int buf = kt & 1;
#pragma unroll
    for (int i = 0; i < 2; ++i)
      *(uint4 *)(&As[buf][((tid >> 2) + 64 * i) * LDK + kv * E]) = ra[i];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      if (DGRAD) {
        union {
          uint4 u;
          T e[E];
        } t;
        t.u = rb[j];
#pragma unroll
        for (int e = 0; e < E; ++e)
          Bs[buf][((tid % BV) * E + e) * LDK + bk0 + BKS * j] = t.e[e];
      } else {
        *(uint4 *)(&Bs[buf][((tid >> 2) + 64 * j) * LDK + kv * E]) = rb[j];
      }
    }
    __syncthreads();
    if (kt + 1 < kend) gload(kt + 1);
    mma_tile<BN>(As[buf], Bs[buf], acc, wm, wn, lane);
  }

  if (gridDim.z > 1) {
    // split-K: raw partial sums, reduced in split order by the epilogue kernel
    float *part = a.part + (long long)blockIdx.z * M * a.N;
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
  const long long drow = (long long)a.Wd * a.N;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int m = m0 + wm + 32 * i + acc_row(v, lane);
      if (m >= M) continue;
      const int x = m % a.Wd;
      const int t = m / a.Wd;
      const int y = a.y0 + t % R;
      const int b = t / R;
      const long long off = b * a.dst.bs + (y - a.dst.row0) * drow + (long long)x * a.N;
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const int n = n0 + wn + 32 * j + col;
        if (n >= a.N) continue;
        float val = acc[i][j][v];
        if (DGRAD) {
          float *d = (float *)a.dst.p + off + n;
          *d += val;
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
template <typename T, bool DGRAD>
__global__ void conv_split_epilogue(ConvArgs a, int splits) {
  const int R = a.y1 - a.y0;
  const long long M = (long long)a.B * R * a.Wd;
  const long long MN = M * a.N;
  const long long drow = (long long)a.Wd * a.N;
  for (long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x; idx < MN;
       idx += (long long)gridDim.x * blockDim.x) {
    float val = 0.f;
    for (int z = 0; z < splits; ++z) val += a.part[z * MN + idx];
    const int n = (int)(idx % a.N);
    const long long m = idx / a.N;
    const int x = (int)(m % a.Wd);
    const long long t = m / a.Wd;
    const int y = a.y0 + (int)(t % R);
    const int b = (int)(t / R);
    const long long off = b * a.dst.bs + (y - a.dst.row0) * drow + (long long)x * a.N + n;
    if (DGRAD) {
      ((float *)a.dst.p)[off] += val;
    } else {
      if (a.scale) val = val * a.scale[n] + a.shift[n];
      if (a.relu) val = val > 0.f ? val : 0.f;
      stf((T *)a.dst.p + off, val);
      if (a.mask)
        a.mask[(((long long)b * a.mask_h + y) * a.Wd + x) * a.N + n] = val > 0.f ? 1 : 0;
    }
  }
}

static unsigned grid_for(long long total);

template <typename T, bool DGRAD>
static int conv_dispatch(const ConvArgs &a0, hipStream_t s) {
  ConvArgs a = a0;
  const int M = a.B * (a.y1 - a.y0) * a.Wd;
  if (M <= 0 || a.N <= 0) return 0;
  const bool vec = (a.KC % Cfg<T>::E) == 0 && (!DGRAD || (a.N % Cfg<T>::E) == 0);
  const int bn = a.N <= 64 ? 64 : 128;
  const int KT = a.kh * a.kw * ((a.KC + Cfg<T>::BK - 1) / Cfg<T>::BK);
  const int splits = conv_split_count(M, a.N, KT, a.part ? a.part_bytes : 0);
  a.kts = (KT + splits - 1) / splits;
  dim3 grid((M + BM - 1) / BM, (a.N + bn - 1) / bn, splits);
  int pr = -1;
  if (prof::on) {
    // algorithmic FLOPs: forward 2*M*N*K; input gradient 2 * consumer pixels
    // * C_out * taps * C_in (taps that a stride skips are not counted)
    const double taps = (double)a.kh * a.kw;
    const double fl = DGRAD ? 2.0 * a.B * (a.sy1 - a.sy0) * a.Ws * a.KC * taps * a.N
                            : 2.0 * M * a.N * taps * a.KC;
    std::string nm = std::string("conv_gemm_kernel<") + (sizeof(T) == 4 ? "float" : "bf16") +
                     ", " + std::to_string(bn) + (DGRAD ? ", dgrad" : ", fwd") +
                     (vec ? ", vec>" : ", scalar>");
    pr = prof::begin(nm, fl, s);
  }
  if (bn == 64) {
    if (vec) conv_gemm_kernel<T, 64, DGRAD, true><<<grid, 256, 0, s>>>(a);
    else conv_gemm_kernel<T, 64, DGRAD, false><<<grid, 256, 0, s>>>(a);
  } else {
    if (vec) conv_gemm_kernel<T, 128, DGRAD, true><<<grid, 256, 0, s>>>(a);
    else conv_gemm_kernel<T, 128, DGRAD, false><<<grid, 256, 0, s>>>(a);
  }
  prof::end(pr, s);
  if (splits > 1) {
    int p2 = prof::begin("conv_split_epilogue", 0.0, s);
    conv_split_epilogue<T, DGRAD><<<grid_for((long long)M * a.N), 256, 0, s>>>(a, splits);
    prof::end(p2, s);
  }
  return (int)hipGetLastError();
}

int launch_conv(int dt, int dgrad, const ConvArgs &a, void *stream) {
  hipStream_t s = (hipStream_t)stream;
  if (dt == DT_F32)
    return dgrad ? conv_dispatch<float, true>(a, s) : conv_dispatch<float, false>(a, s);
  return dgrad ? conv_dispatch<bf16, true>(a, s) : conv_dispatch<bf16, false>(a, s);
}

// ------------------------------------------------------------ weight grad
// A[m = co][k = pixel] = dc[pixel][co] and B[k = pixel][n = (tap, ci)] =
// input pixel under tap; both are K-outer in memory, so tiles are written
// to LDS transposed into the same [row][k] layout used above.
template <typename T, bool VEC>
__global__ __launch_bounds__(256) void wgrad_kernel(WgradArgs a, int kchunk,
                                                    float *dw) {
  constexpr int E = Cfg<T>::E, BK = Cfg<T>::BK, LDK = Cfg<T>::LDK;
  constexpr int BN = 128, NB = 2;
  constexpr int RV = BM / E;        // 16-byte vectors per 128-wide tile row
  constexpr int KS = 256 / RV;      // pixels loaded per pass
  __shared__ __align__(16) T As[2][BM * LDK];
  __shared__ __align__(16) T Bs[2][BN * LDK];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int R = a.y1 - a.y0;
  const int K = a.B * R * a.Wv;
  const int taps = a.kh * a.kw;
  const int N = taps * a.Ci;
  const int m0 = blockIdx.x * BM, n0 = blockIdx.y * BN;
  const int kbeg = blockIdx.z * kchunk;
  const int kend = min(K, kbeg + kchunk);
  const int rv = tid % RV, kk0 = tid / RV;
  const T *dc = (const T *)a.dc;
  const T *src = (const T *)a.src.p;
  const long long srow = (long long)a.src.W * a.src.C;

  // this thread's B columns n0 + rv*E + e: (tap, channel) of each element
  const int nb0 = n0 + rv * E;
  int tapv = nb0 / a.Ci, cv = nb0 - (nb0 / a.Ci) * a.Ci;
  const int tiv = tapv / a.kw, tjv = tapv - (tapv / a.kw) * a.kw;
  const int ov = m0 + rv * E;

  T ra[2][E], rb[2][E];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int p = k0 + kk0 + KS * i;
      const bool pk = p < kend;
      // A: E output channels of pixel p
      if (VEC) {
        uint4 u = (pk && ov < a.Co) ? *(const uint4 *)(dc + (long long)p * a.Co + ov)
                                    : make_uint4(0, 0, 0, 0);
        *(uint4 *)ra[i] = u;
      } else {
#pragma unroll
        for (int e = 0; e < E; ++e)
          ra[i][e] = (pk && ov + e < a.Co) ? dc[(long long)p * a.Co + ov + e] : (T)0;
      }
      // B: E input values of pixel p under the column's tap
      int x = 0, y = 0, b = 0;
      if (pk) {
        x = p % a.Wv;
        int t = p / a.Wv;
        y = a.y0 + t % R;
        b = t / R;
      }
      if (VEC) {
        int sy = y * a.sh - a.ph + tiv, sx = x * a.sw - a.pw + tjv;
        bool ok = pk && nb0 < N && sy >= 0 && sy < a.Hs && sx >= 0 && sx < a.Ws;
        uint4 u = make_uint4(0, 0, 0, 0);
        if (ok)
          u = *(const uint4 *)(src + b * a.src.bs + (sy - a.src.row0) * srow +
                               (long long)sx * a.src.C + cv);
        *(uint4 *)rb[i] = u;
      } else {
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const int n = nb0 + e;
          const int tap = n / a.Ci, c = n - (n / a.Ci) * a.Ci;
          const int ti = tap / a.kw, tj = tap - (tap / a.kw) * a.kw;
          const int sy = y * a.sh - a.ph + ti, sx = x * a.sw - a.pw + tj;
          const bool ok = pk && n < N && sy >= 0 && sy < a.Hs && sx >= 0 && sx < a.Ws;
          rb[i][e] = ok ? src[b * a.src.bs + (sy - a.src.row0) * srow +
                              (long long)sx * a.src.C + c]
                        : (T)0;
        }
      }
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
  const int KT = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;
  if (KT > 0) gload(kbeg);
  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int e = 0; e < E; ++e) {
        As[buf][(rv * E + e) * LDK + kk0 + KS * i] = ra[i][e];
        Bs[buf][(rv * E + e) * LDK + kk0 + KS * i] = rb[i][e];
      }
    __syncthreads();
    if (kt + 1 < KT) gload(kbeg + (kt + 1) * BK);
    mma_tile<BN>(As[buf], Bs[buf], acc, wm, wn, lane);
  }

  const int col = lane & 31;
  float *out = gridDim.z == 1 ? dw : a.out + (long long)blockIdx.z * a.Co * N;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int m = m0 + wm + 32 * i + acc_row(v, lane);
      if (m >= a.Co) continue;
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const int n = n0 + wn + 32 * j + col;
        if (n >= N) continue;
        float *d = out + (long long)m * N + n;
        if (gridDim.z == 1) *d += acc[i][j][v];
        else *d = acc[i][j][v];
      }
    }
}

// dW += sum over splits, in split order (deterministic).
__global__ void wgrad_reduce_kernel(const float *part, float *dw, long long mn,
                                    int splits) {
  long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= mn) return;
  float s = 0.f;
  for (int z = 0; z < splits; ++z) s += part[z * mn + i];
  dw[i] += s;
}

template <typename T>
static int wgrad_dispatch(const WgradArgs &a, float *dw, hipStream_t s) {
  const int K = a.B * (a.y1 - a.y0) * a.Wv;
  const int N = a.kh * a.kw * a.Ci;
  if (K <= 0) return 0;
  constexpr int BK = Cfg<T>::BK;
  int splits = a.splits < 1 ? 1 : a.splits;
  int kchunk = (K + splits - 1) / splits;
  kchunk = (kchunk + BK - 1) / BK * BK;
  splits = (K + kchunk - 1) / kchunk;
  const bool vec = (a.Co % Cfg<T>::E) == 0 && (a.Ci % Cfg<T>::E) == 0;
  dim3 grid((a.Co + BM - 1) / BM, (N + 127) / 128, splits);
  int pr = -1;
  if (prof::on)
    pr = prof::begin(std::string("wgrad_kernel<") + (sizeof(T) == 4 ? "float" : "bf16") +
                         (vec ? ", vec>" : ", scalar>"),
                     2.0 * K * a.Co * N, s);
  if (vec) wgrad_kernel<T, true><<<grid, 256, 0, s>>>(a, kchunk, dw);
  else wgrad_kernel<T, false><<<grid, 256, 0, s>>>(a, kchunk, dw);
  prof::end(pr, s);
  if (splits > 1) {
    long long mn = (long long)a.Co * N;
    int p2 = prof::begin("wgrad_reduce_kernel", 0.0, s);
    wgrad_reduce_kernel<<<(unsigned)((mn + 255) / 256), 256, 0, s>>>(a.out, dw, mn, splits);
    prof::end(p2, s);
  }
  return (int)hipGetLastError();
}

int launch_wgrad(int dt, const WgradArgs &a, float *dw, void *stream) {
  hipStream_t s = (hipStream_t)stream;
  return dt == DT_F32 ? wgrad_dispatch<float>(a, dw, s) : wgrad_dispatch<bf16>(a, dw, s);
}

// ------------------------------------------------------------- max-pool
template <typename T>
__global__ void pool_fwd_kernel(PoolArgs a) {
  const int R = a.y1 - a.y0;
  const long long total = (long long)a.B * R * a.Wd * a.C;
  const long long srow = (long long)a.src.W * a.src.C;
  const long long drow = (long long)a.Wd * a.C;
  for (long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (long long)gridDim.x * blockDim.x) {
    const int c = (int)(idx % a.C);
    long long t = idx / a.C;
    const int x = (int)(t % a.Wd);
    t /= a.Wd;
    const int yy = (int)(t % R);
    const int b = (int)(t / R);
    const int y = a.y0 + yy;
    const T *src = (const T *)a.src.p + b * a.src.bs;
    float best = 0.f;
    int bi = 0;
    for (int i = 0; i < a.kh; ++i) {
      const int sy = y * a.sh - a.ph + i;
      for (int j = 0; j < a.kw; ++j) {
        const int sx = x * a.sw - a.pw + j;
        float v = -__builtin_huge_valf();
        if (sy >= 0 && sy < a.Hs && sx >= 0 && sx < a.Ws)
          v = ldf(src + (sy - a.src.row0) * srow + (long long)sx * a.src.C + c);
        const int tp = i * a.kw + j;
        if (tp == 0 || v > best) {
          best = v;
          bi = tp;
        }
      }
    }
    T *dst = (T *)a.dst.p + b * a.dst.bs + (y - a.dst.row0) * drow + (long long)x * a.C + c;
    stf(dst, best);
    if (a.am) a.am[idx] = (uint8_t)bi;
    if (a.mask)
      a.mask[(((long long)b * a.mask_h + y) * a.Wd + x) * a.C + c] = (uint8_t)bi;
  }
}

static unsigned grid_for(long long total) {
  long long g = (total + 255) / 256;
  if (g > 65536) g = 65536;
  return (unsigned)(g < 1 ? 1 : g);
}

int launch_pool_fwd(int dt, const PoolArgs &a, void *stream) {
  const long long total = (long long)a.B * (a.y1 - a.y0) * a.Wd * a.C;
  if (total <= 0) return 0;
  hipStream_t s = (hipStream_t)stream;
  if (dt == DT_F32) pool_fwd_kernel<float><<<grid_for(total), 256, 0, s>>>(a);
  else pool_fwd_kernel<bf16><<<grid_for(total), 256, 0, s>>>(a);
  return (int)hipGetLastError();
}

__global__ void pool_bwd_kernel(PoolBwdArgs a) {
  const int Ru = a.ub - a.ua, R = a.y1 - a.y0;
  const long long total = (long long)a.B * Ru * a.Wu * a.C;
  const long long vrow = (long long)a.Wv * a.C, urow = (long long)a.Wu * a.C;
  for (long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (long long)gridDim.x * blockDim.x) {
    const int c = (int)(idx % a.C);
    long long t = idx / a.C;
    const int xi = (int)(t % a.Wu);
    t /= a.Wu;
    const int yi = a.ua + (int)(t % Ru);
    const int b = (int)(t / Ru);
    // windows y with y*sh - ph <= yi < y*sh - ph + kh, inside [y0, y1)
    const int ylo = max(a.y0, fdiv(yi + a.ph - a.kh, a.sh) + 1);
    const int yhi = min(a.y1 - 1, fdiv(yi + a.ph, a.sh));
    const int xlo = max(0, fdiv(xi + a.pw - a.kw, a.sw) + 1);
    const int xhi = min(a.Wv - 1, fdiv(xi + a.pw, a.sw));
    float sum = 0.f;
    for (int y = ylo; y <= yhi; ++y)
      for (int x = xlo; x <= xhi; ++x) {
        const int tp = (yi - (y * a.sh - a.ph)) * a.kw + (xi - (x * a.sw - a.pw));
        const long long ai = (((long long)b * R + (y - a.y0)) * a.Wv + x) * a.C + c;
        if (a.am[ai] == tp)
          sum += ((const float *)a.dv.p)[b * a.dv.bs + (y - a.dv.row0) * vrow +
                                         (long long)x * a.C + c];
      }
    float *d = (float *)a.du.p + b * a.du.bs + (yi - a.du.row0) * urow + (long long)xi * a.C + c;
    *d += sum;
  }
}

int launch_pool_bwd(const PoolBwdArgs &a, void *stream) {
  const long long total = (long long)a.B * (a.ub - a.ua) * a.Wu * a.C;
  if (total <= 0) return 0;
  pool_bwd_kernel<<<grid_for(total), 256, 0, (hipStream_t)stream>>>(a);
  return (int)hipGetLastError();
}

// ------------------------------------------------------- elementwise rows
struct RowIdx {
  long long off;  // element offset of (b, row, inner) in a view
};

__device__ __forceinline__ long long view_off(const View &v, int b, int row,
                                              int inner) {
  return b * v.bs + (long long)(row - v.row0) * v.W * v.C + inner;
}

template <typename T>
__global__ void add_fwd_kernel(View a, View bb, View z, int relu, uint8_t *mask,
                               int mask_h, int B, int y0, int y1, int W, int C) {
  const int R = y1 - y0;
  const long long inner = (long long)W * C;
  const long long total = (long long)B * R * inner;
  for (long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (long long)gridDim.x * blockDim.x) {
    const int in = (int)(idx % inner);
    const long long t = idx / inner;
    const int y = y0 + (int)(t % R);
    const int b = (int)(t / R);
    float v = ldf((const T *)a.p + view_off(a, b, y, in)) +
              ldf((const T *)bb.p + view_off(bb, b, y, in));
    if (relu) v = v > 0.f ? v : 0.f;
    stf((T *)z.p + view_off(z, b, y, in), v);
    if (mask) mask[((long long)b * mask_h + y) * inner + in] = v > 0.f ? 1 : 0;
  }
}

int launch_add_fwd(int dt, View a, View b, View z, int relu, uint8_t *mask,
                   int mask_h, int B, int y0, int y1, int W, int C, void *stream) {
  const long long total = (long long)B * (y1 - y0) * W * C;
  if (total <= 0) return 0;
  hipStream_t s = (hipStream_t)stream;
  if (dt == DT_F32)
    add_fwd_kernel<float><<<grid_for(total), 256, 0, s>>>(a, b, z, relu, mask, mask_h, B, y0, y1, W, C);
  else
    add_fwd_kernel<bf16><<<grid_for(total), 256, 0, s>>>(a, b, z, relu, mask, mask_h, B, y0, y1, W, C);
  return (int)hipGetLastError();
}

template <typename T>
__global__ void add_bwd_kernel(View dz, View z, View da, View db, int relu, int B,
                               int y0, int y1, int W, int C) {
  const int R = y1 - y0;
  const long long inner = (long long)W * C;
  const long long total = (long long)B * R * inner;
  for (long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (long long)gridDim.x * blockDim.x) {
    const int in = (int)(idx % inner);
    const long long t = idx / inner;
    const int y = y0 + (int)(t % R);
    const int b = (int)(t / R);
    float d = ((const float *)dz.p)[view_off(dz, b, y, in)];
    if (relu && !(ldf((const T *)z.p + view_off(z, b, y, in)) > 0.f)) d = 0.f;
    ((float *)da.p)[view_off(da, b, y, in)] += d;
    ((float *)db.p)[view_off(db, b, y, in)] += d;
  }
}

int launch_add_bwd(int dt, View dz, View z, View da, View db, int relu, int B,
                   int y0, int y1, int W, int C, void *stream) {
  const long long total = (long long)B * (y1 - y0) * W * C;
  if (total <= 0) return 0;
  hipStream_t s = (hipStream_t)stream;
  if (dt == DT_F32)
    add_bwd_kernel<float><<<grid_for(total), 256, 0, s>>>(dz, z, da, db, relu, B, y0, y1, W, C);
  else
    add_bwd_kernel<bf16><<<grid_for(total), 256, 0, s>>>(dz, z, da, db, relu, B, y0, y1, W, C);
  return (int)hipGetLastError();
}

template <typename T>
__global__ void act_bwd_kernel(View dz, View z, const float *scale, int relu,
                               T *dc, int B, int y0, int y1, int W, int C) {
  const int R = y1 - y0;
  const long long inner = (long long)W * C;
  const long long total = (long long)B * R * inner;
  for (long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (long long)gridDim.x * blockDim.x) {
    const int in = (int)(idx % inner);
    const long long t = idx / inner;
    const int y = y0 + (int)(t % R);
    const int b = (int)(t / R);
    float d = ((const float *)dz.p)[view_off(dz, b, y, in)];
    if (relu && !(ldf((const T *)z.p + view_off(z, b, y, in)) > 0.f)) d = 0.f;
    if (scale) d *= scale[in % C];
    stf(dc + idx, d);
  }
}

int launch_act_bwd(int dt, View dz, View z, const float *scale, int relu,
                   void *dc, int B, int y0, int y1, int W, int C, void *stream) {
  const long long total = (long long)B * (y1 - y0) * W * C;
  if (total <= 0) return 0;
  hipStream_t s = (hipStream_t)stream;
  if (dt == DT_F32)
    act_bwd_kernel<float><<<grid_for(total), 256, 0, s>>>(dz, z, scale, relu, (float *)dc, B, y0, y1, W, C);
  else
    act_bwd_kernel<bf16><<<grid_for(total), 256, 0, s>>>(dz, z, scale, relu, (bf16 *)dc, B, y0, y1, W, C);
  return (int)hipGetLastError();
}

template <typename TS, typename TD>
__global__ void rows_copy_kernel(View src, View dst, int accumulate, int B,
                                 int r0, int r1, int W, int C) {
  const int R = r1 - r0;
  const long long inner = (long long)W * C;
  const long long total = (long long)B * R * inner;
  for (long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (long long)gridDim.x * blockDim.x) {
    const int in = (int)(idx % inner);
    const long long t = idx / inner;
    const int y = r0 + (int)(t % R);
    const int b = (int)(t / R);
    float v = ldf((const TS *)src.p + view_off(src, b, y, in));
    TD *d = (TD *)dst.p + view_off(dst, b, y, in);
    if (accumulate) v += ldf(d);
    stf(d, v);
  }
}

int launch_rows_copy(int st, int dtt, View src, View dst, int accumulate, int B,
                     int r0, int r1, int W, int C, void *stream) {
  const long long total = (long long)B * (r1 - r0) * W * C;
  if (total <= 0) return 0;
  hipStream_t s = (hipStream_t)stream;
  unsigned g = grid_for(total);
  if (st == DT_F32 && dtt == DT_F32)
    rows_copy_kernel<float, float><<<g, 256, 0, s>>>(src, dst, accumulate, B, r0, r1, W, C);
  else if (st == DT_F32)
    rows_copy_kernel<float, bf16><<<g, 256, 0, s>>>(src, dst, accumulate, B, r0, r1, W, C);
  else if (dtt == DT_F32)
    rows_copy_kernel<bf16, float><<<g, 256, 0, s>>>(src, dst, accumulate, B, r0, r1, W, C);
  else
    rows_copy_kernel<bf16, bf16><<<g, 256, 0, s>>>(src, dst, accumulate, B, r0, r1, W, C);
  return (int)hipGetLastError();
}

__global__ void rows_zero_kernel(View dst, int B, int r0, int r1, int W, int C) {
  const int R = r1 - r0;
  const long long inner = (long long)W * C;
  const long long total = (long long)B * R * inner;
  for (long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (long long)gridDim.x * blockDim.x) {
    const int in = (int)(idx % inner);
    const long long t = idx / inner;
    const int y = r0 + (int)(t % R);
    const int b = (int)(t / R);
    ((float *)dst.p)[view_off(dst, b, y, in)] = 0.f;
  }
}

int launch_rows_zero(View dst, int B, int r0, int r1, int W, int C, void *stream) {
  const long long total = (long long)B * (r1 - r0) * W * C;
  if (total <= 0) return 0;
  rows_zero_kernel<<<grid_for(total), 256, 0, (hipStream_t)stream>>>(dst, B, r0, r1, W, C);
  return (int)hipGetLastError();
}

__global__ void zero_kernel(float *p, long long n) {
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (long long)gridDim.x * blockDim.x)
    p[i] = 0.f;
}

int launch_zero_f32(float *p, size_t n, void *stream) {
  if (n == 0) return 0;
  zero_kernel<<<grid_for((long long)n), 256, 0, (hipStream_t)stream>>>(p, (long long)n);
  return (int)hipGetLastError();
}

}  // namespace lrcnn
