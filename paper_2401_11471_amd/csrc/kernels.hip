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
//
// This file: launch timing, the convolution dispatch and the pooling and
// row kernels; the convolution kernels are in kconv.hpp (conv_*.hip), the
// weight gradient in wgrad.hip, the shared device helpers in kdev.hpp.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <map>
#include <string>
#include <algorithm>
#include <vector>

#include "kdev.hpp"

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
  double flops, bytes, roof_ms;
};
bool on = false;
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
// Roofline time of a launch on MI355X: the larger of its FLOPs at the dense
// matrix-core peak of its storage type (bf16 2.5 PFLOP/s, fp32 157.3
// TFLOP/s) and its algorithmic bytes at the HBM3E peak (8 TB/s).
int begin(const std::string &name, double flops, hipStream_t, double bytes, int es) {
  if (!on) return -1;
  hipEvent_t a = take(), b = take();
  if (!a || !b) return -1;
  const double peak = es == 2 ? 2.5e15 : es == 4 ? 157.3e12 : 0.0;
  const double roof_ms = 1e3 * std::max(peak > 0 ? flops / peak : 0.0, bytes / 8e12);
  recs.push_back(Rec{name, a, b, flops, bytes, roof_ms});
  return (int)recs.size() - 1;
}
hipEvent_t start(int i) { return recs[i].a; }
hipEvent_t stop(int i) { return recs[i].b; }
struct Agg {
  int64_t launches = 0;
  double ms = 0, flops = 0, bytes = 0, roof_ms = 0;
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
    g.bytes += r.bytes;
    g.roof_ms += r.roof_ms;
  }
  prof::table.assign(m.begin(), m.end());
  return (int)prof::table.size();
}

int profile_entry_roofline(int i, double *bytes, double *roof_ms) {
  if (i < 0 || i >= (int)prof::table.size()) return -1;
  *bytes = prof::table[i].second.bytes;
  *roof_ms = prof::table[i].second.roof_ms;
  return 0;
}

int profile_entry(int i, const char **name, int64_t *launches, double *ms, double *flops) {
  if (i < 0 || i >= (int)prof::table.size()) return -1;
  *name = prof::table[i].first.c_str();
  *launches = prof::table[i].second.launches;
  *ms = prof::table[i].second.ms;
  *flops = prof::table[i].second.flops;
  return 0;
}

thread_local int g_phases = 0;  // 0: by estimate, 1: always, 2: never
void set_dgrad_phases(int mode) { g_phases = mode; }

int launch_conv(int dt, int dgrad, const ConvArgs &a, void *stream) {
  hipStream_t s = (hipStream_t)stream;
  if (dt == DT_F32) return dgrad ? launch_conv_f32_dgrad(a, s) : launch_conv_f32_fwd(a, s);
  return dgrad ? launch_conv_bf16_dgrad(a, s) : launch_conv_bf16_fwd(a, s);
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

// A window row above the add's rows: its initial value (carry or zero).
template <int V>
__device__ __forceinline__ void add_init_row(const AddSide &sd, const RowIter &e, long long j) {
  int b, y, in;
  e.at(j, V, b, y, in);
  float x[4] = {0.f, 0.f, 0.f, 0.f};
  float *p = (float *)sd.win.p + view_off(sd.win, b, y, in);
  const float *bp = err_base(1, sd.cinit, sd.cinit_t, b, y, in, p);
  if (bp) ldv<float, V>(bp, x);
  stv<float, V>(p, x);
}

template <typename T, int V>
__global__ void add_bwd_kernel(View dz, View z, AddSide sa, AddSide sb, int relu, RowIter it,
                               RowIter ea, RowIter eb) {
  GRID_STRIDE(idx, it.total + ea.total + eb.total) {
    int b, y, in;
    if (idx >= it.total) {
      const long long j = idx - it.total;
      if (j < ea.total) add_init_row<V>(sa, ea, j);
      else add_init_row<V>(sb, eb, j - ea.total);
      continue;
    }
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
  // initialised rows above the add's rows: window sides with init only
  for (const AddSide *sd : {&sa, &sb})
    if (sd->init_hi > y1 && (!sd->init || sd->dc)) return (int)hipErrorInvalidValue;
  const RowIter ea = row_iter(B, y1, std::max(y1, sa.init_hi), W, C, V);
  const RowIter eb = row_iter(B, y1, std::max(y1, sb.init_hi), W, C, V);
  hipStream_t s = (hipStream_t)stream;
  const unsigned g = grid_for(it.total + ea.total + eb.total);
  if (dt == DT_F32) {
    if (V == 4) add_bwd_kernel<float, 4><<<g, 256, 0, s>>>(dz, z, sa, sb, relu, it, ea, eb);
    else add_bwd_kernel<float, 1><<<g, 256, 0, s>>>(dz, z, sa, sb, relu, it, ea, eb);
  } else {
    if (V == 4) add_bwd_kernel<bf16, 4><<<g, 256, 0, s>>>(dz, z, sa, sb, relu, it, ea, eb);
    else add_bwd_kernel<bf16, 1><<<g, 256, 0, s>>>(dz, z, sa, sb, relu, it, ea, eb);
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

// The same copy in whole 16-byte vectors (storage dtype unchanged, every
// row and view base 16-byte aligned): one load and one store per thread.
template <typename T>
__global__ void rows_copy_batch16_kernel(CopyBatch cb) {
  constexpr int V = 16 / (int)sizeof(T);
  GRID_STRIDE(idx, cb.start[cb.n]) {
    int s = 0;
    while (s + 1 < cb.n && idx >= cb.start[s + 1]) ++s;
    const CopySeg &g = cb.seg[s];
    int b, y, in;
    cb.it[s].at(idx - cb.start[s], V, b, y, in);
    *(uint4 *)((T *)g.dst.p + view_off(g.dst, b, y, in)) =
        *(const uint4 *)((const T *)g.src.p + view_off(g.src, b, y, in));
  }
}

int launch_rows_copy_batch(int dt, const CopySeg *segs, int n, void *stream) {
  if (n <= 0) return 0;
  if (n > kMaxCopySegs) return (int)hipErrorInvalidValue;
  CopyBatch cb{};
  // 16-byte vectors when every row holds whole vectors and every view base
  // is 16-byte aligned, else 4 or 1 elements per thread
  const int V16 = dt == DT_F32 ? 4 : 8;
  bool wide = true;
  for (int i = 0; i < n; ++i)
    wide = wide && ((long long)segs[i].W * segs[i].C) % V16 == 0 &&
           segs[i].src.bs % V16 == 0 && segs[i].dst.bs % V16 == 0 &&
           ((uintptr_t)segs[i].src.p & 15) == 0 && ((uintptr_t)segs[i].dst.p & 15) == 0;
  int V = wide ? V16 : 4;
  for (int i = 0; i < n && !wide; ++i)
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
    if (wide) rows_copy_batch16_kernel<float><<<g, 256, 0, s>>>(cb);
    else if (V == 4) rows_copy_batch_kernel<float, 4><<<g, 256, 0, s>>>(cb);
    else rows_copy_batch_kernel<float, 1><<<g, 256, 0, s>>>(cb);
  } else {
    if (wide) rows_copy_batch16_kernel<bf16><<<g, 256, 0, s>>>(cb);
    else if (V == 4) rows_copy_batch_kernel<bf16, 4><<<g, 256, 0, s>>>(cb);
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

// One pixel per thread when the padded pixel is one 16-byte vector (bf16
// with 8 channels, float32 with 4): C loads and one 16-byte store.
template <typename T>
__global__ void pad_channels16_kernel(View src, View dst, int C, RowIter it) {
  constexpr int CP = 16 / (int)sizeof(T);
  GRID_STRIDE(idx, it.total) {
    int b, y, in;
    it.at(idx, CP, b, y, in);
    const int x = in / CP;
    union {
      uint4 u;
      T e[CP];
    } v;
    const T *sp = (const T *)src.p + view_off(src, b, y, x * C);
#pragma unroll
    for (int c = 0; c < CP; ++c) v.e[c] = c < C ? sp[c] : (T)0;
    *(uint4 *)((T *)dst.p + view_off(dst, b, y, in)) = v.u;
  }
}

int launch_pad_channels(int dt, View src, View dst, int C, int Cp, int B, int r0, int r1,
                        int W, void *stream) {
  hipStream_t s = (hipStream_t)stream;
  if (Cp * (dt == DT_F32 ? 4 : 2) == 16 && C <= Cp && dst.bs % Cp == 0 &&
      ((uintptr_t)dst.p & 15) == 0) {
    RowIter iv = row_iter(B, r0, r1, W, Cp, Cp);
    if (iv.total <= 0) return 0;
    if (dt == DT_F32)
      pad_channels16_kernel<float><<<grid_for(iv.total), 256, 0, s>>>(src, dst, C, iv);
    else
      pad_channels16_kernel<bf16><<<grid_for(iv.total), 256, 0, s>>>(src, dst, C, iv);
    return (int)hipGetLastError();
  }
  RowIter it = row_iter(B, r0, r1, W, Cp, 1);
  if (it.total <= 0) return 0;
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
