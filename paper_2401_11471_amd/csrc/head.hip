// Classifier head, loss and parameter update of a full training step
// (Algorithm 1: fully connected FP, Loss, fully connected BP, and the update
// of every kernel and of the fully connected weights). The trunk's output y
// ([B][H][W][C] NHWC, flattened per image to K = H*W*C features) feeds one
// fully connected layer (fc_w [n_classes][K], fc_b [n_classes], float32);
// the loss is softmax cross-entropy averaged over the batch; the update is
// plain SGD. Every reduction runs in a fixed order, so results are
// reproducible run to run.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <string>

#include "lrcnn.h"
#include "plan.hpp"

namespace lrcnn {
namespace {

constexpr int kMaxClasses = 64;
constexpr int kChunk = 8192;  // features per block of the logits pass

typedef uint16_t bf16;
__device__ __forceinline__ float ld(const float *p) { return *p; }
__device__ __forceinline__ float ld(const bf16 *p) {
  return __uint_as_float((uint32_t)(*p) << 16);
}
// float32 -> bfloat16, round to nearest, ties to even (NaN kept quiet)
__device__ __forceinline__ void st(float *p, float v) { *p = v; }
__device__ __forceinline__ void st(bf16 *p, float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) {
    *p = (bf16)((u >> 16) | 0x40u);
    return;
  }
  u += 0x7fffu + ((u >> 16) & 1u);
  *p = (bf16)(u >> 16);
}

// part[b][chunk][c] = sum over the chunk's features k of y[b, k] * fc_w[c, k]:
// each thread sums its strided features, the block's 256 sums of a class
// are then added in thread order.
template <typename T>
__global__ __launch_bounds__(256) void head_partial_kernel(const T *y, const float *fw,
                                                           long long K, int C, int chunks,
                                                           float *part) {
  __shared__ float red[kMaxClasses][257];
  const int ch = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const long long k0 = (long long)ch * kChunk;
  const long long k1 = k0 + kChunk < K ? k0 + kChunk : K;
  float acc[kMaxClasses];
#pragma unroll
  for (int c = 0; c < kMaxClasses; ++c) acc[c] = 0.f;
  const T *yb = y + (long long)b * K;
  for (long long k = k0 + tid; k < k1; k += 256) {
    const float v = ld(yb + k);
#pragma unroll
    for (int c = 0; c < kMaxClasses; ++c)
      if (c < C) acc[c] += v * fw[(long long)c * K + k];
  }
#pragma unroll
  for (int c = 0; c < kMaxClasses; ++c)
    if (c < C) red[c][tid] = acc[c];
  __syncthreads();
  if (tid < C) {
    float s = 0.f;
    for (int t = 0; t < 256; ++t) s += red[tid][t];
    part[((long long)b * chunks + ch) * C + tid] = s;
  }
}

// One block: logits, softmax, per-sample loss and dL/dlogits = (p - onehot)/B
// for every sample, then the mean loss and dL/dfc_b (sums over samples in
// sample order). A label outside [0, C) makes its loss term NaN; nothing is
// read out of bounds.
__global__ __launch_bounds__(256) void head_softmax_kernel(const float *part, int chunks,
                                                           const float *fb,
                                                           const int32_t *labels, int B,
                                                           int C, float *logits, float *dlog,
                                                           float *lossv, float *loss,
                                                           float *dfb) {
  const int tid = threadIdx.x;
  for (int b = tid; b < B; b += 256) {
    float z[kMaxClasses];
    float m = -INFINITY;
#pragma unroll
    for (int c = 0; c < kMaxClasses; ++c) {
      if (c >= C) continue;
      float s = fb[c];
      for (int ch = 0; ch < chunks; ++ch) s += part[((long long)b * chunks + ch) * C + c];
      z[c] = s;
      logits[(long long)b * C + c] = s;
      m = fmaxf(m, s);
    }
    float se = 0.f;
#pragma unroll
    for (int c = 0; c < kMaxClasses; ++c)
      if (c < C) se += expf(z[c] - m);
    const int lab = labels[b];
    const float lse = m + logf(se);
    float zl = NAN;
#pragma unroll
    for (int c = 0; c < kMaxClasses; ++c)
      if (c < C && c == lab) zl = z[c];
    lossv[b] = lse - zl;
#pragma unroll
    for (int c = 0; c < kMaxClasses; ++c)
      if (c < C)
        dlog[(long long)b * C + c] = (expf(z[c] - lse) - (c == lab ? 1.f : 0.f)) / (float)B;
  }
  __syncthreads();
  if (tid == 0) {
    float s = 0.f;
    for (int b = 0; b < B; ++b) s += lossv[b];
    *loss = s / (float)B;
  }
  if (tid < C) {
    float s = 0.f;
    for (int b = 0; b < B; ++b) s += dlog[(long long)b * C + tid];
    dfb[tid] = s;
  }
}

// dy[b, k] = sum_c dlog[b, c] * fc_w[c, k] (storage dtype)
template <typename T>
__global__ void head_dy_kernel(const float *dlog, const float *fw, long long K, int B, int C,
                               T *dy) {
  const long long total = (long long)B * K;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (long long)gridDim.x * blockDim.x) {
    const long long b = i / K, k = i - b * K;
    float s = 0.f;
    for (int c = 0; c < C; ++c) s += dlog[b * C + c] * fw[(long long)c * K + k];
    st(dy + i, s);
  }
}

// dfc_w[c, k] = sum_b dlog[b, c] * y[b, k]
template <typename T>
__global__ void head_dw_kernel(const float *dlog, const T *y, long long K, int B, int C,
                               float *dfw) {
  const long long total = (long long)C * K;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (long long)gridDim.x * blockDim.x) {
    const long long c = i / K, k = i - c * K;
    float s = 0.f;
    for (int b = 0; b < B; ++b) s += dlog[(long long)b * C + c] * ld(y + (long long)b * K + k);
    dfw[i] = s;
  }
}

// theta <- theta - lr * g, computed in float32 and stored in theta's dtype
template <typename T>
__global__ void sgd_kernel(T *w, const float *g, long long n, float lr) {
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (long long)gridDim.x * blockDim.x)
    st(w + i, ld(w + i) - lr * g[i]);
}

unsigned blocks_for(long long n) {
  long long g = (n + 255) / 256;
  if (g > 65536) g = 65536;
  return (unsigned)(g < 1 ? 1 : g);
}

struct HeadLayout {
  long long K;
  int B, chunks;
  size_t part, dlog, lossv, total;
};
HeadLayout head_layout(const Plan &P, int C) {
  HeadLayout h;
  const Shape &s = P.shp[P.n - 1];
  h.K = (long long)s.h * s.w * s.c;
  h.B = P.cfg.batch;
  h.chunks = (int)((h.K + kChunk - 1) / kChunk);
  auto a256 = [](size_t x) { return (x + 255) & ~(size_t)255; };
  h.part = 0;
  h.dlog = a256((size_t)h.B * h.chunks * C * 4);
  h.lossv = a256(h.dlog + (size_t)h.B * C * 4);
  h.total = a256(h.lossv + (size_t)h.B * 4);
  return h;
}

bool misaligned(const void *p) { return ((uintptr_t)p & 15u) != 0; }

}  // namespace
}  // namespace lrcnn

using lrcnn::Plan;

extern "C" int lrcnn_head_workspace_bytes(const lrcnn_plan_t *plan, int32_t n_classes,
                                          size_t *bytes) {
  if (!plan || !bytes) return lrcnn_fail(LRCNN_EINVAL, "null plan or output");
  if (n_classes < 1 || n_classes > lrcnn::kMaxClasses)
    return lrcnn_fail(LRCNN_EINVAL, "n_classes must be in [1, 64]");
  *bytes = lrcnn::head_layout(*reinterpret_cast<const Plan *>(plan), n_classes).total;
  return LRCNN_OK;
}

extern "C" int lrcnn_head_loss(const lrcnn_plan_t *plan, const void *y, const float *fc_w,
                               const float *fc_b, const int32_t *labels, int32_t n_classes,
                               float *logits, float *loss, void *dy, float *d_fc_w,
                               float *d_fc_b, void *head_ws, size_t head_ws_bytes,
                               void *stream) {
  using namespace lrcnn;
  if (!plan) return lrcnn_fail(LRCNN_EINVAL, "null plan");
  if (n_classes < 1 || n_classes > kMaxClasses)
    return lrcnn_fail(LRCNN_EINVAL, "n_classes must be in [1, 64]");
  const void *ptrs[] = {y, fc_w, fc_b, labels, logits, loss, dy, d_fc_w, d_fc_b, head_ws};
  for (const void *p : ptrs)
    if (!p || misaligned(p)) return lrcnn_fail(LRCNN_EINVAL, "null or misaligned head argument");
  const Plan &P = *reinterpret_cast<const Plan *>(plan);
  const HeadLayout h = head_layout(P, n_classes);
  if (head_ws_bytes < h.total)
    return lrcnn_fail(LRCNN_EWORKSPACE, "head workspace needs " + std::to_string(h.total) +
                                            " bytes, got " + std::to_string(head_ws_bytes));
  hipStream_t s = (hipStream_t)stream;
  char *ws = (char *)head_ws;
  float *part = (float *)(ws + h.part), *dlog = (float *)(ws + h.dlog),
        *lossv = (float *)(ws + h.lossv);
  const int C = n_classes;
  const bool bf = P.cfg.dtype == LRCNN_BF16;
  dim3 g1(h.chunks, h.B);
  if (bf)
    head_partial_kernel<bf16><<<g1, 256, 0, s>>>((const bf16 *)y, fc_w, h.K, C, h.chunks, part);
  else
    head_partial_kernel<float><<<g1, 256, 0, s>>>((const float *)y, fc_w, h.K, C, h.chunks,
                                                  part);
  head_softmax_kernel<<<1, 256, 0, s>>>(part, h.chunks, fc_b, labels, h.B, C, logits, dlog,
                                        lossv, loss, d_fc_b);
  const unsigned gd = blocks_for((long long)h.B * h.K), gw = blocks_for((long long)C * h.K);
  if (bf) {
    head_dy_kernel<bf16><<<gd, 256, 0, s>>>(dlog, fc_w, h.K, h.B, C, (bf16 *)dy);
    head_dw_kernel<bf16><<<gw, 256, 0, s>>>(dlog, (const bf16 *)y, h.K, h.B, C, d_fc_w);
  } else {
    head_dy_kernel<float><<<gd, 256, 0, s>>>(dlog, fc_w, h.K, h.B, C, (float *)dy);
    head_dw_kernel<float><<<gw, 256, 0, s>>>(dlog, (const float *)y, h.K, h.B, C, d_fc_w);
  }
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess)
    return lrcnn_fail(LRCNN_EHIP, std::string("head: ") + hipGetErrorString(e));
  return LRCNN_OK;
}

extern "C" int lrcnn_sgd_update(const lrcnn_plan_t *plan, float lr, void *const *w,
                                float *const *dw, float *fc_w, const float *d_fc_w,
                                float *fc_b, const float *d_fc_b, int32_t n_classes,
                                void *stream) {
  using namespace lrcnn;
  if (!plan || !w || !dw) return lrcnn_fail(LRCNN_EINVAL, "null plan or parameter array");
  const Plan &P = *reinterpret_cast<const Plan *>(plan);
  hipStream_t s = (hipStream_t)stream;
  const bool bf = P.cfg.dtype == LRCNN_BF16;
  for (int v = 1; v < P.n; ++v) {
    const lrcnn_node &d = P.nodes[v];
    if (d.op != LRCNN_OP_CONV) continue;
    if (!w[v] || !dw[v] || misaligned(w[v]) || misaligned(dw[v]))
      return lrcnn_fail(LRCNN_EINVAL, "weights or dw of node " + std::to_string(v) +
                                          " null or misaligned");
    const long long n = (long long)d.c_out * d.kh * d.kw * P.shp[d.in0].c;
    if (bf) sgd_kernel<bf16><<<blocks_for(n), 256, 0, s>>>((bf16 *)w[v], dw[v], n, lr);
    else sgd_kernel<float><<<blocks_for(n), 256, 0, s>>>((float *)w[v], dw[v], n, lr);
  }
  if (fc_w || fc_b) {
    if (!fc_w || !d_fc_w || !fc_b || !d_fc_b || n_classes < 1)
      return lrcnn_fail(LRCNN_EINVAL, "head parameters and gradients must all be given");
    const Shape &o = P.shp[P.n - 1];
    const long long nw = (long long)n_classes * o.h * o.w * o.c;
    sgd_kernel<float><<<blocks_for(nw), 256, 0, s>>>(fc_w, d_fc_w, nw, lr);
    sgd_kernel<float><<<1, 256, 0, s>>>(fc_b, d_fc_b, n_classes, lr);
  }
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess)
    return lrcnn_fail(LRCNN_EHIP, std::string("sgd: ") + hipGetErrorString(e));
  return LRCNN_OK;
}
