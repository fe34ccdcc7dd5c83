// Launchers for the gfx950 kernels of one band step. All launches are
// asynchronous on the given stream; each returns the hipError_t of the
// launch as an int (0 = success).
#pragma once

#include <cstddef>
#include <cstdint>

namespace lrcnn {

// A band window of an NHWC feature map: element (b, y, x, c) of the global
// map lives at p + b*bs + (y - row0)*W*C + x*C + c, for the rows the buffer
// holds. Strides are in elements of the buffer's type.
struct View {
  void *p;
  long long bs;
  int row0;
  int W, C;
  int rows;  // rows held: [row0, row0 + rows); checked on the host only
};

enum Dt { DT_F32 = 0, DT_BF16 = 1 };

// Conv forward over rows [y0, y1) of the output, or (dgrad = 1) the input
// gradient over rows [y0, y1) of the producer from the consumer rows
// [sy0, sy1). See kernels.hip for the operand conventions.
struct ConvArgs {
  View src, dst;
  const void *w;
  const float *scale, *shift;
  int relu;
  uint8_t *mask;  // FWD: optional full-size [B][H][W][C] ReLU mask
  int mask_h;
  int B, y0, y1, Wd, N, KC, Hs, Ws, sy0, sy1;
  int kh, kw, sh, sw, ph, pw;
  float *part;        // split-K partial sums (nullable: no split)
  size_t part_bytes;  // capacity of `part`
  int kts;            // K iterations per split (set by the launcher)
};
int launch_conv(int dt, int dgrad, const ConvArgs &a, void *stream);

// Number of K splits of a conv launch with M x N outputs and KT K-iterations:
// enough workgroups for two per CU when the output tiles alone are too few,
// at least 8 K-iterations per split, and partial sums that fit in `cap`
// bytes. Shared by the launcher and the planner's workspace sizing.
inline int conv_split_count(long long M, int N, int KT, size_t cap) {
  const long long bn = N <= 64 ? 64 : 128;
  const long long tiles = ((M + 127) / 128) * ((N + bn - 1) / bn);
  const long long cus = 256;
  if (tiles >= 2 * cus || KT < 16) return 1;
  const long long per = M * (long long)N * 4;
  // score: balance over the CUs (every CU gets the same number of
  // workgroups), enough workgroups for two per CU, a small charge per
  // split for the partial sums
  auto score = [&](long long s) {
    const long long wg = tiles * s;
    const double bal = (double)wg / (double)(cus * ((wg + cus - 1) / cus));
    const double fill = wg >= 2 * cus ? 1.0 : (double)wg / (2.0 * cus);
    return bal * fill - 0.01 * (double)(s - 1);
  };
  long long best = 1;
  double bs = score(1);
  for (long long s = 2; s <= KT / 8 && s <= 64; ++s) {
    if (per > 0 && s * per > (long long)cap) break;
    const double sc = score(s);
    if (sc > bs + 1e-9) {
      bs = sc;
      best = s;
    }
  }
  const long long kts = (KT + best - 1) / best;
  return (int)((KT + kts - 1) / kts);
}
// K iterations of a conv for storage element size es (bytes); one
// iteration covers LRCNN_CONV_KR 16-byte vectors of a tile row.
#ifndef LRCNN_CONV_KR
#define LRCNN_CONV_KR 4
#endif
inline int conv_k_iters(int taps, int kc, int es) {
  const int bk = 16 * LRCNN_CONV_KR / es;
  return taps * ((kc + bk - 1) / bk);
}

struct WgradArgs {
  const void *dc;  // error operand, own rows [B][R][Wv][Co], contiguous
  View src;        // producer window
  float *out;      // dW [Co][kh*kw*Ci] (split == 1) or partial sums
  int splits;
  int B, y0, y1, Wv, Co, Ci, Hs, Ws;
  int kh, kw, sh, sw, ph, pw;
};
int launch_wgrad(int dt, const WgradArgs &a, float *dw, void *stream);

struct PoolArgs {
  View src, dst;
  uint8_t *am;    // argmax of own rows [B][R][Wd][C] (nullable)
  uint8_t *mask;  // full-size argmax export (nullable)
  int mask_h;
  int B, y0, y1, Wd, C, Hs, Ws;
  int kh, kw, sh, sw, ph, pw;
};
int launch_pool_fwd(int dt, const PoolArgs &a, void *stream);

// Gather form of the max-pool backward: producer rows [ua, ub) of the
// float32 error window `du` receive the consumer error `dv` (float32 window)
// routed through `am` (argmax of consumer rows [y0, y1)).
struct PoolBwdArgs {
  View dv, du;
  const uint8_t *am;
  int B, y0, y1, Wv, C, ua, ub, Wu;
  int kh, kw, sh, sw, ph, pw;
};
int launch_pool_bwd(const PoolBwdArgs &a, void *stream);

// z = relu?(a + b) over rows [y0, y1) (storage dtype).
int launch_add_fwd(int dt, View a, View b, View z, int relu, uint8_t *mask,
                   int mask_h, int B, int y0, int y1, int W, int C,
                   void *stream);
// d = dz * [z > 0]; da += d; db += d (float32 windows) over rows [y0, y1).
int launch_add_bwd(int dt, View dz, View z, View da, View db, int relu, int B,
                   int y0, int y1, int W, int C, void *stream);
// Error operand of a conv: dc = rnd(scale[c] * dz * [z > 0]) over rows
// [y0, y1), written contiguously (storage dtype).
int launch_act_bwd(int dt, View dz, View z, const float *scale, int relu,
                   void *dc, int B, int y0, int y1, int W, int C, void *stream);
// Rows [r0, r1) from src to dst with conversion (types 0 = f32, 1 = bf16);
// accumulate adds into dst.
int launch_rows_copy(int st, int dtt, View src, View dst, int accumulate,
                     int B, int r0, int r1, int W, int C, void *stream);
// Zero rows [r0, r1) of a float32 view.
int launch_rows_zero(View dst, int B, int r0, int r1, int W, int C,
                     void *stream);
int launch_zero_f32(float *p, size_t n, void *stream);

// Launch timing of the matrix-core kernels (test hook).
void profile_enable(int enable);
int profile_collect();
int profile_entry(int i, const char **name, int64_t *launches, double *ms, double *flops);

}  // namespace lrcnn
