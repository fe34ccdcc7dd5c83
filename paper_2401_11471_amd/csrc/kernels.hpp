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
};
int launch_conv(int dt, int dgrad, const ConvArgs &a, void *stream);

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
// W[co][t][ci] -> Wt[t][ci][co]
int launch_wtranspose(int dt, const void *w, void *wt, int co, int taps,
                      int ci, void *stream);

}  // namespace lrcnn
