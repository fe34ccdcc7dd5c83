// Launchers for the gfx950 kernels of one band step. All launches are
// asynchronous on the given stream; each returns the hipError_t of the
// launch as an int (0 = success).
#pragma once

#include <cstddef>
#include <cstdint>

#if defined(__HIPCC__)
#define LRCNN_HD __host__ __device__
#else
#define LRCNN_HD
#endif

namespace lrcnn {

// Division of an unsigned 32-bit n by an invariant divisor 1 <= d < 2^31
// with one multiply-high, an add and a shift (Granlund and Montgomery,
// "Division by invariant integers using multiplication", PLDI 1994,
// Section 4): with l = ceil(log2 d) and m = floor(2^32 (2^l - d) / d) + 1,
// which fits in 32 bits, n / d = (mulhi(m, n) + n) >> l, the sum taken in
// 64 bits. The index arithmetic of the kernels uses it in place of integer
// division, whose expansion costs tens of instructions per quotient.
struct FastDiv {
  uint32_t d, m, l;
};
inline FastDiv fast_div(uint32_t d) {
  uint32_t l = 0;
  while (l < 31 && (uint32_t(1) << l) < d) ++l;
  const uint64_t m = ((uint64_t(1) << 32) * ((uint64_t(1) << l) - d)) / d + 1;
  return FastDiv{d, (uint32_t)m, l};
}
LRCNN_HD inline uint32_t fdiv_q(uint32_t n, const FastDiv &f) {
  return (uint32_t)(((((uint64_t)f.m * n) >> 32) + n) >> f.l);
}
// q = n / d and r = n % d
LRCNN_HD inline void fdiv_qr(uint32_t n, const FastDiv &f, uint32_t &q, uint32_t &r) {
  q = fdiv_q(n, f);
  r = n - q * f.d;
}

// Taps of a kh x kw kernel (at most 64 taps, kw < 64) under which an
// implicit-GEMM row whose tap-0 source position is (by, bx) reads inside
// the source window (rows [sy0, sy1), columns [0, Ws)), as bits
// tap = ti * kw + tj. Forward: source (by + ti, bx + tj). Mirrored (input
// gradient): source (by - ti, bx - tj).
LRCNN_HD inline uint64_t tap_window_mask(int by, int bx, int kh, int kw, int sy0, int sy1,
                                         int Ws, bool mirrored) {
  const int r0 = mirrored ? (by - sy1 + 1 > 0 ? by - sy1 + 1 : 0) : (sy0 - by > 0 ? sy0 - by : 0);
  const int r1 = mirrored ? (by - sy0 + 1 < kh ? by - sy0 + 1 : kh) : (sy1 - by < kh ? sy1 - by : kh);
  const int q0 = mirrored ? (bx - Ws + 1 > 0 ? bx - Ws + 1 : 0) : (-bx > 0 ? -bx : 0);
  const int q1 = mirrored ? (bx + 1 < kw ? bx + 1 : kw) : (Ws - bx < kw ? Ws - bx : kw);
  const uint64_t cm = q1 > q0 ? ((1ull << (q1 - q0)) - 1ull) << q0 : 0ull;
  uint64_t m = 0;
  for (int r = r0; r < r1; ++r) m |= cm << (r * kw);
  return m;
}

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

// Where a backward launch that completes a producer's error for the band
// puts it (fact = 1): rows >= fa, masked by ReLU of z (when relu) and
// scaled per channel by scale (nullable), go in the storage dtype to the
// producer's error operand dc; rows < fa go as float32 to carry. With
// fact = 0 the launch writes the producer's float32 error window.
struct ErrOut {
  int fact;
  View dc, z, carry;
  const float *scale;
  int relu, fa;
};

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
  int splits;         // > 0: this split count (the layer's fixed one); 0: the
                      // launcher's estimate picks it
  int kts;            // K iterations per split (set by the launcher)
  // forward only: residual add fused into the epilogue (res.p nullable):
  // the conv value (rounded to the storage dtype) plus the other input of
  // the add at the same element, then the add's ReLU when res_relu; dst and
  // mask are then the add's
  View res;
  int res_relu;
  // input gradient only: dst_init = 1 makes this launch initialize the
  // error window instead of adding to it: it writes cinit's float32 value
  // (the error carried from the next band, rows >= cinit_t, when cinit.p is
  // set; zero elsewhere) plus the gradient. The launch must cover every row
  // of the window the band uses.
  int dst_init;
  View cinit;
  int cinit_t;
  FastDiv fw, fr, fn;  // division by Wd, y1 - y0 and N (set by the launcher)
  // forward with KC channels in one vector: each K iteration covers KR taps,
  // one per 16-byte vector of a tile row (set by the launcher)
  int tpack;
  FastDiv fkw;  // division by kw
  // input gradient of a strided convolution split into phases (pst > 1,
  // set by the launcher): this launch covers the producer pixels
  // y = y0 + pst * yy (yy < y1 - y0), x = px0 + pst * xx (xx < Wd), which
  // receive exactly the taps (ty0 + pst * i, tx0 + pst * j), i < kh, j < kw,
  // of the kh_full x kw_full kernel; W is read with the full kernel's
  // strides (taps_full taps, kw_full columns)
  int pst, px0, ty0, tx0, kw_full, taps_full;
  // input gradient: where the producer's completed error goes
  ErrOut eo;
};
int launch_conv(int dt, int dgrad, const ConvArgs &a, void *stream);
// input gradients of strided convolutions on the calling thread: 0 = split
// into stride phases when estimated faster, 1 = always, 2 = never
void set_dgrad_phases(int mode);

// Split-K selection. A launch of `tiles` output tiles whose K loop has KT
// iterations runs split s ways as tiles*s workgroups of ceil(KT/s)
// iterations each, plus a pass that adds the s partial sums in a fixed
// order. The estimated duration of each choice is
//   K loop:   iterations * (workgroups on the busiest of the 256 CUs)
//             * time of one iteration, which falls when two workgroups
//             share a CU (latency hiding) and does not improve beyond
//             that;
//   fixed:    prologue, pipeline fill and epilogue of a workgroup;
//   splits:   the extra launch and the partial sums written and read back
//             (they stay in the last-level cache at these sizes).
// The constants are measured on gfx950 for the 128-row tiles of the
// kernels in kernels.hip. The count is the cheapest estimate whose partial
// sums fit in `cap` bytes; it is shared by the launchers and the planner's
// workspace sizing, so both always agree.
// Constants of the launch-duration estimates (microseconds; measured on
// gfx950 with the kernels of kernels.hip).
#ifndef LRCNN_SHARE2
#define LRCNN_SHARE2 0.8   // time factor of a workgroup sharing its CU with another
#endif
#ifndef LRCNN_STEP_N64
#define LRCNN_STEP_N64 0.75  // one K iteration of a lone 128 x 64 tile (fp32)
#endif
#ifndef LRCNN_STEP_N128
#define LRCNN_STEP_N128 1.35  // one K iteration of a lone 128 x 128 tile (fp32)
#endif
#ifndef LRCNN_NARROW_GAIN
#define LRCNN_NARROW_GAIN 1.5  // narrow tiles are taken unless wide ones are 1.5x faster
#endif
// 16-byte vectors per K iteration of a convolution launch: LRCNN_CONV_KR
// (4 or 8), and LRCNN_CONV_KR_WIN for the bfloat16 forward of windowed
// kernels (conv_kr below)
#ifndef LRCNN_CONV_KR
#define LRCNN_CONV_KR 4
#endif
#ifndef LRCNN_CONV_KR_WIN
#define LRCNN_CONV_KR_WIN 8
#endif
struct SplitCost {
  double step_us;   // one K iteration of a lone workgroup
  int occ;          // workgroups one CU holds (LDS bound)
  double fixed_us;  // per-launch fixed cost
  int max_s = 128;  // largest split count considered
  double share = LRCNN_SHARE2;  // time factor of a workgroup sharing its CU
};
struct SplitChoice {
  int s;
  double us;  // estimated duration
};
// Estimated duration of a launch of `tiles` tiles split s ways.
inline double split_cost(long long tiles, int KT, long long part_elems, const SplitCost &c,
                         long long s) {
  const long long wg = tiles * s;
  const long long per_cu = (wg + 255) / 256;
  const long long kts = (KT + s - 1) / s;
  const double share = per_cu >= 2 && c.occ >= 2 ? c.share : 1.0;
  double t = (double)kts * (double)per_cu * c.step_us * share + c.fixed_us;
  if (s > 1) t += 6.0 + (double)s * (double)part_elems * 8.0 / 1.5e7;
  return t;
}
// A split count s of a K loop of KT iterations is used only when no smaller
// count gives the same chunks (each of the s chunks has ceil(KT / s)
// iterations, the last one possibly fewer, none empty).
inline bool split_valid(int KT, long long s, int max_s = 128) {
  if (s == 1) return true;
  if (s < 1 || s > max_s || s > KT / 2) return false;
  const long long kts = (KT + s - 1) / s;
  return (KT + kts - 1) / kts == s;
}
inline SplitChoice split_choice(long long tiles, int KT, long long part_elems, size_t cap,
                                const SplitCost &c) {
  SplitChoice best{1, split_cost(tiles, KT, part_elems, c, 1)};
  if (tiles <= 0 || KT <= 1) return best;
  for (long long s = 2; s <= c.max_s && s <= KT / 2; ++s) {
    if ((size_t)s * (size_t)part_elems * 4 > cap) break;
    if (!split_valid(KT, s, c.max_s)) continue;  // same work as a smaller s
    const double t = split_cost(tiles, KT, part_elems, c, s);
    if (t < best.us * 0.98) best = SplitChoice{(int)s, t};
  }
  return best;
}
// The guard every split launch passes before it is enqueued: its partial
// sums (splits x M x N float32) fit the buffer it was given, and M x N
// indexes in 32 bits (the reduction's index arithmetic). A launch that
// fails it is refused with an error instead of writing past the buffer.
inline bool split_fits(long long splits, long long M, long long N, const void *part,
                       size_t part_bytes) {
  if (splits <= 1) return true;
  if (!part || M <= 0 || N <= 0) return false;
  if (M * N >= (1ll << 32)) return false;
  return (unsigned long long)splits * (unsigned long long)M * (unsigned long long)N * 4ull <=
         (unsigned long long)part_bytes;
}
inline int split_count(long long tiles, int KT, long long part_elems, size_t cap,
                       const SplitCost &c) {
  return split_choice(tiles, KT, part_elems, cap, c).s;
}
// Tile width and split count of a convolution launch (forward or input
// gradient, M x N outputs, KT K iterations): 128-row tiles, 64 or 128
// columns wide. Narrow tiles double the workgroup count of a launch, which
// fills the CUs better when a band gives only a few hundred 128 x 128
// tiles; the cheaper of the two estimates is taken.
struct ConvTiles {
  int bn, splits;
  double us;  // estimated duration
};
// (kr: 16-byte vectors per K iteration; an iteration of 8 costs about twice
// one of 4, and its 72 KiB LDS ring fits two 64-wide workgroups per CU;
// 8-vector launches use 64-wide tiles only)
inline ConvTiles conv_tiles(long long M, int N, int KT, size_t cap, int es,
                            int kr = LRCNN_CONV_KR) {
  const double f = (es == 2 ? 0.75 : 1.0) * kr / 4.0;
  const long long mt = (M + 127) / 128;
  SplitChoice n64 = split_choice(mt * ((N + 63) / 64), KT, M * (long long)N, cap,
                                 SplitCost{LRCNN_STEP_N64 * f, kr > 4 ? 2 : 3, 5.0});
  if (N <= 64 || kr > 4) return ConvTiles{64, n64.s, n64.us};
  SplitChoice n128 = split_choice(mt * ((N + 127) / 128), KT, M * (long long)N, cap,
                                  SplitCost{LRCNN_STEP_N128 * f, 2, 5.0});
  return n64.us < n128.us * LRCNN_NARROW_GAIN ? ConvTiles{64, n64.s, n64.us}
                                              : ConvTiles{128, n128.s, n128.us};
}
// split count of a convolution launch (the planner sizes partial sums with it)
inline int conv_split_count(long long M, int N, int KT, size_t cap, int es) {
  return conv_tiles(M, N, KT, cap, es).splits;
}
// Tile width of a convolution launch whose split count is fixed (the
// forward launches of one layer all use the layer's count, so every output
// element sums K in the same chunks whatever the band); `us` its estimate.
inline ConvTiles conv_tiles_split(long long M, int N, int KT, int s, int es,
                                  int kr = LRCNN_CONV_KR) {
  const double f = (es == 2 ? 0.75 : 1.0) * kr / 4.0;
  const long long mt = (M + 127) / 128;
  const double u64 = split_cost(mt * ((N + 63) / 64), KT, M * (long long)N,
                                SplitCost{LRCNN_STEP_N64 * f, kr > 4 ? 2 : 3, 5.0}, s);
  if (N <= 64 || kr > 4) return ConvTiles{64, s, u64};
  const double u128 = split_cost(mt * ((N + 127) / 128), KT, M * (long long)N,
                                 SplitCost{LRCNN_STEP_N128 * f, 2, 5.0}, s);
  return u64 < u128 * LRCNN_NARROW_GAIN ? ConvTiles{64, s, u64} : ConvTiles{128, s, u128};
}
// K iterations of a conv for storage element size es (bytes); one
// iteration covers kr 16-byte vectors of a tile row (LRCNN_CONV_KR, or
// LRCNN_CONV_KR_WIN for the bfloat16 forward of a windowed kernel whose
// channels fill whole vectors: twice the MFMAs per K step there).
// A forward convolution whose input channels fit in one 16-byte vector
// (kc * es < 16, e.g. a 3-channel image) packs LRCNN_CONV_KR taps into one
// iteration instead (tap_packed).
inline bool conv_tap_packed(int kc, int es, bool dgrad) { return !dgrad && kc * es < 16; }
// the 16-byte loaders (taps tested against a 64-bit mask)
inline bool conv_vec(int kh, int kw, int kc, int n, int es, bool dgrad) {
  const int E = 16 / es;
  return kc % E == 0 && (!dgrad || n % E == 0) && kh * kw <= 64 && kw < 64;
}
inline int conv_kr(int kh, int kw, int kc, int n, int es, bool dgrad) {
  return !dgrad && es == 2 && kh * kw > 1 && conv_vec(kh, kw, kc, n, es, dgrad)
             ? LRCNN_CONV_KR_WIN
             : LRCNN_CONV_KR;
}
inline int conv_k_iters(int taps, int kc, int es, bool dgrad = false,
                        int kr = LRCNN_CONV_KR) {
  if (conv_tap_packed(kc, es, dgrad)) return (taps + LRCNN_CONV_KR - 1) / LRCNN_CONV_KR;
  const int bk = 16 * kr / es;
  return taps * ((kc + bk - 1) / bk);
}

struct WgradArgs {
  const void *dc;  // error operand, own rows [B][R][Wv][Co], contiguous
  View src;        // producer window
  float *out;         // partial sums of a split launch
  size_t part_bytes;  // capacity of `out`
  int B, y0, y1, Wv, Co, Ci, Hs, Ws;
  int kh, kw, sh, sw, ph, pw;
  int overwrite;  // 1: dw = this launch's sum (the first band); 0: dw += it
  FastDiv fw, fr;  // division by Wv and by y1 - y0 (set by the launcher)
  // one K step of BK pixels as a mixed-radix (b, row, column) increment:
  // BK = wdb * (Wv * R) + wdy * Wv + wdx (set by the launcher; with Wp
  // columns per row for the row-group kernel)
  int wdx, wdy, wdb;
  // row-group kernel: rows padded to Wp = Wv rounded up to 8 columns, so an
  // aligned group of 8 pixels never spans two rows (set by the launcher)
  int Wp;
};
int launch_wgrad(int dt, const WgradArgs &a, float *dw, void *stream);
// K iterations of a weight-gradient launch over K pixels
inline int wgrad_k_iters(long long K, int es) { return (int)((K + 64 / es - 1) / (64 / es)); }
// Rows (output channels) and split count of a weight-gradient tile of a
// launch with Co x N outputs (N = taps * C_in) over K pixels: 64-row tiles
// for layers with at most 64 output channels; otherwise, in bfloat16, the
// cheaper estimate of 64- and 128-row tiles (narrow tiles give more
// workgroups when a layer has few output tiles; measured faster on the
// ResNet-50 bands), and in float32 128 rows (measured faster on VGG-16).
#ifndef LRCNN_WG_NARROW
#define LRCNN_WG_NARROW 1
#endif
// Split counts up to LRCNN_WG_MAXS are considered for the weight gradient
// (its launches have few output tiles and long K loops); LRCNN_WG_SHARE is
// its time factor for a workgroup that shares the CU.
#ifndef LRCNN_WG_MAXS
#define LRCNN_WG_MAXS 128
#endif
#ifndef LRCNN_WG_SHARE
#define LRCNN_WG_SHARE LRCNN_SHARE2
#endif
struct WgradTiles {
  int rows, splits;
};
inline WgradTiles wgrad_tiles(int Co, long long N, long long K, size_t cap, int es) {
  const double f = es == 2 ? 1.1 : 1.5;
  const int KT = wgrad_k_iters(K, es);
  const long long nt = (N + 127) / 128;
  const SplitChoice r64 = split_choice(((Co + 63) / 64) * nt, KT, (long long)Co * N, cap,
                                       SplitCost{f * 0.55, 3, 12.0, LRCNN_WG_MAXS, LRCNN_WG_SHARE});
  if (Co <= 64) return WgradTiles{64, r64.s};
  const SplitChoice r128 = split_choice(((Co + 127) / 128) * nt, KT, (long long)Co * N, cap,
                                        SplitCost{f, 3, 12.0, LRCNN_WG_MAXS, LRCNN_WG_SHARE});
  if (LRCNN_WG_NARROW && es == 2 && r64.us < r128.us) return WgradTiles{64, r64.s};
  return WgradTiles{128, r128.s};
}
inline int wgrad_split_count(int Co, long long N, long long K, size_t cap, int es) {
  return wgrad_tiles(Co, N, K, cap, es).splits;
}

struct PoolArgs {
  View src, dst;
  uint8_t *am;    // argmax of own rows [B][R][Wd][C] (nullable)
  uint8_t *mask;  // full-size argmax export (nullable)
  int mask_h;
  int B, y0, y1, Wd, C, Hs, Ws;
  int kh, kw, sh, sw, ph, pw;
  FastDiv fcv, fw, fr;  // C / V, Wd, y1 - y0 (set by the launcher)
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
  FastDiv fcv, fw, fr;  // C / V, Wu, ub - ua (set by the launcher)
  // dst_init = 1: initialize the producer's error window (the float32
  // carry from rows >= cinit_t when cinit.p is set, else zero) instead of
  // adding to it; rows [ua, ub) must be every row of the window
  int dst_init;
  View cinit;
  int cinit_t;
  ErrOut eo;  // where the completed error goes
};
int launch_pool_bwd(int dt, const PoolBwdArgs &a, void *stream);

// z = relu?(a + b) over rows [y0, y1) (storage dtype).
int launch_add_fwd(int dt, View a, View b, View z, int relu, uint8_t *mask,
                   int mask_h, int B, int y0, int y1, int W, int C,
                   void *stream);
// d = dz * [z > 0] over rows [y0, y1), sent to both inputs of the add:
// win += d (float32 window), or, when dc is set, dc = rnd(scale[c] * d)
// written contiguously over the rows (the error operand of a conv input
// without ReLU whose only consumer is the add; scale nullable, C channels).
struct AddSide {
  View win;
  void *dc;
  const float *scale;
  int C;
  // window path: init = 1 stores the initial value (the float32 carry from
  // rows >= cinit_t when cinit.p is set, else zero) plus the error instead
  // of adding to the window
  int init;
  View cinit;
  int cinit_t;
  // with init = 1: rows [y1, init_hi) of the window, above the add's rows,
  // get their initial value alone in the same launch (the window's rows
  // start at y0 and end at init_hi); 0 = none
  int init_hi;
};
int launch_add_bwd(int dt, View dz, View z, const AddSide &sa, const AddSide &sb, int relu,
                   int B, int y0, int y1, int W, int C, void *stream);
// Error operand of a conv: dc = rnd(scale[c] * dz * [z > 0]) over rows
// [y0, y1), written contiguously (storage dtype).
// `carry` (nullable): also copy rows [c0, c1) of dz (float32) into it.
int launch_act_bwd(int dt, View dz, View z, const float *scale, int relu,
                   void *dc, int B, int y0, int y1, int W, int C, void *stream,
                   const View *carry = nullptr, int c0 = 0, int c1 = 0);
// Rows [r0, r1) from src to dst with conversion (types 0 = f32, 1 = bf16);
// accumulate adds into dst.
int launch_rows_copy(int st, int dtt, View src, View dst, int accumulate,
                     int B, int r0, int r1, int W, int C, void *stream);
// Several same-dtype row copies in one launch (strips of every node of a
// band). Segments are copied independently; the caller guarantees that no
// segment's destination overlaps another segment's source or destination.
struct CopySeg {
  View src, dst;
  int B, r0, r1, W, C;
};
constexpr int kMaxCopySegs = 24;
int launch_rows_copy_batch(int dt, const CopySeg *segs, int n, void *stream);
// Rows [r0, r1) of a float32 view: zero below t, rows [t, r1) copied from
// `carry` (nullable: all zero).
int launch_rows_init(View dst, const View *carry, int t, int B, int r0, int r1, int W, int C,
                     void *stream);
// Zero rows [r0, r1) of a float32 view.
int launch_rows_zero(View dst, int B, int r0, int r1, int W, int C,
                     void *stream);
int launch_zero_f32(float *p, size_t n, void *stream);
// Rows [r0, r1) of src (C channels) into dst (Cp channels, extra ones zero).
int launch_pad_channels(int dt, View src, View dst, int C, int Cp, int B, int r0, int r1,
                        int W, void *stream);
// dw[t][c] = pad[t][c] for c < C, t over n / C rows of the padded [t][Cp].
int launch_compact_dw(const float *pad, float *dw, int C, int Cp, long long n, void *stream);

// Launch timing of the matrix-core kernels (test hook).
void profile_enable(int enable);
int profile_collect();
int profile_entry(int i, const char **name, int64_t *launches, double *ms, double *flops);
// summed algorithmic bytes and roofline times of entry i's launches
int profile_entry_roofline(int i, double *bytes, double *roof_ms);

}  // namespace lrcnn
