// Weight-gradient kernel and its fixed-order split-K reduction.
#include "kdev.hpp"

namespace lrcnn {

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
// K steps of KRW 16-byte vectors per tile row (BK = KRW * E pixels): 4, or
// 8 for bfloat16 tiles with vector channel counts (twice the MFMAs per
// barrier and per fragment prefetch).
#ifndef LRCNN_WG_KR
#define LRCNN_WG_KR 4
#endif
// Epilogue of a weight-gradient tile: the wave's 64 x 32 NB accumulators
// (rows m0 + [0, 64), columns n0 + [0, 32 NB)) go to dW (one split: dW =
// or += the sum) or to the split's partial-sum slice.
template <int NB>
__device__ __forceinline__ void wgrad_store(const WgradArgs &a, float *dw,
                                            const f32x16 (&acc)[2][NB], int m0, int n0,
                                            int N, int z, int lane) {
  const int col = lane & 31;
  float *out = gridDim.z == 1 ? dw : a.out + (long long)z * a.Co * N;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int m = m0 + 32 * i + acc_row(v, lane);
      if (m >= a.Co) continue;
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const int nn = n0 + 32 * j + col;
        if (nn >= N) continue;
        float *d = out + (long long)m * N + nn;
        if (gridDim.z == 1) *d = a.overwrite ? acc[i][j][v] : *d + acc[i][j][v];
        else *d = acc[i][j][v];
      }
    }
}

template <typename T, int WBM, bool AVEC, bool BVEC, int KRW = 4>
__global__ __launch_bounds__(256, LRCNN_WG_OCC) void wgrad_kernel(WgradArgs a, int kchunk,
                                                    float *dw) {
  static_assert(KRW == 4 || (KRW == 8 && BVEC && AVEC), "K step");
  constexpr int E = Cfg<T>::E, BK = KRW * E;
  constexpr int BN = 128;
  constexpr int FBN = WBM == 128 ? 128 : 64;  // columns per wave: FBN / 2
  constexpr int NB = FBN / 64;
  constexpr int RV = BN / E;        // 16-byte vectors per B tile row
  constexpr int KS = 256 / RV;      // pixels of B loaded per pass
  constexpr int RVA = WBM / E;      // 16-byte vectors per A tile row
  constexpr int KSA = 256 / RVA;    // pixels of A loaded per pass
  constexpr int NPA = BK / KSA;     // A passes per tile
  constexpr int ASZ = BK * KM<T, WBM>::P, BSZ = BK * KM<T, BN>::P;
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
  constexpr int RVH = RV / 2;
  constexpr int NPB = BVEC ? BK / (256 / RVH) : 1;  // B pixel passes (vector path)
  V16 ra[NPA], rb[2 * NPB];
  int k0 = kbeg;
  // B with channel counts that are multiples of E: thread (kkb, rvb)
  // loads pixel k0 + kkb under column vectors rvb and rvb + RV / 2, so one
  // pixel position per thread is walked from K step to K step (a
  // mixed-radix increment, no division in the loop); the taps' offsets in
  // the source window are fixed per thread
  const int kkb = tid / RVH, rvb = tid % RVH;
  // walk state of pixels k0 + kkb + (256 / RVH) * i: column wx and band row
  // wy, the source row / column under tap (0, 0) (ybase, xbase) and the
  // byte offset of that source position (poff); a K step adds uniform
  // deltas, with the column and row carries selecting the wrap corrections
  int wx[NPB], wy[NPB], ybase[NPB], xbase[NPB];
  long long poff[NPB];
  int bti[2], btj[2];
  long long btoff[2];
  bool bnok[2];
  constexpr long long ES = sizeof(T);
  const int dxb = a.wdx * a.sw, wxb = a.Wv * a.sw;
  const int dyb = a.wdy * a.sh, ryb = R * a.sh;
  const long long pd0 =
      ((long long)a.wdb * a.src.bs + (long long)dyb * srow + (long long)dxb * a.src.C) * ES;
  const long long pd1 = ((long long)a.sh * srow - (long long)wxb * a.src.C) * ES;
  const long long pd2 = (a.src.bs - (long long)ryb * srow) * ES;
  if (BVEC) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int nb = n0 + (rvb + RVH * h) * E;
      const int tap = nb / a.Ci;
      const int c = nb - tap * a.Ci;
      bti[h] = tap / a.kw;
      btj[h] = tap - bti[h] * a.kw;
      bnok[h] = nb < N;
      btoff[h] = ((long long)bti[h] * srow + (long long)btj[h] * a.src.C + c) * ES;
    }
#pragma unroll
    for (int i = 0; i < NPB; ++i) {
      uint32_t t, x, yy, b;
      fdiv_qr((uint32_t)(kbeg + kkb + (256 / RVH) * i), a.fw, t, x);
      fdiv_qr(t, a.fr, b, yy);
      wx[i] = (int)x, wy[i] = (int)yy;
      ybase[i] = (a.y0 + wy[i]) * a.sh - a.ph;
      xbase[i] = wx[i] * a.sw - a.pw;
      poff[i] = ((long long)b * a.src.bs + (long long)(ybase[i] - a.src.row0) * srow +
                 (long long)xbase[i] * a.src.C) * ES;
    }
  }
  // A: byte offsets of this thread's pixels, advanced by BK pixels a step
  long long aoff[NPA];
#pragma unroll
  for (int i = 0; i < NPA; ++i)
    aoff[i] = ((long long)(kbeg + kka0 + KSA * i) * a.Co + ov) * ES;
  const long long adk = (long long)BK * a.Co * ES;
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
        ra[i].u = load16z(dc, aoff[i], pk & ovok);
        aoff[i] += adk;
      } else {
#pragma unroll
        for (int e = 0; e < E; ++e)
          ra[i].e[e] = (pk && ov + e < a.Co) ? dc[(long long)p * a.Co + ov + e] : (T)0;
      }
    }
    if (BVEC) {
#pragma unroll
      for (int i = 0; i < NPB; ++i) {
        // B: E input values of pixel p under each of the thread's two taps
        const int p = k0 + kkb + (256 / RVH) * i;
        const bool pk = p < kend;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int sy = ybase[i] + bti[h], sx = xbase[i] + btj[h];
          const bool ok = pk & bnok[h] & (sy >= 0) & (sy < a.Hs) & (sx >= 0) & (sx < a.Ws);
          rb[2 * i + h].u = load16z(src, poff[i] + btoff[h], ok);
        }
        // next K step: pixel + BK
        wx[i] += a.wdx;
        const bool cx = wx[i] >= a.Wv;
        wx[i] -= cx ? a.Wv : 0;
        xbase[i] += dxb - (cx ? wxb : 0);
        wy[i] += a.wdy + (cx ? 1 : 0);
        const bool cy = wy[i] >= R;
        wy[i] -= cy ? R : 0;
        ybase[i] += dyb + (cx ? a.sh : 0) - (cy ? ryb : 0);
        poff[i] += pd0 + (pd1 & -(long long)cx) + (pd2 & -(long long)cy);
      }
    }
#pragma unroll
    for (int i = 0; i < 2 && !BVEC; ++i) {
      // B: E input values of pixel p under the column's tap
      const int p = k0 + kk0 + KS * i;
      const bool pk = p < kend;
      uint32_t t, x, yy, b;
      fdiv_qr((uint32_t)(pk ? p : 0), a.fw, t, x);
      fdiv_qr(t, a.fr, b, yy);
      const int y = a.y0 + (int)yy;
      {
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
      *(uint4 *)(&As[st][KM<T, WBM>::off(kka0 + KSA * i, rva * E)]) = ra[i].u;
    if (BVEC) {
#pragma unroll
      for (int i = 0; i < NPB; ++i)
#pragma unroll
        for (int h = 0; h < 2; ++h)
          *(uint4 *)(&Bs[st][KM<T, BN>::off(kkb + (256 / RVH) * i, (rvb + RVH * h) * E)]) =
              rb[2 * i + h].u;
    } else {
#pragma unroll
      for (int i = 0; i < 2; ++i)
        *(uint4 *)(&Bs[st][KM<T, BN>::off(kk0 + KS * i, rv * E)]) = rb[i].u;
    }
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
  using FR = Frag<T, FBN, KRW, 1, 1, WBM, BN>;
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
    interleave_step<FR::NMFMA, FR::NDSR, NPA + 2 * NPB, NPA + 2 * NPB>();
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

  wgrad_store<NB>(a, dw, acc, m0 + wm, n0 + wn, N, tl.z, lane);
}

// bfloat16 with channel counts that are multiples of 8: both operands are
// copied from global memory straight into the LDS ring
// (global_load_lds_dwordx4), so the tiles t+2 .. t+ST-1 are in flight while
// tile t is multiplied, no wave writes LDS and no registers stage the
// operands. A copy instruction of a wave fills 1 KiB of one k-major tile in
// lane order: 1024 / (2 W) k rows of a W-wide tile, lane l writing the
// 16-byte slot l mod (W / 8) of its row. That slot holds the vector
// slot ^ 4 sw(k) of the row (the chunk swizzle of the k-major layout); since
// every copy starts at a k row that is a multiple of 4 (W = 128) or 8
// (W = 64), sw(k) depends on the lane alone, and so does the vector a
// thread fetches: one output-channel vector of A and one (tap, channel)
// vector of B per thread.
#ifndef LRCNN_WG_DMA
#define LRCNN_WG_DMA 1
#endif
#ifndef LRCNN_WG_DMA_ST
#define LRCNN_WG_DMA_ST 3
#endif
#ifndef LRCNN_WG_DMA_OCC
#define LRCNN_WG_DMA_OCC 2
#endif
// The K index runs over padded pixels q = (b, y, x) with x in [0, Wp),
// Wp = Wv rounded up to a multiple of 8; columns x >= Wv read zeros. A K step's 32 pixels are four
// aligned groups of 8, one per wave, and such a group lies in one row: the
// wave walks its group's (b, y, x) and base offsets with scalar
// instructions, and a lane only adds a constant of its own (its pixel's
// place in the group, its channel vector, its tap) and tests its bounds
// against scalar limits. Wave w's A copies fill tile rows 8w .. 8w+7 and
// so do its B copies, so both operands of a tile row hold the same pixel.
template <int WBM>
__global__ __launch_bounds__(256, LRCNN_WG_DMA_OCC) void wgrad_rowg_kernel(WgradArgs a,
                                                                           int kchunk,
                                                                           float *dw) {
  using T = bf16;
  constexpr int E = 8, BK = 32, BN = 128, ST = LRCNN_WG_DMA_ST;
  static_assert(ST == 3 || ST == 4, "ring depth");
  constexpr int FBN = WBM == 128 ? 128 : 64, NB = FBN / 64;
  constexpr int VA = WBM / E, RA = 64 / VA;  // vectors per A row, A rows per copy
  constexpr int NIA = 8 / RA;                // A copies per wave per tile
  constexpr int NIB = 2;                     // B copies per wave per tile (4 rows each)
  constexpr int LD = NIA + NIB;
  constexpr uint32_t ASB = BK * WBM * 2, BSB = BK * BN * 2;
  static_assert(4 * NIA * 1024 == ASB && 4 * NIB * 1024 == BSB, "copy cover");
  __shared__ __align__(16) char smem[ST * (ASB + BSB)];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int R = a.y1 - a.y0, Wp = a.Wp;
  const int K = a.B * R * Wp;  // padded pixels
  const int N = a.kh * a.kw * a.Ci;
  const TileId tl = xcd_tile(false);
  const int m0 = tl.x * WBM, n0 = tl.y * BN;
  const int kbeg = tl.z * kchunk;
  const int kend = min(K, kbeg + kchunk);
  const char *dc = (const char *)a.dc;
  const char *src = (const char *)a.src.p;
  const long long srow = (long long)a.src.W * a.src.C;
  constexpr long long ES = 2;

  // per-lane constants. A: group place kbA[j] (a lane whose channel vector
  // is past C_out gets a place no group reaches), channel vector at ova
  constexpr int FAR = 1 << 30;
  int kbA[NIA];
  uint32_t lA[NIA];
  const int ova = m0 + E * ((lane % VA) ^ (KM<T, WBM>::sw(lane / VA) << 2));
  const bool ovok = ova < a.Co;
#pragma unroll
  for (int j = 0; j < NIA; ++j) {
    kbA[j] = j * RA + lane / VA;
    lA[j] = (uint32_t)(((long long)kbA[j] * a.Co + ova) * ES);
    kbA[j] = ovok ? kbA[j] : FAR;
  }
  // B: group place kbB[j], (tap, channel) vector nb; column offset of the
  // pixel under the tap relative to the group's first pixel
  const int nb = n0 + E * ((lane % 16) ^ (KM<T, BN>::sw(lane / 16) << 2));
  const int tap = nb / a.Ci;
  const int bti = tap / a.kw, btj = tap - (tap / a.kw) * a.kw;
  const bool bnok = nb < N;
  int kbB[NIB], bx[NIB];
  uint32_t lB[NIB];
#pragma unroll
  for (int j = 0; j < NIB; ++j) {
    kbB[j] = 4 * j + lane / 16;
    bx[j] = btj + kbB[j] * a.sw;
    lB[j] = (uint32_t)(((long long)bti * srow + (long long)bx[j] * a.src.C + (nb - tap * a.Ci)) *
                       ES);
    kbB[j] = bnok ? kbB[j] : FAR;
  }
  // the wave's group: first pixel q = kbeg + 8 wave of the first tile
  int xs, ys, bs_;
  {
    uint32_t t, x, yy, b;
    fdiv_qr((uint32_t)(kbeg + 8 * wave), a.fw, t, x);
    fdiv_qr(t, a.fr, b, yy);
    xs = __builtin_amdgcn_readfirstlane((int)x);
    ys = __builtin_amdgcn_readfirstlane((int)yy);
    bs_ = __builtin_amdgcn_readfirstlane((int)b);
  }
  // scalar walk state: A byte offset of the group's first pixel, B byte
  // offset of the source position under tap (0, 0), that position's row
  // and column, and the pixels of the launch's range left from the group
  long long offA = ((long long)(bs_ * R + ys) * a.Wv + xs) * a.Co * ES;
  int sy = (a.y0 + ys) * a.sh - a.ph, sx = xs * a.sw - a.pw;
  long long offB = ((long long)bs_ * a.src.bs + (long long)(sy - a.src.row0) * srow +
                    (long long)sx * a.src.C) * ES;
  int kl = kend - (kbeg + 8 * wave);  // pixels of the range from the group on
  // per-step increments (BK = wdb (R Wp) + wdy Wp + wdx padded pixels)
  const long long dA0 = ((long long)(a.wdb * R + a.wdy) * a.Wv + a.wdx) * a.Co * ES;
  const long long dA1 = (long long)(a.Wv - Wp) * a.Co * ES;
  const int dyb = a.wdy * a.sh, ryb = R * a.sh;
  const long long dB0 =
      ((long long)a.wdb * a.src.bs + (long long)dyb * srow + (long long)a.wdx * a.sw * a.src.C) *
      ES;
  const long long dB1 = ((long long)a.sh * srow - (long long)Wp * a.sw * a.src.C) * ES;
  const long long dB2 = (a.src.bs - (long long)ryb * srow) * ES;
  const int dsx = a.wdx * a.sw, wsx = Wp * a.sw;
  const uint32_t lds_a = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)smem;
  const uint32_t lds_b = lds_a + ST * ASB;
  const void *zblk = &g_zero16[0];
  asm volatile("" : "+s"(zblk));
  // (bounds as unsigned compares: v in [0, L) iff (unsigned)v < L)
  auto gload = [&](int st) {
    const int lim = min(a.Wv - xs, kl);  // group places inside the row and the range
    const uint32_t yy = (uint32_t)(sy + bti);
#pragma unroll
    for (int j = 0; j < NIA; ++j)
      load16_lds_a(dc + offA + lA[j], kbA[j] < lim,
                   lds_a + st * ASB + (uint32_t)(wave * NIA + j) * 1024u, zblk);
#pragma unroll
    for (int j = 0; j < NIB; ++j) {
      const bool ok = (kbB[j] < lim) & (yy < (uint32_t)a.Hs) & ((uint32_t)(sx + bx[j]) < (uint32_t)a.Ws);
      load16_lds_a(src + offB + lB[j], ok,
                   lds_b + st * BSB + (uint32_t)(wave * NIB + j) * 1024u, zblk);
    }
    // next tile: the group moves BK padded pixels on (scalar; the row and
    // image carries are rare unless rows are shorter than a K step)
    xs += a.wdx;
    ys += a.wdy;
    offA += dA0;
    offB += dB0;
    sy += dyb;
    sx += dsx;
    kl -= BK;
    if (__builtin_expect(xs >= Wp, 0)) {
      xs -= Wp;
      ys += 1;
      offA += dA1;
      offB += dB1;
      sy += a.sh;
      sx -= wsx;
    }
    if (__builtin_expect(ys >= R, 0)) {
      ys -= R;
      offB += dB2;
      sy -= ryb;
    }
  };
  auto As = [&](int st) { return (const T *)(smem + st * ASB); };
  auto Bs = [&](int st) { return (const T *)(smem + ST * ASB + st * BSB); };

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
  using FR = Frag<T, FBN, 4, 1, 1, WBM, BN>;
  FR f0, f1;
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
  if (n > 0) f0.load(As(0), Bs(0), wm, wn, lane);
  int sc = 0;
  auto dstep = [&](int t, FR &cur, FR &nxt) {
    const int s1 = sc == ST - 1 ? 0 : sc + 1;
    if (t + 1 < n) {
      wait_tiles(min(n - 1, t + ST - 1) - t - 1);
      __syncthreads();
      nxt.load(As(s1), Bs(s1), wm, wn, lane);
      if (t + ST < n) gload(sc);
    }
    cur.mma(acc);
    sc = s1;
  };
  auto dstep_full = [&](FR &cur, FR &nxt) {
    const int s1 = sc == ST - 1 ? 0 : sc + 1;
    wait_vmcnt<(ST - 2) * LD>();
    __syncthreads();
    nxt.load(As(s1), Bs(s1), wm, wn, lane);
    gload(sc);
    cur.mma(acc);
    interleave_step<FR::NMFMA, FR::NDSR, 0, LD>();
    sc = s1;
  };
  int t = 0;
  for (; t + ST + 1 < n; t += 2) {
    dstep_full(f0, f1);
    dstep_full(f1, f0);
  }
  for (; t + 1 < n; t += 2) {
    dstep(t, f0, f1);
    dstep(t + 1, f1, f0);
  }
  if (t < n) dstep(t, f0, f1);
  wgrad_store<NB>(a, dw, acc, m0 + wm, n0 + wn, N, tl.z, lane);
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
    // four loads in flight, added in split order
    int z = g;
    for (; z + 24 < splits; z += 32) {
      float q4[4][4];
#pragma unroll
      for (int u = 0; u < 4; ++u) ldv<float, V>(part + (z + 8 * u) * mn + i, q4[u]);
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int k = 0; k < V; ++k) acc[k] += q4[u][k];
    }
    for (; z < splits; z += 8) {
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
  const bool avec = (a.Co % Cfg<T>::E) == 0, bvec = (a.Ci % Cfg<T>::E) == 0;
  // (the split count is chosen in units of BK pixels, as the planner sizes
  // the partial sums; a wide K step rounds each chunk up to its own width,
  // which never adds splits)
  const bool wide = LRCNN_WG_KR == 8 && sizeof(T) == 2 && avec && bvec;
  const bool rowg = LRCNN_WG_DMA && sizeof(T) == 2 && avec && bvec && !wide;
  const int BKL = wide ? 8 * Cfg<T>::E : BK;
  a.wdx = BKL % a.Wv;
  a.wdy = (BKL / a.Wv) % (a.y1 - a.y0);
  a.wdb = BKL / (a.Wv * (a.y1 - a.y0));
  const WgradTiles wt = wgrad_tiles(a.Co, N, K, a.out ? a.part_bytes : 0, (int)sizeof(T));
  int splits = wt.splits;
  const int KT = (K + BK - 1) / BK;
  const int kchunk = ((KT + splits - 1) / splits * BK + BKL - 1) / BKL * BKL;
  splits = (K + kchunk - 1) / kchunk;
  if (!split_fits(splits, a.Co, N, a.out, a.part_bytes)) return (int)hipErrorInvalidValue;
  const int wbm = wt.rows;
  int kchunk_l = kchunk;
  if (rowg) {
    // padded pixels: rows of Wp = Wv rounded up to 8 columns; the split
    // count is the estimate's, each chunk a whole number of K steps
    a.Wp = (a.Wv + 7) / 8 * 8;
    a.fw = fast_div((uint32_t)a.Wp);
    a.wdx = BK % a.Wp;
    a.wdy = (BK / a.Wp) % (a.y1 - a.y0);
    a.wdb = BK / (a.Wp * (a.y1 - a.y0));
    const long long Kp = (long long)a.B * (a.y1 - a.y0) * a.Wp;
    if (Kp >= (1ll << 31)) return (int)hipErrorInvalidValue;
    const long long KTp = (Kp + BK - 1) / BK;
    kchunk_l = (int)((KTp + wt.splits - 1) / wt.splits * BK);
    splits = (int)((Kp + kchunk_l - 1) / kchunk_l);
    if (!split_fits(splits, a.Co, N, a.out, a.part_bytes)) return (int)hipErrorInvalidValue;
  }
  dim3 grid((a.Co + wbm - 1) / wbm, (N + 127) / 128, splits);
  // algorithmic bytes: the error operand, the source rows under the taps
  // (once), and the partial sums (split) or dW (read and written unless
  // this band's launch initializes it)
  const long long rin =
      std::max(0, std::min(a.Hs, (a.y1 - 1) * a.sh - a.ph + a.kh) - std::max(0, a.y0 * a.sh - a.ph));
  const double mnb = 4.0 * a.Co * N;
  const double wbytes = (double)K * a.Co * sizeof(T) + (double)a.B * rin * a.Ws * a.Ci * sizeof(T) +
                        (splits > 1 ? splits * mnb : (a.overwrite ? 1.0 : 2.0) * mnb);
  int pr = -1;
  if (prof::on)
    pr = prof::begin(std::string("wgrad_kernel<") + (sizeof(T) == 4 ? "float" : "bf16") +
                         (avec && bvec ? ", vec>" : ", scalar>"),
                     2.0 * K * a.Co * N, s, wbytes, (int)sizeof(T));
  if (rowg) {
    if (wbm == 64) launch_timed(wgrad_rowg_kernel<64>, grid, s, pr, a, kchunk_l, dw);
    else launch_timed(wgrad_rowg_kernel<128>, grid, s, pr, a, kchunk_l, dw);
  } else if (wide) {
    if (wbm == 64) launch_timed(wgrad_kernel<T, 64, true, true, 8>, grid, s, pr, a, kchunk, dw);
    else launch_timed(wgrad_kernel<T, 128, true, true, 8>, grid, s, pr, a, kchunk, dw);
  } else if (wbm == 64) {
    if (avec && bvec) launch_timed(wgrad_kernel<T, 64, true, true>, grid, s, pr, a, kchunk, dw);
    else if (avec) launch_timed(wgrad_kernel<T, 64, true, false>, grid, s, pr, a, kchunk, dw);
    else launch_timed(wgrad_kernel<T, 64, false, false>, grid, s, pr, a, kchunk, dw);
  } else {
    if (avec && bvec) launch_timed(wgrad_kernel<T, 128, true, true>, grid, s, pr, a, kchunk, dw);
    else if (avec) launch_timed(wgrad_kernel<T, 128, true, false>, grid, s, pr, a, kchunk, dw);
    else launch_timed(wgrad_kernel<T, 128, false, false>, grid, s, pr, a, kchunk, dw);
  }
  if (splits > 1) {
    long long mn = (long long)a.Co * N;
    int p2 = prof::begin("wgrad_reduce_kernel", 0.0, s,
                         4.0 * mn * (splits + (a.overwrite ? 1 : 2)), 4);
    if (mn % 4 == 0)
      launch_timed(wgrad_reduce_kernel<4>, dim3((unsigned)((mn / 4 + 31) / 32)), s, p2,
                   (const float *)a.out, dw, mn, splits, a.overwrite);
    else
      launch_timed(wgrad_reduce_kernel<1>, dim3((unsigned)((mn + 31) / 32)), s, p2,
                   (const float *)a.out, dw, mn, splits, a.overwrite);
  }
  return (int)hipGetLastError();
}

int launch_wgrad(int dt, const WgradArgs &a, float *dw, void *stream) {
  hipStream_t s = (hipStream_t)stream;
  return dt == DT_F32 ? wgrad_dispatch<float>(a, dw, s) : wgrad_dispatch<bf16>(a, dw, s);
}

}  // namespace lrcnn
