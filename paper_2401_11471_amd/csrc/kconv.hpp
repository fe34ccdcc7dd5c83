// Implicit-GEMM convolution kernel (forward and input gradient), its
// split-K reduction and its launchers, instantiated per storage type and
// direction by the conv_*.hip translation units.
#pragma once

#include <type_traits>

#include "kdev.hpp"

namespace lrcnn {

// input gradients of strided convolutions: 0 = by estimate, 1 = always
// stride phases, 2 = never (kernels.hip)
extern thread_local int g_phases;

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
  // swizzled LDS slot is lane mod KR: each wave's rows fill 1 KiB of LDS in
  // lane order, the layout of a direct copy.
  constexpr bool LANE_SLOT = (KR == 4 || KR == 8) && LRCNN_SWZ;
  // Input gradient, stride 1, bfloat16: the same, with the weights' k-major
  // tile copied in lane order too (k rows of BN unpadded elements; a
  // thread's column vector is the one its lane's swizzled slot holds).
  constexpr bool DMA = LRCNN_LDS_DMA && LANE_SLOT && VEC &&
                       (!DGRAD || (LRCNN_DG_DMA && S1 && !ONE && sizeof(T) == 2));
  // LDS stages. Register staging: while tile t is multiplied, the
  // fragments of t+1 are read, tile t+2 is written and tile t+3 is fetched
  // from global memory. Direct copies: tiles t+2 .. t+ST-1 are in flight.
  constexpr int ST = DMA ? LRCNN_DMA_ST : 3;
  // input gradient: weights staged k-major (16-byte stores)
  constexpr int BKM = DGRAD ? 1 : 0;
  constexpr int BSZ = BKM ? BK * KM<T, BN>::P : BN * LDK;
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
  // l puts it in LDS slot l & 3 (the swizzle is an XOR with (row >> 2) & 3;
  // rows are l / 4 + 64 i); with 8 vectors per row (l & 7) ^ ((l >> 4) & 7)
  // puts it in slot l & 7 (XOR with (row >> 1) & 7, rows l / 8 + 32 i)
  const int kv = !LANE_SLOT ? tid % KR
                 : KR == 8   ? ((tid & 7) ^ ((tid >> 4) & 7))
                             : ((tid & 3) ^ ((tid >> 4) & 3));
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
  constexpr bool RMASK = DGRAD && S1 && VEC && !ONE && !DMA;
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
    bn[j] = DGRAD ? n0 + E * (DMA ? (tid % BV) ^ (KM<T, BN>::sw(tid / BV) << 2) : tid % BV)
                  : n0 + tid / KR + RS * j;
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
  // 1x1 forward with a fused residual add (64-wide tiles): the epilogue's
  // residual vectors are fetched here, before the K loop, so their latency
  // overlaps it instead of following it (a 1x1 layer's loop is a few
  // steps). Thread rows r = tid / (BN / E) + i * RPR, as in the epilogue.
  constexpr bool PRE = ONE && !DGRAD && BN == 64 && HR == BM && sizeof(T) == 2;
  constexpr int PCR = BN / E, RPR = 256 / PCR, PRN = PRE ? BM / RPR : 1;
  uint4 pre_res[PRN];
  const bool pre = PRE && a.res.p && (a.N % E) == 0;
  if (PRE && pre) {
    const long long drw = (long long)a.dst.W * a.N;
    const int pn = n0 + (tid % PCR) * E;
#pragma unroll
    for (int i = 0; i < PRN; ++i) {
      const int m = m0 + tid / PCR + RPR * i;
      const bool ok = m < M && pn < a.N;
      uint32_t t_, x_, b_, y_;
      fdiv_qr((uint32_t)(ok ? m : 0), a.fw, t_, x_);
      fdiv_qr(t_, a.fr, b_, y_);
      const int x = a.px0 + (int)x_, y = a.y0 + (int)y_, b = (int)b_;
      const long long ro = b * a.res.bs + (y - a.res.row0) * drw + (long long)x * a.N + pn;
      pre_res[i] = load16z(a.res.p, ro * (long long)sizeof(T), ok);
    }
  }

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
      for (int j = 0; j < NBL; ++j) {
        if (DGRAD) {
          // k rows (wave * 64) / BV + BKS * j + lane / BV of the k-major tile
          load16_lds_a(wp[j] + wb, bvld[j] & (cb + bk0 + BKS * j < a.KC),
                       lds_b + st * BSB +
                           (uint32_t)((wave * 64) / BV + BKS * j) * BN * (uint32_t)sizeof(T),
                       zblk);
        } else {
          load16_lds_a(wp[j] + wb, bvld[j] & cok,
                       lds_b + st * BSB + (wrow + RS * j) * LDK * (uint32_t)sizeof(T), zblk);
        }
      }
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
      *(uint4 *)(&As[st][(tid / KR + RS * i) * LDK + swz<KR>(tid / KR + RS * i, kv) * E]) = ra[i];
#pragma unroll
    for (int j = 0; j < NBL; ++j) {
      if (BKM) {
        *(uint4 *)(&Bs[st][KM<T, BN>::off(bk0 + BKS * j, (tid % BV) * E)]) = rb[j];
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
        *(uint4 *)(&Bs[st][(tid / KR + RS * j) * LDK + swz<KR>(tid / KR + RS * j, kv) * E]) = rb[j];
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
    // the affine parameters of this lane's columns, read once (columns
    // past N are staged but never stored)
    float csc[NB], csh[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int nn = n0 + wn + 32 * j + col;
      const bool ok = a.scale && nn < a.N;
      csc[j] = ok ? a.scale[nn] : 1.f;
      csh[j] = ok ? a.shift[nn] : 0.f;
    }
    // the accumulators of this wave's rows in [h0, h0 + HR), affine and
    // ReLU applied, into the staging tile (SC / RL fixed per launch, so
    // the unrolled loop has no branches)
    auto stage = [&](auto SC, auto RL, int h0) {
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int r = wm - h0 + 32 * i + acc_row(v, lane);
#pragma unroll
          for (int j = 0; j < NB; ++j) {
            float val = acc[i][j][v];
            if constexpr (decltype(SC)::value) val = val * csc[j] + csh[j];
            if constexpr (decltype(RL)::value) val = val > 0.f ? val : 0.f;
            stf(&Ct[r * CP + wn + 32 * j + col], val);
          }
        }
    };
    // (the chunk's mask bytes start at a multiple of E bytes from the base)
    const bool mask_vec = ((uintptr_t)a.mask & (E - 1)) == 0;
    using yes = std::true_type;
    using no = std::false_type;
    for (int h0 = 0; h0 < BM; h0 += HR) {
    if (h0) __syncthreads();
    if (wm >= h0 && wm < h0 + HR) {
      if (a.scale) {
        if (a.relu) stage(yes(), yes(), h0);
        else stage(yes(), no(), h0);
      } else {
        if (a.relu) stage(no(), yes(), h0);
        else stage(no(), no(), h0);
      }
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < HR / RPP; ++i) {
      const int r = h0 + tid / CPR + RPP * i;
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
        // input (prefetched for 1x1 layers), then the add's ReLU
        union {
          uint4 u;
          T e[E];
        } cv, rv;
        cv.u = q;
        if (PRE) rv.u = pre_res[i];
        else
          rv.u = *(const uint4 *)((const T *)a.res.p + b * a.res.bs +
                                  (y - a.res.row0) * drow + (long long)x * a.N + n);
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
        // E mask bytes (1 where the stored value is > 0) in one store
        union {
          uint4 u;
          T e[E];
        } w;
        w.u = q;
        uint64_t bits = 0;
#pragma unroll
        for (int e = 0; e < E; ++e) bits |= (uint64_t)(ldf(&w.e[e]) > 0.f ? 1 : 0) << (8 * e);
        uint8_t *mk = a.mask + (((long long)b * a.mask_h + y) * a.Wd + x) * a.N + n;
        if (mask_vec) {
          if (E == 8) *(uint64_t *)mk = bits;
          else *(uint32_t *)mk = (uint32_t)bits;
        } else {
#pragma unroll
          for (int e = 0; e < E; ++e) mk[e] = (uint8_t)(bits >> (8 * e));
        }
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
    // four loads in flight, added in split order
    int z = g;
    for (; z + 3 * G < splits; z += 4 * G) {
      float q4[4][4];
#pragma unroll
      for (int u = 0; u < 4; ++u) ldv<float, V>(a.part + (z + G * u) * MN + idx, q4[u]);
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int k = 0; k < V; ++k) val[k] += q4[u][k];
    }
    for (; z < splits; z += G) {
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

// Algorithmic HBM bytes of a convolution launch (M output pixels): the
// source rows under the taps and the weights read once, and the output:
// forward, the stored map (plus the fused add's other input and the mask
// when present); input gradient, the float32 error window (read and
// written unless the launch initializes it). A split launch writes its
// partial sums instead, which its epilogue (epi) reads back before writing
// the output.
template <typename T, bool DGRAD>
static double conv_bytes(const ConvArgs &a, long long M, int splits, bool epi) {
  const double es = sizeof(T), mn = (double)M * a.N;
  const double out = DGRAD ? mn * 4.0 * (a.dst_init ? 1.0 : 2.0)
                           : mn * es * (a.res.p ? 2.0 : 1.0) + (a.mask ? mn : 0.0);
  if (epi) return splits * mn * 4.0 + out;
  int lo, hi;
  if (DGRAD) {
    const int s = a.sh > 0 ? a.sh : 1;
    const int t = a.y0 + a.ph - a.kh + 1;
    lo = std::max(a.sy0, t > 0 ? (t + s - 1) / s : 0);
    hi = std::min(a.sy1, (a.y1 - 1 + a.ph) / s + 1);
  } else {
    lo = std::max(a.sy0, a.y0 * a.sh - a.ph);
    hi = std::min(a.sy1, (a.y1 - 1) * a.sh - a.ph + a.kh);
  }
  const double in = (double)a.B * std::max(0, hi - lo) * a.Ws * a.KC * es;
  const double w = (double)a.N * a.kh * a.kw * a.KC * es;
  return in + w + (splits > 1 ? splits * mn * 4.0 : out);
}

template <typename T, bool DGRAD>
static int conv_launch(const ConvArgs &a0, hipStream_t s) {
  constexpr int KR = LRCNN_CONV_KR;
  using CF = Cfg<T, KR>;
  ConvArgs a = a0;
  const int M = a.B * (a.y1 - a.y0) * a.Wd;
  if (M <= 0 || a.N <= 0) return 0;
  // (the 16-byte loaders test taps against a 64-bit mask: larger kernels
  // take the element-wise loader)
  const int es = (int)sizeof(T);
  const bool vec = conv_vec(a.kh, a.kw, a.KC, a.N, es, DGRAD);
  a.tpack = !vec && conv_tap_packed(a.KC, es, DGRAD);
  a.fkw = fast_div((uint32_t)a.kw);
  // K step width of this launch (the planner counts iterations the same way)
  const int kr = conv_kr(a.kh, a.kw, a.KC, a.N, es, DGRAD);
  const int KT = conv_k_iters(a.kh * a.kw, a.KC, es, DGRAD, kr);
  // a fixed split count (the layer's, for the forward) or the estimate's
  if (a.splits > 0 && !split_valid(KT, a.splits)) return (int)hipErrorInvalidValue;
  const ConvTiles ct = a.splits > 0
                           ? conv_tiles_split(M, a.N, KT, a.splits, es, kr)
                           : conv_tiles(M, a.N, KT, a.part ? a.part_bytes : 0, es, kr);
  const int bn = ct.bn;
  const int splits = ct.splits;
  // a fused residual add needs the vector epilogues of the forward
  if (a.res.p && (DGRAD || (a.N % CF::E) != 0)) return (int)hipErrorInvalidValue;
  // split partial sums must fit the buffer (the schedule never exceeds it)
  if (!split_fits(splits, M, a.N, a.part, a.part_bytes)) return (int)hipErrorInvalidValue;
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
    // (1x1 kernels, which carry little reuse per loaded byte, are named
    // apart from the windowed ones)
    const bool one_ = vec && a.kh == 1 && a.kw == 1;
    std::string nm = std::string("conv_gemm_kernel<") + (sizeof(T) == 4 ? "float" : "bf16") +
                     ", " + std::to_string(bn) + (DGRAD ? ", dgrad" : ", fwd") +
                     (!vec ? ", scalar>" : one_ ? ", 1x1>" : ", vec>");
    pr = prof::begin(nm, fl, s, conv_bytes<T, DGRAD>(a, M, splits, false), es);
  }
  // the input gradient of a strided convolution divides by the stride
  // (a phase of it is dense)
  const bool s1 = !DGRAD || (a.sh == 1 && a.sw == 1) || a.pst > 1;
  const bool one = vec && s1 && a.kh == 1 && a.kw == 1;
  bool done = false;
  if constexpr (!DGRAD && sizeof(T) == 2 && LRCNN_CONV_KR_WIN != KR) {
    // bfloat16 forward of a windowed kernel: wider K steps, 64-wide tiles
    if (kr != KR) {
      if (bn != 64 || !vec || one) return (int)hipErrorInvalidValue;
      launch_timed(conv_gemm_kernel<T, 64, LRCNN_CONV_KR_WIN, false, true, true>, grid, s, pr, a);
      done = true;
    }
  }
  if (done) {
  } else if (bn == 64) {
    if (!s1) {
      if (vec) launch_timed(conv_gemm_kernel<T, 64, KR, DGRAD, true, false>, grid, s, pr, a);
      else launch_timed(conv_gemm_kernel<T, 64, KR, DGRAD, false, false>, grid, s, pr, a);
    } else if (one) {
      launch_timed(conv_gemm_kernel<T, 64, KR, DGRAD, true, true, true>, grid, s, pr, a);
    } else if (vec) {
      launch_timed(conv_gemm_kernel<T, 64, KR, DGRAD, true, true>, grid, s, pr, a);
    } else {
      launch_timed(conv_gemm_kernel<T, 64, KR, DGRAD, false, true>, grid, s, pr, a);
    }
  } else {
    if (!s1) {
      if (vec) launch_timed(conv_gemm_kernel<T, 128, KR, DGRAD, true, false>, grid, s, pr, a);
      else launch_timed(conv_gemm_kernel<T, 128, KR, DGRAD, false, false>, grid, s, pr, a);
    } else if (one) {
      launch_timed(conv_gemm_kernel<T, 128, KR, DGRAD, true, true, true>, grid, s, pr, a);
    } else if (vec) {
      launch_timed(conv_gemm_kernel<T, 128, KR, DGRAD, true, true>, grid, s, pr, a);
    } else {
      launch_timed(conv_gemm_kernel<T, 128, KR, DGRAD, false, true>, grid, s, pr, a);
    }
  }
  if (splits > 1) {
    int p2 = prof::begin("conv_split_epilogue", 0.0, s, conv_bytes<T, DGRAD>(a, M, splits, true),
                         es);
    const int G = splits >= 8 ? 8 : splits >= 4 ? 4 : 2;
    const long long vecs = a.N % 4 == 0 ? (long long)M * a.N / 4 : (long long)M * a.N;
    const unsigned blocks = (unsigned)((vecs + 256 / G - 1) / (256 / G));
    if (a.N % 4 == 0)
      launch_timed(conv_split_epilogue<T, DGRAD, 4>, dim3(blocks), s, p2, a, splits, G);
    else
      launch_timed(conv_split_epilogue<T, DGRAD, 1>, dim3(blocks), s, p2, a, splits, G);
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

}  // namespace lrcnn
