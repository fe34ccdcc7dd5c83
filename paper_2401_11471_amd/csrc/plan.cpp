// Planner: shapes, per-band row intervals, workspace layout and analytic
// figures. Host only (no HIP calls), so it runs without a GPU.
#include <algorithm>
#include <climits>
#include <cstring>
#include <new>
#include <string>

#include "kernels.hpp"
#include "plan.hpp"

namespace {
thread_local std::string g_err;

int floordiv(int a, int b) { return (a >= 0) ? a / b : -((-a + b - 1) / b); }

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

struct Alloc {
  size_t top = 0;
  size_t take(size_t bytes) {
    size_t off = top;
    top = align256(top + bytes);
    return off;
  }
};
}  // namespace

int lrcnn_fail(int code, const std::string &msg) {
  g_err = msg;
  return code;
}

extern "C" const char *lrcnn_last_error(void) { return g_err.c_str(); }

namespace lrcnn {

thread_local bool g_no_act_fusion = false;

// k, s, p of the window through which node v reads its input(s); an ADD
// reads row y of each input for output row y.
static void ksp(const lrcnn_node &nd, int &k, int &s, int &p) {
  if (nd.op == LRCNN_OP_ADD) {
    k = 1, s = 1, p = 0;
  } else {
    k = nd.kh, s = nd.sh, p = nd.ph;
  }
}

// Rows of node v's output that can be computed once rows [0, f) of its
// input exist: output row y reads input rows [y*s-p, y*s-p+k) (clipped to
// the image, whose top and bottom are padded; Section III-B).
static int frontier(int f, int h_in, int h_out, int k, int s, int p) {
  if (f >= h_in) return h_out;
  int last = floordiv(f + p - k, s);
  return std::max(0, std::min(h_out, last + 1));
}

// CARRY intervals for the given input-row bounds.
static void carry_rows(Plan &P, const std::vector<int> &bounds) {
  const int n = P.n, nb = (int)bounds.size() - 1;
  std::vector<std::vector<int>> F(nb + 1, std::vector<int>(n, 0));
  for (int r = 1; r <= nb; ++r) {
    F[r][0] = bounds[r];
    for (int v = 1; v < n; ++v) {
      const lrcnn_node &nd = P.nodes[v];
      if (nd.op == LRCNN_OP_ADD) {
        F[r][v] = std::min(F[r][nd.in0], F[r][nd.in1]);
      } else {
        int k, s, p;
        ksp(nd, k, s, p);
        F[r][v] = frontier(F[r][nd.in0], P.shp[nd.in0].h, P.shp[v].h, k, s, p);
      }
    }
  }
  // first row of v that a later band may still read: consumers' next rows
  // start at F[r][c], whose windows begin at F[r][c]*s - p
  std::vector<std::vector<int>> T(nb + 1, std::vector<int>(n, 0));
  for (int r = 1; r <= nb; ++r)
    for (int v = 0; v < n; ++v) {
      int t = F[r][v];
      for (int c : P.cons[v]) {
        int k, s, p;
        ksp(P.nodes[c], k, s, p);
        t = std::min(t, F[r][c] * s - p);
      }
      T[r][v] = std::max(0, std::min(t, F[r][v]));
    }
  P.rows.assign(nb, std::vector<Rows>(n));
  P.tail.assign(nb, std::vector<int>(n));
  for (int r = 1; r <= nb; ++r)
    for (int v = 0; v < n; ++v) {
      P.rows[r - 1][v] = Rows{F[r - 1][v], F[r][v], T[r - 1][v], F[r][v]};
      P.tail[r - 1][v] = T[r][v];
    }
}

// RECOMPUTE cones for the given output-row bounds (Eq. (15) read as an
// interval recursion from the last layer down to the input).
static void cone_rows(Plan &P, const std::vector<int> &bounds) {
  const int n = P.n, nb = (int)bounds.size() - 1;
  P.rows.assign(nb, std::vector<Rows>(n));
  for (int r = 0; r < nb; ++r) {
    std::vector<int> lo(n, 0), hi(n, 0);
    lo[n - 1] = bounds[r];
    hi[n - 1] = bounds[r + 1];
    for (int v = n - 2; v >= 0; --v) {
      int a = INT_MAX, b = INT_MIN;
      for (int c : P.cons[v]) {
        if (hi[c] <= lo[c]) continue;
        int k, s, p;
        ksp(P.nodes[c], k, s, p);
        a = std::min(a, std::max(0, lo[c] * s - p));
        b = std::max(b, std::min(P.shp[v].h, (hi[c] - 1) * s - p + k));
      }
      if (a == INT_MAX || b <= a) {
        lo[v] = hi[v] = 0;
      } else {
        lo[v] = a;
        hi[v] = b;
      }
    }
    for (int v = 0; v < n; ++v) P.rows[r][v] = Rows{lo[v], hi[v], lo[v], hi[v]};
  }
}

// Largest per-band cache (bytes of all held rows) for CARRY bounds.
static double max_band_cache(Plan &P, const std::vector<int> &bounds) {
  carry_rows(P, bounds);
  double best = 0;
  for (auto &br : P.rows) {
    double tot = 0;
    for (int v = 1; v < P.n; ++v)
      tot += (double)P.elems(v, br[v].hi - br[v].lo) * P.es;
    best = std::max(best, tot);
  }
  return best;
}

// BALANCED: smallest bound on the per-band cache that N bands can meet,
// found by bisection; each band is extended greedily as far as the bound
// allows (a band's cache grows with its end row and shrinks with its start
// row, so the greedy extension is optimal).
static std::vector<int> balanced_bounds(Plan &P, int H, int nb) {
  auto cache_of = [&](int a, int b) {
    std::vector<int> bd = {0, a, b, H};
    if (a == 0) bd = {0, b, H};
    carry_rows(P, bd);
    const auto &br = P.rows[a == 0 ? 0 : 1];
    double tot = 0;
    for (int v = 1; v < P.n; ++v)
      tot += (double)P.elems(v, br[v].hi - br[v].lo) * P.es;
    return tot;
  };
  auto greedy = [&](double cap, std::vector<int> &out) {
    out.assign(1, 0);
    int a = 0;
    for (int r = 0; r < nb && a < H; ++r) {
      if (r == nb - 1) {
        if (cache_of(a, H) > cap) return false;
        a = H;
        out.push_back(H);
        break;
      }
      int lo = a, hi = H;  // largest b with cache_of(a, b) <= cap
      while (lo < hi) {
        int mid = lo + (hi - lo + 1) / 2;
        if (cache_of(a, mid) <= cap) lo = mid; else hi = mid - 1;
      }
      a = lo;
      out.push_back(a);
    }
    if (a < H) return false;
    while ((int)out.size() < nb + 1) out.push_back(H);
    return true;
  };
  std::vector<int> even(nb + 1), cur;
  for (int r = 0; r <= nb; ++r) even[r] = (int)((int64_t)r * H / nb);
  double hi = max_band_cache(P, even), lo = 0;
  std::vector<int> best = even;
  for (int it = 0; it < 60 && hi - lo > 1.0; ++it) {
    double mid = 0.5 * (lo + hi);
    if (greedy(mid, cur)) {
      hi = mid;
      best = cur;
    } else {
      lo = mid;
    }
  }
  return best;
}

// Rows of the last node completed once input rows [0, x) exist (the
// frontiers of every node, as in carry_rows).
static int last_frontier(const Plan &P, int x) {
  std::vector<int> F(P.n, 0);
  F[0] = x;
  for (int v = 1; v < P.n; ++v) {
    const lrcnn_node &nd = P.nodes[v];
    if (nd.op == LRCNN_OP_ADD) {
      F[v] = std::min(F[nd.in0], F[nd.in1]);
    } else {
      int k, s, p;
      ksp(nd, k, s, p);
      F[v] = frontier(F[nd.in0], P.shp[nd.in0].h, P.shp[v].h, k, s, p);
    }
  }
  return F[P.n - 1];
}

// PAPER_2PS: the greedy partition of two-phase sharing (Section IV-A). The
// first band completes `first` rows of the last node (H_1^L), the others
// share the remaining rows evenly; each band's input height is inferred
// from the last layer back to the input: the end of band r is the smallest
// input row count whose last-node frontier reaches the band's target t_r.
// For a chain this is Eq. (11) for the first band (H_1^l = (H_1^{l+1} - 1)
// s + k - p) and Eq. (13) for the middle bands (H_r^l = H_r^{l+1} s); the
// last band takes the rest of the input (Eq. (14)). The frontier is
// monotone in the input rows, so the smallest count is found by bisection.
static std::vector<int> paper_bounds(const Plan &P, int H, int nb, int first) {
  const int HL = P.shp[P.n - 1].h;
  const int h1 = first > 0 ? std::min(first, HL) : (HL + nb - 1) / nb;
  std::vector<int> bd(nb + 1, 0);
  bd[nb] = H;
  for (int r = 1; r < nb; ++r) {
    const int t = h1 + (int)((int64_t)(r - 1) * (HL - h1) / std::max(1, nb - 1));
    int lo = bd[r - 1], hi = H;  // smallest x in [bd[r-1], H] with frontier >= t
    while (lo < hi) {
      const int mid = lo + (hi - lo) / 2;
      if (last_frontier(P, mid) >= t) hi = mid; else lo = mid + 1;
    }
    bd[r] = lo;
  }
  return bd;
}

static int validate(const lrcnn_node *nodes, int n, const lrcnn_config *cfg) {
  if (!nodes || !cfg) return lrcnn_fail(LRCNN_EINVAL, "null nodes or config");
  if (n < 2) return lrcnn_fail(LRCNN_ESHAPE, "need an input node and at least one layer");
  if (nodes[0].op != LRCNN_OP_INPUT)
    return lrcnn_fail(LRCNN_ESHAPE, "node 0 must be the input");
  if (cfg->batch < 1 || cfg->in_c < 1 || cfg->in_h < 1 || cfg->in_w < 1)
    return lrcnn_fail(LRCNN_ESHAPE, "batch and input sizes must be positive");
  if (cfg->dtype != LRCNN_F32 && cfg->dtype != LRCNN_BF16)
    return lrcnn_fail(LRCNN_EDTYPE, "dtype must be LRCNN_F32 or LRCNN_BF16");
  if (cfg->mode != LRCNN_CARRY && cfg->mode != LRCNN_RECOMPUTE)
    return lrcnn_fail(LRCNN_EINVAL, "mode must be LRCNN_CARRY or LRCNN_RECOMPUTE");
  if (cfg->n_bands < 1) return lrcnn_fail(LRCNN_EPARTITION, "n_bands must be >= 1");
  if (cfg->policy < LRCNN_EVEN || cfg->policy > LRCNN_PAPER_2PS)
    return lrcnn_fail(LRCNN_EINVAL, "bad partition policy");
  if (cfg->policy == LRCNN_BALANCED && cfg->mode != LRCNN_CARRY)
    return lrcnn_fail(LRCNN_EINVAL, "BALANCED applies to CARRY mode only");
  if (cfg->policy == LRCNN_PAPER_2PS && cfg->mode != LRCNN_CARRY)
    return lrcnn_fail(LRCNN_EINVAL, "PAPER_2PS applies to CARRY mode only");
  if (cfg->policy == LRCNN_PAPER_2PS && cfg->first_rows < 0)
    return lrcnn_fail(LRCNN_EPARTITION, "first_rows must be >= 0");
  if (cfg->policy == LRCNN_EXPLICIT && !cfg->bounds)
    return lrcnn_fail(LRCNN_EINVAL, "EXPLICIT policy needs bounds");
  if (cfg->bp_refine < 0 || cfg->bp_refine > 64)
    return lrcnn_fail(LRCNN_EINVAL, "bp_refine must be in [0, 64]");
  if (cfg->hybrid_from < LRCNN_HYBRID_AUTO || cfg->hybrid_from == 1 ||
      (cfg->hybrid_from > 0 && cfg->hybrid_from > n - 1))
    return lrcnn_fail(LRCNN_EINVAL, "hybrid_from must be 0 or in [2, n_nodes - 1]");
  for (int v = 1; v < n; ++v) {
    const lrcnn_node &d = nodes[v];
    std::string at = "node " + std::to_string(v) + ": ";
    if (d.op < LRCNN_OP_CONV || d.op > LRCNN_OP_ADD)
      return lrcnn_fail(LRCNN_ESHAPE, at + "bad op");
    if (d.in0 < 0 || d.in0 >= v)
      return lrcnn_fail(LRCNN_ESHAPE, at + "in0 must name an earlier node");
    if (d.op == LRCNN_OP_ADD && (d.in1 < 0 || d.in1 >= v))
      return lrcnn_fail(LRCNN_ESHAPE, at + "in1 must name an earlier node");
    if (d.op == LRCNN_OP_CONV || d.op == LRCNN_OP_MAXPOOL) {
      if (d.kh < 1 || d.kw < 1 || d.sh < 1 || d.sw < 1 || d.ph < 0 || d.pw < 0 ||
          d.ph >= d.kh || d.pw >= d.kw)
        return lrcnn_fail(LRCNN_ESHAPE, at + "need k >= 1, s >= 1, 0 <= p < k");
    }
    if (d.op == LRCNN_OP_CONV && d.c_out < 1)
      return lrcnn_fail(LRCNN_ESHAPE, at + "c_out must be >= 1");
    if (d.op == LRCNN_OP_MAXPOOL && d.kh * d.kw > 255)
      return lrcnn_fail(LRCNN_ESHAPE, at + "pool window larger than 255");
  }
  return LRCNN_OK;
}

// Interval first-fit packing of buffers with [start, end] live steps.
struct LiveBuf {
  int start, end;
  size_t bytes;
  size_t off;
};

static size_t pack(std::vector<LiveBuf> &bufs) {
  std::vector<int> order(bufs.size());
  for (size_t i = 0; i < order.size(); ++i) order[i] = (int)i;
  std::sort(order.begin(), order.end(), [&](int a, int b) {
    return bufs[a].bytes != bufs[b].bytes ? bufs[a].bytes > bufs[b].bytes : a < b;
  });
  std::vector<int> placed;
  size_t peak = 0;
  for (int i : order) {
    LiveBuf &b = bufs[i];
    // candidate offsets: 0 and the end of every overlapping placed buffer
    std::vector<size_t> cand = {0};
    for (int j : placed) {
      const LiveBuf &o = bufs[j];
      if (o.end < b.start || b.end < o.start) continue;
      cand.push_back(align256(o.off + o.bytes));
    }
    std::sort(cand.begin(), cand.end());
    for (size_t c : cand) {
      bool ok = true;
      for (int j : placed) {
        const LiveBuf &o = bufs[j];
        if (o.end < b.start || b.end < o.start) continue;
        if (c < o.off + o.bytes && o.off < c + b.bytes) { ok = false; break; }
      }
      if (ok) { b.off = c; break; }
    }
    placed.push_back(i);
    peak = std::max(peak, align256(b.off + b.bytes));
  }
  return peak;
}

// Bytes of split-K partial sums one launch may use.
#ifndef LRCNN_PART_MIB
#define LRCNN_PART_MIB 24
#endif
static constexpr size_t kPartCap = (size_t)LRCNN_PART_MIB << 20;

// Split-K count of every conv's forward launches. All forward launches of a
// layer -- the row-centric bands, their backward recompute and the
// layer-wise launch -- use one count, so each output element sums the same
// K chunks in the same order whatever band computes it: the row-centric and
// layer-wise forwards (and the ReLU / argmax decisions) are then bitwise
// equal. The count is the one with the smallest summed duration estimate
// over those launches (the layer-wise launch in row chunks whose partial
// sums fit the buffer), among the counts whose partial sums fit the buffer
// at every row-centric launch.
static void forward_splits(Plan &P,
                           const std::vector<const std::vector<std::vector<Rows>> *> &tabs) {
  if ((int)P.fsplit_fixed.size() == P.n) {
    P.fsplit = P.fsplit_fixed;
    return;
  }
  P.fsplit.assign(P.n, 0);
  const long long B = P.cfg.batch;
  for (int v = 1; v < P.n; ++v) {
    const lrcnn_node &d = P.nodes[v];
    if (d.op != LRCNN_OP_CONV) continue;
    const Shape &su = P.shp[d.in0], &sv = P.shp[v];
    const int kr = conv_kr(d.kh, d.kw, su.c, sv.c, P.es, false);
    const int KT = conv_k_iters(d.kh * d.kw, su.c, P.es, false, kr);
    std::vector<long long> ms;
    long long mmax = 0;
    for (auto *tab : tabs)
      for (auto &br : *tab)
        if (br[v].b > br[v].a) {
          ms.push_back(B * (br[v].b - br[v].a) * sv.w);
          mmax = std::max(mmax, ms.back());
        }
    int best_s = 1;
    double best = -1;
    for (int sp = 1; sp <= 128; ++sp) {
      if (!split_valid(KT, sp)) continue;
      if (sp > 1 && (size_t)sp * (size_t)mmax * sv.c * 4 > kPartCap) break;
      double t = 0;
      for (long long m : ms) t += conv_tiles_split(m, sv.c, KT, sp, P.es, kr).us;
      // the layer-wise launch, in chunks of rows
      const size_t row_part = (size_t)sp * B * sv.w * sv.c * 4;
      const int rows = sp > 1 ? (int)std::min<size_t>(sv.h, std::max<size_t>(1, kPartCap / row_part))
                              : sv.h;
      const int full = sv.h / rows, rest = sv.h - full * rows;
      t += full * conv_tiles_split(B * rows * sv.w, sv.c, KT, sp, P.es, kr).us;
      if (rest) t += conv_tiles_split(B * rest * sv.w, sv.c, KT, sp, P.es, kr).us;
      if (best < 0 || t < best * 0.98) {
        best = t;
        best_s = sp;
      }
    }
    P.fsplit[v] = best_s;
  }
}

// Lay out one workspace. Backward (and, unless packed, forward) windows
// hold cap[v] rows, a band owns at most own[v] rows, carry[v] rows of error
// are carried (CARRY). `bands` lists the row intervals of every launch
// (forward and backward partitions) for sizing the partial sums; `fpw`
// (nullable) gives the forward windows' rows when they are packed by
// lifetime.
static void layout(Plan &P, Layout &L, const Fuse &F, const std::vector<int> &cap,
                   const std::vector<int> &own, const std::vector<int> &carry,
                   const std::vector<const std::vector<std::vector<Rows>> *> &bands,
                   bool strips, bool layerwise, bool dxacc, const std::vector<int> *fpw) {
  const int n = P.n;
  Alloc A;
  L = Layout();
  L.win.assign(n, 0);
  L.win_cap = cap;
  L.argmax.assign(n, 0);
  L.argmax_cap.assign(n, 0);
  L.delta.assign(n, 0);
  L.carry.assign(n, 0);
  L.carry2.assign(n, 0);
  L.carry_cap = carry;
  L.strip.assign(P.nb, std::vector<size_t>(n, 0));
  L.fwin.assign(n, 0);
  L.fwin_cap.assign(n, 0);
  // strips: shared rows kept from FP to BP at every backward band boundary
  if (strips) {
    size_t s0 = A.top;
    for (int r = 0; r + 1 < P.nb; ++r)
      for (int v = 1; v < n; ++v) {
        int rows_ = P.rows[r][v].b - P.tail[r][v];
        if (rows_ > 0) L.strip[r][v] = A.take(P.elems(v, rows_) * P.es);
      }
    L.strip_bytes = A.top - s0;
  }
  // partial sums (used by FP and BP): split-K of the weight gradient and of
  // the convolution forward / input gradient, for every launch the
  // schedule makes, with the launchers' own split rule
  size_t part = 0;
  std::vector<size_t> wpn(n, 0);  // per conv node: weight-gradient partial bytes
  // a first layer whose input channels do not fill 16-byte vectors computes
  // its weight gradient from a channel-padded copy of the input rows
  const int vec_e = 16 / P.es;
  L.cpad = P.shp[0].c % vec_e ? (P.shp[0].c + vec_e - 1) / vec_e * vec_e : 0;
  int xrows = 0;
  const size_t pcap = kPartCap;
  // The layer-wise schedule's partial sums get a buffer that does not
  // depend on the row partition (the baseline's memory must not move with
  // it): what the largest split of the largest launch would need, capped
  // at the launch cap; its forward launches run in row chunks that fit.
  size_t lw_part = 0;
  if (layerwise) {
    for (int v = 1; v < n; ++v)
      if (P.nodes[v].op == LRCNN_OP_CONV) {
        const Shape &su = P.shp[P.nodes[v].in0], &sv = P.shp[v];
        const size_t mf = (size_t)P.cfg.batch * sv.h * sv.w * sv.c;
        const size_t md = (size_t)P.cfg.batch * su.h * su.w * su.c;
        lw_part = std::max(lw_part, 128 * std::max(mf, md) * 4);
      }
    lw_part = std::min(lw_part, pcap);
  }
  L.fchunk.assign(n, 0);
  for (int v = 1; v < n; ++v)
    if (P.nodes[v].op == LRCNN_OP_CONV) {
      const lrcnn_node &d = P.nodes[v];
      const Shape &su = P.shp[d.in0], &sv = P.shp[v];
      const int taps = d.kh * d.kw;
      const bool padded = L.cpad && d.in0 == 0;
      const int64_t nw = (int64_t)taps * (padded ? L.cpad : su.c);
      // forward launches: the layer's fixed split count; a layer-wise launch
      // too large for the partial buffer runs as several row chunks
      const int sf = P.fsplit[v];
      const size_t row_part = (size_t)sf * P.cfg.batch * sv.w * sv.c * 4;
      if (layerwise && sf > 1) {
        const int rows_fit = (int)std::max<size_t>(1, lw_part / row_part);
        L.fchunk[v] = rows_fit < sv.h ? rows_fit : 0;
      }
      std::vector<Rows> qs;
      if (layerwise) qs.push_back(Rows{0, sv.h, 0, sv.h});
      for (auto *tab : bands)
        for (auto &br : *tab) qs.push_back(br[v]);
      for (const Rows &q : qs) {
        if (q.b <= q.a) continue;
        const long long mf = (long long)P.cfg.batch * (q.b - q.a) * sv.w;
        const int sw_ = wgrad_split_count(d.c_out, nw, mf, pcap, P.es);
        if (sw_ > 1) wpn[v] = std::max(wpn[v], (size_t)sw_ * d.c_out * nw * 4);
        if (sf > 1 && !layerwise) part = std::max(part, (size_t)sf * (size_t)mf * sv.c * 4);
        const int u0 = std::max(0, q.a * d.sh - d.ph);
        const int u1 = std::min(su.h, (q.b - 1) * d.sh - d.ph + d.kh);
        if (padded) xrows = std::max(xrows, u1 - u0);
        const long long md = (long long)P.cfg.batch * (u1 - u0) * su.w;
        const int sd = conv_split_count(md, su.c, conv_k_iters(taps, sv.c, P.es, true), pcap, P.es);
        if (sd > 1) part = std::max(part, (size_t)(sd * md * su.c * 4));
      }
    }
  if (layerwise) part = lw_part;
  L.part_bytes = part;
  L.part = A.take(part);
  const size_t ubase = A.top;
  L.ubase = ubase;
  // --- backward region (also the forward windows unless packed)
  size_t c0 = A.top;
  for (int v = 1; v < n; ++v) {
    if (layerwise && v == n - 1 && !P.lw_keep_out) continue;  // the output lives in y
    L.win[v] = A.take(P.elems(v, cap[v]) * P.es);
  }
  L.cache_bytes = A.top - c0;
  L.dwpad.assign(n, 0);
  if (L.cpad) {
    L.xpad_cap = xrows;
    L.xpad = A.take((size_t)P.cfg.batch * xrows * P.shp[0].w * L.cpad * P.es);
    for (int v = 1; v < n; ++v)
      if (P.nodes[v].op == LRCNN_OP_CONV && P.nodes[v].in0 == 0)
        L.dwpad[v] = A.take((size_t)P.nodes[v].c_out * P.nodes[v].kh * P.nodes[v].kw * L.cpad * 4);
  }
  for (int v = 1; v < n; ++v)
    if (P.nodes[v].op == LRCNN_OP_MAXPOOL) {
      L.argmax_cap[v] = own[v];
      L.argmax[v] = A.take(P.elems(v, own[v]));
    }
  size_t k0 = A.top;
  for (int v = 0; v < n; ++v)
    if (carry[v] > 0) {
      L.carry[v] = A.take(P.elems(v, carry[v]) * 4);
      if (F.act[v] != 0) L.carry2[v] = A.take(P.elems(v, carry[v]) * 4);
    }
  L.carry_bytes = A.top - k0;
  // BP arena, packed by lifetime over the backward steps (step s handles
  // node n-1-s):
  //  - node v's error window lives from the step of its first consumer in
  //    reverse order (the largest consumer id) to its own step;
  //  - a conv's error operand and weight-gradient partial sums are read by
  //    the weight gradient on the side stream, which the caller's stream
  //    joins at the start of the next conv's step, so they live from the
  //    conv's own step up to that one.
  std::vector<LiveBuf> bufs(n);
  for (int v = 0; v < n; ++v) {
    int first = v;
    for (int c : P.cons[v]) first = std::max(first, c);
    // (an act-fused conv's error window only stages the rows its consumer's
    // input gradient carries out, which the launch may not write into the
    // carry buffer it reads the rows carried in from)
    const bool staged = F.act[v] != 0;
    bufs[v] = LiveBuf{n - 1 - first, n - 1 - v, P.elems(v, staged ? carry[v] : cap[v]) * 4, 0};
  }
  std::vector<int> dc_i(n, -1), wp_i(n, -1);
  for (int v = 1; v < n; ++v) {
    if (P.nodes[v].op != LRCNN_OP_CONV) continue;
    int nxt = 0;  // next conv in backward order
    for (int u = v - 1; u >= 1 && !nxt; --u)
      if (P.nodes[u].op == LRCNN_OP_CONV) nxt = u;
    // (a conv fed by an add's backward gets its error operand at the add's step)
    // (or at the step of the conv whose input gradient forms it)
    const int early = F.add[v] ? F.add[v] : F.act[v] ? F.act[v] : v;
    const int s0 = n - 1 - early;
    const int s1 = nxt ? n - 2 - nxt : n - 1;
    dc_i[v] = (int)bufs.size();
    bufs.push_back(LiveBuf{s0, s1, P.elems(v, own[v]) * P.es, 0});
    if (wpn[v] > 0) {
      wp_i[v] = (int)bufs.size();
      bufs.push_back(LiveBuf{s0, s1, wpn[v], 0});
    }
  }
  size_t dpeak = pack(bufs);
  size_t d0 = A.take(dpeak);
  L.arena = d0;
  L.arena_bytes = dpeak;
  for (int v = 0; v < n; ++v) L.delta[v] = d0 + bufs[v].off;
  L.dc.assign(n, 0);
  L.wpart.assign(n, 0);
  L.wpart_bytes.assign(n, 0);
  for (int v = 1; v < n; ++v) {
    if (dc_i[v] >= 0) L.dc[v] = d0 + bufs[dc_i[v]].off;
    if (wp_i[v] >= 0) {
      L.wpart[v] = d0 + bufs[wp_i[v]].off;
      L.wpart_bytes[v] = wpn[v];
    }
  }
  L.delta_bytes = dpeak;
  if (dxacc) {
    L.dxacc_bytes = P.elems(0, P.shp[0].h) * 4;
    L.dxacc = A.take(L.dxacc_bytes);
  }
  const size_t bp_end = A.top;
  // --- forward windows packed by lifetime: node v's window lives from its
  // own step to its last consumer's step (topological order); they reuse
  // the backward region, which FP does not touch
  size_t fp_end = ubase;
  if (fpw) {
    L.fp_packed = true;
    L.fwin_cap = *fpw;
    std::vector<LiveBuf> fb;
    std::vector<int> ids;
    for (int v = 1; v + 1 < n; ++v) {
      int last = v;
      for (int c : P.cons[v]) last = std::max(last, c);
      fb.push_back(LiveBuf{v, last, P.elems(v, (*fpw)[v]) * P.es, 0});
      ids.push_back(v);
    }
    size_t fpeak = pack(fb);
    for (size_t t = 0; t < ids.size(); ++t) L.fwin[ids[t]] = ubase + fb[t].off;
    L.fwin_bytes = fpeak;
    fp_end = ubase + align256(fpeak);
  }
  L.total = std::max<size_t>(std::max(bp_end, fp_end), 256);
}

// Fusions of a schedule whose backward bands have rows `rows` and forward
// bands `rows_fp` (act_ok: the schedule may form a conv's error operand in
// its consumer's backward launch -- CARRY and layer-wise).
static Fuse decide_fusions(const Plan &P, const std::vector<std::vector<Rows>> &rows,
                           const std::vector<std::vector<Rows>> &rows_fp, bool act_ok) {
  const int n = P.n, nb = (int)rows.size();
  Fuse F;
  // convs whose error operand the residual add's backward can write
  F.add.assign(n, 0);
  for (int v = 1; v < n; ++v) {
    const lrcnn_node &d = P.nodes[v];
    if (d.op != LRCNN_OP_CONV || d.relu || P.cons[v].size() != 1) continue;
    const int c = P.cons[v][0];
    if (P.nodes[c].op != LRCNN_OP_ADD || P.nodes[c].in0 == P.nodes[c].in1) continue;
    bool ok = true;
    for (int r = 0; r < nb && ok; ++r) ok = rows[r][v].lo == rows[r][v].a;
    if (ok) F.add[v] = c;
  }
  F.fwd.assign(n, 0);
  for (int v = 1; v < n; ++v) {
    const int c = F.add[v];
    if (!c || v != std::max(P.nodes[c].in0, P.nodes[c].in1)) continue;
    if (P.shp[v].c % (16 / P.es) != 0) continue;
    bool ok = true;
    for (int r = 0; r < nb && ok; ++r)
      ok = rows[r][v].a == rows[r][c].a && rows[r][v].b == rows[r][c].b;
    for (size_t r = 0; r < rows_fp.size() && ok; ++r)
      ok = rows_fp[r][v].a == rows_fp[r][c].a && rows_fp[r][v].b == rows_fp[r][c].b &&
           rows_fp[r][v].lo == rows_fp[r][v].a;
    if (ok) F.fwd[v] = c;
  }
  // convs whose error operand the backward launch of their only consumer v
  // (a conv's input gradient, a max-pool's backward) forms: in every band
  // v's launch must cover exactly u's error-window rows, which end with u's
  // own rows, or the band must hold nothing of u; u's float32 error window
  // is then never used
  F.act.assign(n, 0);
  if (act_ok && !g_no_act_fusion)
    for (int u = 1; u < n; ++u) {
      if (P.nodes[u].op != LRCNN_OP_CONV || F.add[u] || P.cons[u].size() != 1) continue;
      const int v = P.cons[u][0];
      const lrcnn_node &d = P.nodes[v];
      if (d.op != LRCNN_OP_CONV && d.op != LRCNN_OP_MAXPOOL) continue;
      const int hu = P.shp[u].h;
      bool ok = true;
      for (int r = 0; r < nb && ok; ++r) {
        const Rows &qv = rows[r][v], &qu = rows[r][u];
        if (qv.b > qv.a) {
          const int y0 = std::max(0, qv.a * d.sh - d.ph);
          const int y1 = std::min(hu, (qv.b - 1) * d.sh - d.ph + d.kh);
          ok = y0 == qu.lo && y1 == qu.hi && qu.hi == qu.b && qu.lo <= qu.a;
        } else {
          ok = qu.b <= qu.a && qu.lo == qu.a;
        }
      }
      if (ok) F.act[u] = v;
    }
  return F;
}

static int shapes_and_consumers(Plan &P) {
  const int n = P.n;
  // shapes
  P.shp.assign(n, Shape{});
  P.shp[0] = Shape{P.cfg.in_h, P.cfg.in_w, P.cfg.in_c};
  for (int v = 1; v < n; ++v) {
    const lrcnn_node &d = P.nodes[v];
    const Shape &u = P.shp[d.in0];
    std::string at = "node " + std::to_string(v) + ": ";
    if (d.op == LRCNN_OP_ADD) {
      const Shape &u1 = P.shp[d.in1];
      if (u1.h != u.h || u1.w != u.w || u1.c != u.c)
        return lrcnn_fail(LRCNN_ESHAPE, at + "ADD inputs differ in shape");
      P.shp[v] = u;
    } else {
      int ho = floordiv(u.h + 2 * d.ph - d.kh, d.sh) + 1;
      int wo = floordiv(u.w + 2 * d.pw - d.kw, d.sw) + 1;
      if (ho < 1 || wo < 1) return lrcnn_fail(LRCNN_ESHAPE, at + "empty output");
      P.shp[v] = Shape{ho, wo, d.op == LRCNN_OP_CONV ? d.c_out : u.c};
    }
  }
  P.cons.assign(n, {});
  for (int v = 1; v < n; ++v) {
    P.cons[P.nodes[v].in0].push_back(v);
    if (P.nodes[v].op == LRCNN_OP_ADD) P.cons[P.nodes[v].in1].push_back(v);
  }
  for (int v = 0; v + 1 < n; ++v)
    if (P.cons[v].empty())
      return lrcnn_fail(LRCNN_ESHAPE, "node " + std::to_string(v) +
                                          " feeds nothing (only the last node is an output)");
  return LRCNN_OK;
}

static void finish(Plan &P, const std::vector<int> &bd, const std::vector<int> &bb,
                   bool quick = false);

// Peak workspace of the row-centric step for forward bounds `bd` (the
// backward bands refine each evenly), planned on a scratch copy.
static size_t workspace_for(const Plan &P, const std::vector<int> &bd) {
  Plan Q;
  Q.nodes = P.nodes;
  Q.cfg = P.cfg;
  Q.cfg.bounds = nullptr;
  Q.n = P.n;
  Q.es = P.es;
  Q.shp = P.shp;
  Q.cons = P.cons;
  Q.no_keep = P.no_keep;
  Q.dy_f32 = P.dy_f32;
  Q.lw_keep_out = P.lw_keep_out;
  const int refine = P.cfg.bp_refine > 1 ? P.cfg.bp_refine : 1;
  const int nbf = (int)bd.size() - 1;
  std::vector<int> bb;
  for (int r = 0; r < nbf; ++r)
    for (int j = 0; j < refine; ++j)
      bb.push_back(bd[r] + (int)((int64_t)(bd[r + 1] - bd[r]) * j / refine));
  bb.push_back(bd[nbf]);
  finish(Q, bd, bb, true);
  return Q.rc.total;
}

// BALANCED: forward bounds that minimise the step's peak workspace (every
// buffer the plan lays out: band windows, shared-row strips, error
// windows, carries, partial sums). Starts from the better of the even split
// and the bounds that balance the per-band caches (the skew of Section
// IV-A), then moves one boundary at a time by decreasing steps while the
// workspace shrinks (a bounded local search over exact plans).
static std::vector<int> balanced_peak_bounds(Plan &P, int H, int nb) {
  std::vector<int> even(nb + 1);
  for (int r = 0; r <= nb; ++r) even[r] = (int)((int64_t)r * H / nb);
  std::vector<int> best = even;
  size_t best_ws = workspace_for(P, even);
  if (nb <= 1) return best;
  {
    std::vector<int> bal = balanced_bounds(P, H, nb);
    const size_t w = workspace_for(P, bal);
    if (w < best_ws) {
      best_ws = w;
      best = bal;
    }
  }
  int evals = 0;
  const int max_evals = 400;
  for (int step = std::max(1, H / (2 * nb)); step >= 1 && evals < max_evals; step /= 2) {
    bool moved = true;
    while (moved && evals < max_evals) {
      moved = false;
      for (int r = 1; r < nb && evals < max_evals; ++r)
        for (int sgn = -1; sgn <= 1; sgn += 2) {
          std::vector<int> cand = best;
          cand[r] += sgn * step;
          if (cand[r] < cand[r - 1] || cand[r] > cand[r + 1]) continue;
          const size_t w = workspace_for(P, cand);
          ++evals;
          if (w < best_ws) {
            best_ws = w;
            best = cand;
            moved = true;
          }
        }
    }
  }
  return best;
}

static int build(Plan &P) {
  const int n = P.n;
  int st = shapes_and_consumers(P);
  if (st != LRCNN_OK) return st;
  // bounds of the forward partition, refined evenly for the backward one
  const bool carry = P.cfg.mode == LRCNN_CARRY;
  const int H = carry ? P.shp[0].h : P.shp[n - 1].h;
  const int nbf = P.cfg.n_bands;
  const int refine = P.cfg.bp_refine > 1 ? P.cfg.bp_refine : 1;
  std::vector<int> bd(nbf + 1);
  if (P.cfg.policy == LRCNN_EXPLICIT) {
    for (int r = 0; r <= nbf; ++r) bd[r] = P.cfg.bounds[r];
    if (bd[0] != 0 || bd[nbf] != H)
      return lrcnn_fail(LRCNN_EPARTITION, "bounds must run from 0 to " + std::to_string(H));
    for (int r = 0; r < nbf; ++r)
      if (bd[r + 1] < bd[r]) return lrcnn_fail(LRCNN_EPARTITION, "bounds must be non-decreasing");
  } else if (P.cfg.policy == LRCNN_BALANCED) {
    bd = balanced_peak_bounds(P, H, nbf);
  } else if (P.cfg.policy != LRCNN_PAPER_2PS) {
    for (int r = 0; r <= nbf; ++r) bd[r] = (int)((int64_t)r * H / nbf);
  }
  std::vector<int> bb;
  if (P.cfg.policy == LRCNN_PAPER_2PS) {
    // the partition is made for the backward bands; the forward bands are
    // every refine-th of them
    bb = paper_bounds(P, H, nbf * refine, P.cfg.first_rows);
    for (int r = 0; r <= nbf; ++r) bd[r] = bb[r * refine];
  } else {
    for (int r = 0; r < nbf; ++r)
      for (int j = 0; j < refine; ++j)
        bb.push_back(bd[r] + (int)((int64_t)(bd[r + 1] - bd[r]) * j / refine));
    bb.push_back(H);
  }
  (void)n;
  finish(P, bd, bb);
  return LRCNN_OK;
}

// Everything after the bounds: row intervals of both partitions, fusions,
// split counts, the two workspace layouts and the FLOP figures (quick:
// only what the row-centric workspace size needs).
static void finish(Plan &P, const std::vector<int> &bd, const std::vector<int> &bb, bool quick) {
  const int n = P.n;
  const bool carry = P.cfg.mode == LRCNN_CARRY;
  const int nbf = (int)bd.size() - 1;
  const int refine = (int)(bb.size() - 1) / std::max(1, nbf);
  P.nb_fp = nbf;
  P.refine = refine;
  P.nb = nbf * refine;
  P.bounds_fp = bd;
  P.bounds = bb;
  if (carry) carry_rows(P, bd); else cone_rows(P, bd);
  P.rows_fp = P.rows;
  if (carry) carry_rows(P, bb); else cone_rows(P, bb);
  const int nb = P.nb;
  P.fz = decide_fusions(P, P.rows, P.rows_fp, carry);
  {
    // the layer-wise schedule: one band of whole maps
    std::vector<std::vector<Rows>> whole(1, std::vector<Rows>(n));
    for (int v = 0; v < n; ++v) whole[0][v] = Rows{0, P.shp[v].h, 0, P.shp[v].h};
    P.fz_lw = decide_fusions(P, whole, whole, true);
  }
  // capacities
  std::vector<int> cap(n, 0), own(n, 0), cry(n, 0), fcap(n, 0);
  for (int r = 0; r < nb; ++r)
    for (int v = 0; v < n; ++v) {
      const Rows &q = P.rows[r][v];
      cap[v] = std::max(cap[v], q.hi - q.lo);
      own[v] = std::max(own[v], q.b - q.a);
      if (carry) cry[v] = std::max(cry[v], q.b - P.tail[r][v]);
    }
  for (int r = 0; r < nbf; ++r)
    for (int v = 0; v < n; ++v) {
      const Rows &q = P.rows_fp[r][v];
      fcap[v] = std::max(fcap[v], q.hi - q.lo);
    }
  std::vector<const std::vector<std::vector<Rows>> *> tabs = {&P.rows, &P.rows_fp};
  forward_splits(P, tabs);
  layout(P, P.rc, P.fz, cap, own, cry, tabs, carry, false, !carry && P.cfg.dtype == LRCNN_BF16,
         refine > 1 ? &fcap : nullptr);
  if (quick) return;
  std::vector<int> full(n), zero(n, 0);
  for (int v = 0; v < n; ++v) full[v] = P.shp[v].h;
  layout(P, P.lw, P.fz_lw, full, full, zero, {}, false, true, false, nullptr);
  // FLOPs: tau of Section IV-B and the row-centric total (FP over the
  // forward bands; BP recompute, input and weight gradient over the backward
  // bands; without recomputing the last band when FP left it in place)
  P.tau = 0;
  double fp = 0, bp = 0, last = 0;
  for (int v = 1; v < n; ++v)
    if (P.nodes[v].op == LRCNN_OP_CONV) {
      const lrcnn_node &d = P.nodes[v];
      double per_row = 2.0 * d.kh * d.kw * P.cfg.batch * P.shp[d.in0].c * d.c_out * P.shp[v].w;
      P.tau += per_row * P.shp[v].h;
      for (int r = 0; r < nbf; ++r) fp += per_row * (P.rows_fp[r][v].b - P.rows_fp[r][v].a);
      for (int r = 0; r < nb; ++r) bp += per_row * (P.rows[r][v].b - P.rows[r][v].a);
      last += per_row * (P.rows[nb - 1][v].b - P.rows[nb - 1][v].a);
    }
  P.flops_rows = fp + 3.0 * bp - (refine == 1 ? last : 0.0);
  P.shared_rows = 0;
  P.halo_rows = 0;
  for (int r = 0; r < nb; ++r)
    for (int v = 0; v < n; ++v) {
      if (carry && r + 1 < nb) P.shared_rows += P.rows[r][v].b - P.tail[r][v];
      if (!carry) P.halo_rows += P.rows[r][v].b - P.rows[r][v].a;
    }
  if (!carry)
    for (int v = 0; v < n; ++v) P.halo_rows -= P.shp[v].h;
}

}  // namespace lrcnn

using lrcnn::Plan;

namespace lrcnn {

// Hybrid depth (2PS-H / OverL-H): a checkpoint at node c = hyb - 1 splits
// the network into a row-centric part (nodes 0..c) and a layer-wise part
// (nodes hyb..n-1, which read c as their input). Built as two sub-plans.
static int build_hybrid(Plan &P, bool quiet = false) {
  const int k = P.cfg.hybrid_from, c = k - 1, n = P.n;
  for (int v = k; v < n; ++v) {
    const lrcnn_node &d = P.nodes[v];
    if (d.in0 < c || (d.op == LRCNN_OP_ADD && d.in1 < c)) {
      if (quiet) return LRCNN_EINVAL;
      return lrcnn_fail(LRCNN_EINVAL, "hybrid checkpoint at node " + std::to_string(c) +
                                          " is crossed by an edge into node " +
                                          std::to_string(v));
    }
  }
  auto sub = [&](std::vector<lrcnn_node> nodes, const lrcnn_config &cfg, Plan *&out) -> int {
    Plan *Q = new (std::nothrow) Plan();
    if (!Q) return lrcnn_fail(LRCNN_EINVAL, "out of host memory");
    Q->nodes = std::move(nodes);
    Q->cfg = cfg;
    Q->n = (int)Q->nodes.size();
    Q->es = P.es;
    out = Q;
    return LRCNN_OK;
  };
  lrcnn_config rc = P.cfg;
  rc.hybrid_from = 0;
  std::vector<lrcnn_node> rn(P.nodes.begin(), P.nodes.begin() + k);
  int st = sub(rn, rc, P.row);
  if (st != LRCNN_OK) return st;
  P.row->no_keep = true;
  P.row->dy_f32 = true;
  P.row->fsplit_fixed.assign(P.fsplit.begin(), P.fsplit.begin() + k);
  st = build(*P.row);
  P.row->cfg.bounds = nullptr;
  if (st != LRCNN_OK) return st;
  lrcnn_config cc = P.cfg;
  cc.hybrid_from = 0;
  cc.in_c = P.shp[c].c, cc.in_h = P.shp[c].h, cc.in_w = P.shp[c].w;
  cc.mode = LRCNN_CARRY;
  cc.n_bands = 1;
  cc.policy = LRCNN_EVEN;
  cc.bounds = nullptr;
  cc.bp_refine = 1;
  std::vector<lrcnn_node> cn(1 + n - k);
  cn[0] = P.nodes[0];
  for (int v = k; v < n; ++v) {
    lrcnn_node d = P.nodes[v];
    d.in0 -= c;
    if (d.op == LRCNN_OP_ADD) d.in1 -= c;
    cn[v - c] = d;
  }
  if ((st = sub(cn, cc, P.col)) != LRCNN_OK) return st;
  P.col->lw_keep_out = true;
  P.col->fsplit_fixed.assign(1 + n - k, 0);
  for (int v = k; v < n; ++v) P.col->fsplit_fixed[v - c] = P.fsplit[v];
  if ((st = build(*P.col)) != LRCNN_OK) return st;
  P.hyb = k;
  P.h_col = P.row->rc.ubase;
  const size_t top = std::max(P.row->rc.total, P.h_col + P.col->lw.total);
  P.h_ck = align256(top);
  P.h_dck = align256(P.h_ck + P.elems(c, P.shp[c].h) * P.es);
  P.h_total = align256(P.h_dck + P.elems(c, P.shp[c].h) * 4);
  P.flops_rows = P.row->flops_rows + 3.0 * P.col->tau;
  return LRCNN_OK;
}

}  // namespace lrcnn

extern "C" int lrcnn_plan(const lrcnn_node *nodes, int32_t n_nodes,
                          const lrcnn_config *cfg, lrcnn_plan_t **out) {
  if (!out) return lrcnn_fail(LRCNN_EINVAL, "null output pointer");
  *out = nullptr;
  int st = lrcnn::validate(nodes, n_nodes, cfg);
  if (st != LRCNN_OK) return st;
  Plan *P = new (std::nothrow) Plan();
  if (!P) return lrcnn_fail(LRCNN_EINVAL, "out of host memory");
  P->nodes.assign(nodes, nodes + n_nodes);
  P->cfg = *cfg;
  P->cfg.bounds = nullptr;
  P->n = n_nodes;
  P->es = cfg->dtype == LRCNN_BF16 ? 2 : 4;
  if (cfg->policy == LRCNN_EXPLICIT) {
    // keep the caller's bounds only for the duration of build()
    P->cfg.bounds = cfg->bounds;
  }
  st = lrcnn::build(*P);
  if (st == LRCNN_OK && cfg->hybrid_from == LRCNN_HYBRID_AUTO) {
    // budget-driven choice of the checkpoint: the smallest workspace over
    // every valid cut (each is planned on a scratch copy), none if no cut
    // beats the all-row-centric plan
    int best = 0;
    size_t best_ws = P->rc.total;
    for (int k = 2; k < n_nodes; ++k) {
      Plan Q;
      Q.nodes = P->nodes;
      Q.cfg = P->cfg;
      Q.cfg.hybrid_from = k;
      Q.n = P->n;
      Q.es = P->es;
      if (lrcnn::build(Q) != LRCNN_OK || lrcnn::build_hybrid(Q, true) != LRCNN_OK) continue;
      if (Q.h_total < best_ws) {
        best_ws = Q.h_total;
        best = k;
      }
    }
    P->cfg.hybrid_from = best;
  }
  if (st == LRCNN_OK && P->cfg.hybrid_from > 0) st = lrcnn::build_hybrid(*P);
  P->cfg.bounds = nullptr;
  if (st != LRCNN_OK) {
    delete P;
    return st;
  }
  *out = reinterpret_cast<lrcnn_plan_t *>(P);
  return LRCNN_OK;
}

extern "C" int lrcnn_plan_query(const lrcnn_plan_t *plan, lrcnn_plan_info *info) {
  if (!plan || !info) return lrcnn_fail(LRCNN_EINVAL, "null plan or info");
  const Plan &P = *reinterpret_cast<const Plan *>(plan);
  std::memset(info, 0, sizeof(*info));
  info->n_nodes = P.n;
  info->hybrid_from = P.hyb;
  info->n_bands = P.hyb ? P.row->nb_fp : P.nb_fp;
  info->bp_bands = P.hyb ? P.row->nb : P.nb;
  info->fp_window_bytes = P.rc.fp_packed ? P.rc.fwin_bytes : P.rc.cache_bytes;
  info->mode = P.cfg.mode;
  info->dtype = P.cfg.dtype;
  info->out_h = P.shp[P.n - 1].h;
  info->out_w = P.shp[P.n - 1].w;
  info->out_c = P.shp[P.n - 1].c;
  info->workspace_bytes = P.hyb ? P.h_total : P.rc.total;
  info->layerwise_workspace_bytes = P.lw.total;
  info->strip_bytes = P.rc.strip_bytes;
  info->band_cache_bytes = P.rc.cache_bytes;
  info->delta_bytes = P.rc.delta_bytes;
  info->carry_bytes = P.rc.carry_bytes;
  info->partial_bytes = P.rc.part_bytes;
  double omega = 0;
  for (int v = 1; v < P.n; ++v) omega += (double)P.elems(v, P.shp[v].h) * P.es;
  double ybytes = (double)P.elems(P.n - 1, P.shp[P.n - 1].h) * P.es;
  info->omega_bytes = omega;
  info->omega_fp_bytes = (double)P.rc.strip_bytes + P.rc.part_bytes +
                         (P.rc.fp_packed ? P.rc.fwin_bytes : P.rc.cache_bytes) + ybytes;
  info->omega_bp_bytes = (double)(P.hyb ? P.h_total : P.rc.total) + ybytes;
  if (P.hyb) {
    // the row part's figures; the layer-wise part keeps whole maps
    const Plan &R = *P.row;
    info->strip_bytes = R.rc.strip_bytes;
    info->band_cache_bytes = R.rc.cache_bytes;
    info->delta_bytes = R.rc.delta_bytes;
    info->carry_bytes = R.rc.carry_bytes;
    info->partial_bytes = R.rc.part_bytes;
    info->fp_window_bytes = R.rc.fp_packed ? R.rc.fwin_bytes : R.rc.cache_bytes;
    info->omega_fp_bytes = (double)P.h_total + ybytes;
  }
  info->flops_tau = P.tau;
  info->flops_rows = P.flops_rows;
  info->flops_layerwise = 3.0 * P.tau;
  info->shared_rows = P.shared_rows;
  info->halo_rows = P.halo_rows;
  return LRCNN_OK;
}

extern "C" int lrcnn_plan_node_shape(const lrcnn_plan_t *plan, int32_t node,
                                     int32_t shape[3]) {
  if (!plan || !shape) return lrcnn_fail(LRCNN_EINVAL, "null argument");
  const Plan &P = *reinterpret_cast<const Plan *>(plan);
  if (node < 0 || node >= P.n) return lrcnn_fail(LRCNN_EINVAL, "node out of range");
  shape[0] = P.shp[node].h;
  shape[1] = P.shp[node].w;
  shape[2] = P.shp[node].c;
  return LRCNN_OK;
}

extern "C" int lrcnn_plan_band_rows(const lrcnn_plan_t *plan, int32_t phase, int32_t band,
                                    int32_t node, int32_t rows[4]) {
  if (!plan || !rows) return lrcnn_fail(LRCNN_EINVAL, "null argument");
  const Plan &P = *reinterpret_cast<const Plan *>(plan);
  const int nbands = phase == 0 ? P.nb_fp : P.nb;
  if (node < 0 || node >= P.n || band < 0 || band >= nbands || (phase != 0 && phase != 1))
    return lrcnn_fail(LRCNN_EINVAL, "phase, band or node out of range");
  lrcnn::Rows q = phase == 0 ? P.rows_fp[band][node] : P.rows[band][node];
  if (P.hyb) {
    // hybrid: the row part's bands; layer-wise nodes are whole in band 0
    if (node < P.hyb) {
      const Plan &R = *P.row;
      const int rb = phase == 0 ? R.nb_fp : R.nb;
      if (band >= rb) return lrcnn_fail(LRCNN_EINVAL, "band out of range");
      q = phase == 0 ? R.rows_fp[band][node] : R.rows[band][node];
    } else {
      const int h = band == 0 ? P.shp[node].h : 0;
      q = lrcnn::Rows{0, h, 0, h};
    }
  }
  rows[0] = q.a;
  rows[1] = q.b;
  rows[2] = q.lo;
  rows[3] = q.hi;
  return LRCNN_OK;
}

extern "C" void lrcnn_plan_destroy(lrcnn_plan_t *plan) {
  if (!plan) return;
  Plan *p = reinterpret_cast<Plan *>(plan);
  if (p->row) release_side(*p->row);
  if (p->col) release_side(*p->col);
  release_side(*p);
  delete p;
}

namespace lrcnn {

// The xi of Eqs. (9)-(10): device bytes of a step outside the workspace.
static size_t other_bytes(const Plan &P, bool want_dx) {
  const size_t es = (size_t)P.es;
  size_t t = 0;
  const size_t xb = P.elems(0, P.shp[0].h) * es;
  const size_t yb = P.elems(P.n - 1, P.shp[P.n - 1].h) * es;
  t += align256(xb) + 2 * align256(yb);  // x, y, dy
  if (want_dx) t += align256(xb);
  for (int v = 1; v < P.n; ++v) {
    const lrcnn_node &d = P.nodes[v];
    if (d.op != LRCNN_OP_CONV) continue;
    const size_t wn = (size_t)d.c_out * d.kh * d.kw * P.shp[d.in0].c;
    t += align256(wn * es) + align256(wn * 4);  // weights, float32 dW
    if (d.affine) t += 2 * align256((size_t)d.c_out * 4);
  }
  return t;
}

static size_t step_bytes(const Plan &P, bool layerwise, bool want_dx) {
  return (layerwise ? P.lw.total : (P.hyb ? P.h_total : P.rc.total)) + other_bytes(P, want_dx);
}

}  // namespace lrcnn

extern "C" int lrcnn_plan_step_bytes(const lrcnn_plan_t *plan, int32_t layerwise,
                                     int32_t want_dx, size_t *bytes) {
  if (!plan || !bytes) return lrcnn_fail(LRCNN_EINVAL, "null plan or output");
  *bytes = lrcnn::step_bytes(*reinterpret_cast<const Plan *>(plan), layerwise != 0,
                             want_dx != 0);
  return LRCNN_OK;
}

extern "C" int lrcnn_plan_for_budget(const lrcnn_node *nodes, int32_t n_nodes,
                                     const lrcnn_config *cfg, const lrcnn_budget *budget,
                                     lrcnn_plan_t **out) {
  if (!out) return lrcnn_fail(LRCNN_EINVAL, "null output pointer");
  *out = nullptr;
  if (!nodes || !cfg || !budget) return lrcnn_fail(LRCNN_EINVAL, "null argument");
  if (cfg->policy == LRCNN_EXPLICIT)
    return lrcnn_fail(LRCNN_EINVAL,
                      "the budget search takes the EVEN, BALANCED or PAPER_2PS policy");
  if (budget->max_bands < 0 || budget->max_refine < 0 || budget->max_refine > 64)
    return lrcnn_fail(LRCNN_EINVAL, "max_bands must be >= 0 and max_refine in [0, 64]");
  lrcnn_config c = *cfg;
  c.n_bands = 1;
  c.bp_refine = 1;
  c.bounds = nullptr;
  // shapes from a one-band plan give the partitioned height
  lrcnn_plan_t *probe = nullptr;
  int st = lrcnn_plan(nodes, n_nodes, &c, &probe);
  if (st != LRCNN_OK) return st;
  const Plan &P1 = *reinterpret_cast<const Plan *>(probe);
  const int H = c.mode == LRCNN_CARRY ? P1.shp[0].h : P1.shp[P1.n - 1].h;
  const bool fits1 = lrcnn::step_bytes(P1, false, budget->want_dx != 0) <= budget->budget_bytes;
  if (fits1) {
    *out = probe;
    return LRCNN_OK;
  }
  const int HL_probe = P1.shp[P1.n - 1].h;
  lrcnn_plan_destroy(probe);
  const int maxb = budget->max_bands > 0 ? std::min(budget->max_bands, H) : std::min(256, H);
  const int maxr = budget->max_refine > 1 ? budget->max_refine : 1;
  // PAPER_2PS (Eq. (12)): for each N_BP the largest H_1^L whose step fits,
  // from all H_L rows in the first band down to an even share
  const int HL = HL_probe;
  for (int nbp = 2; nbp <= maxb; ++nbp) {
    for (int nfp = 1; nfp <= nbp; ++nfp) {
      if (nbp % nfp != 0 || nbp / nfp > maxr) continue;
      c.n_bands = nfp;
      c.bp_refine = nbp / nfp;
      const bool paper = c.policy == LRCNN_PAPER_2PS;
      const int h_lo = paper ? (HL + nbp - 1) / nbp : 0;
      for (int h1 = paper ? HL : 0; h1 >= h_lo; --h1) {
        c.first_rows = h1;
        lrcnn_plan_t *p = nullptr;
        st = lrcnn_plan(nodes, n_nodes, &c, &p);
        if (st != LRCNN_OK) return st;
        if (lrcnn::step_bytes(*reinterpret_cast<const Plan *>(p), false,
                              budget->want_dx != 0) <= budget->budget_bytes) {
          *out = p;
          return LRCNN_OK;
        }
        lrcnn_plan_destroy(p);
      }
    }
  }
  return lrcnn_fail(LRCNN_EINFEASIBLE, "no plan with at most " + std::to_string(maxb) +
                                           " backward bands fits " +
                                           std::to_string(budget->budget_bytes) + " bytes");
}

extern "C" int lrcnn_max_batch(const lrcnn_node *nodes, int32_t n_nodes,
                               const lrcnn_config *cfg, int32_t layerwise,
                               const lrcnn_budget *budget, int32_t *batch) {
  if (!nodes || !cfg || !budget || !batch) return lrcnn_fail(LRCNN_EINVAL, "null argument");
  *batch = 0;
  lrcnn_config c = *cfg;
  // 1: fits, 0: does not fit, < 0: planner error
  auto fits = [&](int b) -> int {
    c.batch = b;
    lrcnn_plan_t *p = nullptr;
    const int st = lrcnn_plan(nodes, n_nodes, &c, &p);
    if (st != LRCNN_OK) return st;
    const bool ok = lrcnn::step_bytes(*reinterpret_cast<const Plan *>(p), layerwise != 0,
                                      budget->want_dx != 0) <= budget->budget_bytes;
    lrcnn_plan_destroy(p);
    return ok ? 1 : 0;
  };
  int f = fits(1);
  if (f < 0) return f;
  if (f == 0)
    return lrcnn_fail(LRCNN_EINFEASIBLE, "a batch of one does not fit " +
                                             std::to_string(budget->budget_bytes) + " bytes");
  int lo = 1, hi = 2;  // lo fits; hi is the next candidate above it
  const int cap = 1 << 24;
  for (;;) {
    if (hi > cap) {
      *batch = lo;
      return LRCNN_OK;
    }
    f = fits(hi);
    if (f < 0) return f;
    if (f == 0) break;
    lo = hi;
    hi *= 2;
  }
  while (hi - lo > 1) {  // fits(lo) == 1, fits(hi) == 0
    const int mid = lo + (hi - lo) / 2;
    f = fits(mid);
    if (f < 0) return f;
    (f ? lo : hi) = mid;
  }
  *batch = lo;
  return LRCNN_OK;
}
