// Band executor: walks the plan's bands and nodes and enqueues the kernels
// of kernels.hip on the caller's stream. Implements the three entry points
// lrcnn_forward_rows, lrcnn_backward_rows and
// lrcnn_layerwise_reference_gpu (Algorithm 1 and its column baseline).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <string>
#include <vector>

#include "kernels.hpp"
#include "plan.hpp"

namespace lrcnn {
namespace {

enum Sched { S_CARRY, S_RECOMPUTE, S_LAYERWISE };

// Dry-run mode (test hook): the executor walks the schedule and runs every
// host-side check but enqueues nothing, so it runs without a GPU.
thread_local bool g_dry = false;
// forward bands one after another (the pipelined forward is opt-in: a
// ResNet-50 bfloat16 graph-captured run with it ended in an abort whose
// cause is not yet known)
thread_local bool g_no_fp_pipe = true;
thread_local bool g_serial_wg = false;

#define LAUNCH(call, what)                                                 \
  do {                                                                     \
    int e_ = g_dry ? 0 : (call);                                           \
    if (e_ != 0)                                                           \
      return lrcnn_fail(LRCNN_EHIP, std::string(what) + ": " +             \
                                        hipGetErrorString((hipError_t)e_)); \
  } while (0)

// The weight gradient of a convolution does not depend on the input
// gradient of the same layer, and a band's launches of either are often too
// small to fill the GPU, so the backward runs the weight gradients on a side
// stream beside the caller's stream. Events order them: the side stream
// waits until the error operand is formed; the caller's stream waits for the
// last weight gradient before the error-operand buffer is formed again and
// at the end of every band (the next band's recompute overwrites the
// windows the weight gradient reads).
bool ensure_side(Plan &P) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return false;
  if (P.side_stream && P.side_dev == dev) return true;
  release_side(P);
  hipStream_t s = nullptr;
  hipEvent_t a = nullptr, b = nullptr;
  if (hipStreamCreateWithFlags(&s, hipStreamNonBlocking) != hipSuccess) return false;
  if (hipEventCreateWithFlags(&a, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&b, hipEventDisableTiming) != hipSuccess) {
    if (a) (void)hipEventDestroy(a);
    (void)hipStreamDestroy(s);
    return false;
  }
  P.side_stream = s;
  P.ev_act = a;
  P.ev_wg = b;
  P.side_dev = dev;
  return true;
}

// Events of the pipelined forward pass (created once per plan and device,
// with the side stream).
bool ensure_fp_events(Plan &P) {
  if ((int)P.ev_fp.size() == 2 * P.n && P.ev_fork) return true;
  for (void *e : P.ev_fp)
    if (e) (void)hipEventDestroy((hipEvent_t)e);
  P.ev_fp.assign(2 * P.n, nullptr);
  for (auto &e : P.ev_fp) {
    hipEvent_t h = nullptr;
    if (hipEventCreateWithFlags(&h, hipEventDisableTiming) != hipSuccess) return false;
    e = h;
  }
  if (!P.ev_fork) {
    hipEvent_t h = nullptr;
    if (hipEventCreateWithFlags(&h, hipEventDisableTiming) != hipSuccess) return false;
    P.ev_fork = h;
  }
  return true;
}

struct Run {
  Plan &P;
  const Layout &L;
  Sched sched;
  const Fuse &F;  // the schedule's fusions
  char *ws;
  const void *x;
  const void *const *w;
  const float *const *sc;
  const float *const *sf;
  void *stream;
  int dt;
  std::vector<View> act;   // current feature-map view of every node
  std::vector<View> dlt;   // current float32 error view of every node
  std::vector<int> first_consumer;
  std::vector<char> dw_set;  // per conv: a band has written its weight gradient
  // per node: its error window is initialized by the pending input gradient
  // (with the carried rows in dinit_cv from row dinit_t when dinit_carry)
  std::vector<char> dinit, dinit_carry;
  // per conv: its error operand (and carry) were formed by its consumer's
  // input gradient in this band (no activation-backward pass)
  std::vector<char> act_done;
  std::vector<View> dinit_cv;
  std::vector<int> dinit_t;
  hipStream_t side = nullptr;  // weight-gradient stream (backward only)
  bool wg_pending = false;     // a weight gradient on `side` not yet joined
  bool dx_f32 = false;         // store dL/dx as float32 (a checkpoint's error)
  // forward pass pipelined over bands (two streams by band parity): band r's
  // step of node v waits until band r-1 has finished every step that reads
  // the windows this step writes, and records ev_cur[v]
  bool pipe = false;
  hipEvent_t *ev_cur = nullptr, *ev_prev = nullptr;
  size_t part_off = 0;  // split-K partial sums of this band's stream

  Run(Plan &p, const Layout &l, Sched s, void *wsp, const void *x_,
      const void *const *w_, const float *const *sc_, const float *const *sf_,
      void *st)
      : P(p), L(l), sched(s), F(s == S_LAYERWISE ? p.fz_lw : p.fz), ws((char *)wsp), x(x_), w(w_), sc(sc_), sf(sf_),
        stream(st), dt(p.cfg.dtype == LRCNN_BF16 ? DT_BF16 : DT_F32) {
    act.resize(P.n);
    dlt.resize(P.n);
    first_consumer.assign(P.n, -1);
    dinit.assign(P.n, 0);
    dinit_carry.assign(P.n, 0);
    dinit_cv.assign(P.n, View{});
    dinit_t.assign(P.n, 0);
    act_done.assign(P.n, 0);
    for (int v = 0; v < P.n; ++v)
      for (int c : P.cons[v]) first_consumer[v] = std::max(first_consumer[v], c);
    const Shape &s0 = P.shp[0];
    act[0] = View{const_cast<void *>(x), (long long)s0.h * s0.w * s0.c, 0, s0.w, s0.c, s0.h};
    part_off = L.part;
  }

  // last step (node index) of a band that reads node v's window
  int last_reader(int v) const {
    int c = v;
    for (int k : P.cons[v]) c = std::max(c, k);
    return c;
  }
  // the windows node v's step writes (its own, and the residual add's when
  // the conv computes it) are no longer read by the previous band
  int pipe_wait(int v) {
    if (!pipe || !ev_prev) return LRCNN_OK;
    int w = last_reader(v);
    if (F.fwd[v]) w = std::max(w, last_reader(F.fwd[v]));
    LAUNCH(hipStreamWaitEvent((hipStream_t)stream, ev_prev[w], 0), "band wait");
    return LRCNN_OK;
  }
  int pipe_record(int v) {
    if (!pipe) return LRCNN_OK;
    LAUNCH(hipEventRecord(ev_cur[v], (hipStream_t)stream), "band record");
    return LRCNN_OK;
  }

  View full(void *p, int v) const {
    const Shape &s = P.shp[v];
    return View{p, (long long)s.h * s.w * s.c, 0, s.w, s.c, s.h};
  }
  View win(size_t off, int v, int cap, int row0) const {
    const Shape &s = P.shp[v];
    return View{ws + off, (long long)cap * s.w * s.c, row0, s.w, s.c, cap};
  }
  // Host-side guard: every row a launch touches must be held by its view,
  // so a planning error is reported instead of reaching the GPU.
  static bool holds(const View &v, int r0, int r1) {
    return r1 <= r0 || (r0 >= v.row0 && r1 <= v.row0 + v.rows);
  }
  // rows of the producer read by output rows [a, b) of a windowed op
  static void in_rows(const lrcnn_node &d, int h_in, int a, int b, int &r0, int &r1) {
    if (d.op == LRCNN_OP_ADD) {
      r0 = a, r1 = b;
    } else {
      r0 = std::max(0, a * d.sh - d.ph);
      r1 = std::min(h_in, (b - 1) * d.sh - d.ph + d.kh);
    }
  }

  // Forward of node v over rows [a, b) into `dst`.
  // `res` (conv only, nullable view): the residual add fused into the
  // epilogue; dst and mask are then the add's, res_relu its ReLU
  int node_fwd(int v, int a, int b, View dst, uint8_t *am, uint8_t *mask,
               const View *res = nullptr, int res_relu = 0) {
    if (b <= a) return LRCNN_OK;
    const lrcnn_node &d = P.nodes[v];
    const Shape &sv = P.shp[v], &su = P.shp[d.in0];
    const int B = P.cfg.batch;
    {
      int r0, r1;
      in_rows(d, su.h, a, b, r0, r1);
      bool ok = holds(dst, a, b) && holds(act[d.in0], r0, r1) && (!res || holds(*res, a, b));
      if (d.op == LRCNN_OP_ADD) ok = ok && holds(act[d.in1], r0, r1);
      if (!ok)
        return lrcnn_fail(LRCNN_EINVAL, "internal: band rows of node " + std::to_string(v) +
                                            " not held by its buffers");
    }
    if (d.op == LRCNN_OP_CONV) {
      ConvArgs c{};
      c.src = act[d.in0];
      c.dst = dst;
      c.w = w[v];
      c.scale = d.affine ? sc[v] : nullptr;
      c.shift = d.affine ? sf[v] : nullptr;
      c.relu = d.relu;
      c.mask = mask;
      c.mask_h = sv.h;
      c.B = B;
      c.y0 = a;
      c.y1 = b;
      c.Wd = sv.w;
      c.N = sv.c;
      c.KC = su.c;
      c.Hs = su.h;
      c.Ws = su.w;
      c.sy0 = 0;
      c.sy1 = su.h;
      c.kh = d.kh, c.kw = d.kw, c.sh = d.sh, c.sw = d.sw, c.ph = d.ph, c.pw = d.pw;
      c.part = (float *)(ws + part_off);
      c.part_bytes = L.part_bytes;
      c.splits = P.fsplit[v];
      if (res) {
        c.res = *res;
        c.res_relu = res_relu;
      }
      // (a layer-wise launch whose partial sums exceed the buffer runs in row
      // chunks; each output element's sum is the same)
      const int chunk = L.fchunk.empty() || L.fchunk[v] <= 0 ? b - a : L.fchunk[v];
      for (int y = a; y < b; y += chunk) {
        c.y0 = y;
        c.y1 = std::min(b, y + chunk);
        LAUNCH(launch_conv(dt, 0, c, stream), "conv forward");
      }
    } else if (d.op == LRCNN_OP_MAXPOOL) {
      PoolArgs p{};
      p.src = act[d.in0];
      p.dst = dst;
      p.am = am;
      p.mask = mask;
      p.mask_h = sv.h;
      p.B = B;
      p.y0 = a;
      p.y1 = b;
      p.Wd = sv.w;
      p.C = sv.c;
      p.Hs = su.h;
      p.Ws = su.w;
      p.kh = d.kh, p.kw = d.kw, p.sh = d.sh, p.sw = d.sw, p.ph = d.ph, p.pw = d.pw;
      LAUNCH(launch_pool_fwd(dt, p, stream), "max-pool forward");
    } else {
      LAUNCH(launch_add_fwd(dt, act[d.in0], act[d.in1], dst, d.relu, mask, sv.h,
                            B, a, b, sv.w, sv.c, stream),
             "add forward");
    }
    return LRCNN_OK;
  }

  // Compute the feature maps of band `r` for every node (FP, or the BP
  // recompute of Algorithm 1). The output node goes to `y` when given.
  // Feature maps of one band for every node: the forward pass (bp = false,
  // forward band r) or the BP recompute (bp = true, backward band r) of
  // Algorithm 1. The output node goes to `y` when given.
  // `keep`: the band's maps stay in the window buffers for the BP that
  // follows (the output node is computed into its window and copied to y,
  // pool argmax bytes are recorded), so BP can skip recomputing this band.
  // `views_only`: set the band's views without launching anything (the
  // maps are already in place).
  // Copies of one band's strips. Unless the forward windows are packed by
  // lifetime, every node has a window of its own, so all strip loads of a
  // band can run in one launch before its first node and all strip stores
  // in one launch after its last; otherwise each copy runs at its node.
  int flush_copies(std::vector<CopySeg> &segs, const char *what) {
    for (size_t i = 0; i < segs.size(); i += kMaxCopySegs) {
      const int cnt = (int)std::min<size_t>(kMaxCopySegs, segs.size() - i);
      LAUNCH(launch_rows_copy_batch(dt, segs.data() + i, cnt, stream), what);
    }
    segs.clear();
    return LRCNN_OK;
  }
  int strip_copy(bool batch, std::vector<CopySeg> &segs, View src, View dst, int r0, int r1,
                 int v, const char *what) {
    if (batch) {
      segs.push_back(CopySeg{src, dst, P.cfg.batch, r0, r1, P.shp[v].w, P.shp[v].c});
      return LRCNN_OK;
    }
    LAUNCH(launch_rows_copy(dt, dt, src, dst, 0, P.cfg.batch, r0, r1, P.shp[v].w, P.shp[v].c,
                            stream),
           what);
    return LRCNN_OK;
  }

  int band_fwd(int r, void *y, void *const *mask_out, bool bp, bool keep = false,
               bool views_only = false) {
    const int n = P.n;
    const bool fp = !bp && sched != S_LAYERWISE;
    const bool packed = fp && L.fp_packed;
    // (pipelined: strips loaded and stored at each node's own step)
    const bool batch = !packed && !(fp && pipe);
    std::vector<CopySeg> segs;
    int st;
    // views of every node's rows, and the strip loads
    for (int v = 1; v < n; ++v) {
      const Rows q = fp ? P.rows_fp[r][v] : band_rows(r, v);
      View dst;
      if (v == n - 1 && y && !keep) {
        dst = full(y, v);
      } else if (packed) {
        dst = win(L.fwin[v], v, L.fwin_cap[v], q.lo);
      } else {
        dst = win(L.win[v], v, L.win_cap[v], q.lo);
      }
      act[v] = dst;
      if (views_only) continue;
      if (sched == S_CARRY && r > 0 && q.a > q.lo && batch) {
        // rows shared from earlier bands (two-phase sharing): kept at the
        // backward boundary that ends where this band starts
        const int sidx = fp ? r * P.refine - 1 : r - 1;
        View strip = win(L.strip[sidx][v], v, q.a - q.lo, q.lo);
        if (!holds(strip, P.tail[sidx][v], P.rows[sidx][v].b) || P.tail[sidx][v] != q.lo ||
            P.rows[sidx][v].b != q.a)
          return lrcnn_fail(LRCNN_EINVAL, "internal: strip rows do not match the band");
        if ((st = strip_copy(true, segs, strip, dst, q.lo, q.a, v, "strip load")) != LRCNN_OK)
          return st;
      }
    }
    if (views_only) return LRCNN_OK;
    if ((st = flush_copies(segs, "strip load")) != LRCNN_OK) return st;
    for (int v = 1; v < n; ++v) {
      const Rows q = fp ? P.rows_fp[r][v] : band_rows(r, v);
      const View dst = act[v];
      if (fp && (st = pipe_wait(v)) != LRCNN_OK) return st;
      if (sched == S_CARRY && r > 0 && q.a > q.lo && !batch) {
        const int sidx = fp ? r * P.refine - 1 : r - 1;
        View strip = win(L.strip[sidx][v], v, q.a - q.lo, q.lo);
        if (!holds(strip, P.tail[sidx][v], P.rows[sidx][v].b) || P.tail[sidx][v] != q.lo ||
            P.rows[sidx][v].b != q.a)
          return lrcnn_fail(LRCNN_EINVAL, "internal: strip rows do not match the band");
        if ((st = strip_copy(false, segs, strip, dst, q.lo, q.a, v, "strip load")) != LRCNN_OK)
          return st;
      }
      uint8_t *am = ((bp || keep) && P.nodes[v].op == LRCNN_OP_MAXPOOL)
                        ? (uint8_t *)(ws + L.argmax[v]) : nullptr;
      // (not with lifetime-packed forward windows: the add's window may
      // still belong to another node while the conv runs)
      const bool can_fuse = !packed;
      const int fa = can_fuse ? F.fwd[v] : 0;
      const lrcnn_node &nd = P.nodes[v];
      if (fa) {
        // this conv's epilogue computes the residual add fa (its only
        // consumer): output into the add's view, with the add's mask
        const lrcnn_node &an = P.nodes[fa];
        const View other = act[an.in0 == v ? an.in1 : an.in0];
        uint8_t *amk = mask_out ? (uint8_t *)mask_out[fa] : nullptr;
        if ((st = node_fwd(v, q.a, q.b, act[fa], am, amk, &other, an.relu)) != LRCNN_OK)
          return st;
      } else if (can_fuse && nd.op == LRCNN_OP_ADD && F.fwd[std::max(nd.in0, nd.in1)] == v) {
        // computed with its later input
      } else {
        uint8_t *mk = mask_out ? (uint8_t *)mask_out[v] : nullptr;
        if ((st = node_fwd(v, q.a, q.b, dst, am, mk)) != LRCNN_OK) return st;
      }
      if (v == n - 1 && y && keep)
        LAUNCH(launch_rows_copy(dt, dt, dst, full(y, v), 0, P.cfg.batch, q.a, q.b,
                                P.shp[v].w, P.shp[v].c, stream),
               "output store");
      if (sched == S_CARRY && fp && v != n - 1) {
        // keep the shared rows of every backward boundary inside this band
        for (int j = 0; j < P.refine; ++j) {
          const int sidx = r * P.refine + j;
          if (sidx + 1 >= P.nb) break;
          const int t = P.tail[sidx][v], e = P.rows[sidx][v].b;
          if (e <= t) continue;
          View strip = win(L.strip[sidx][v], v, e - t, t);
          if (!holds(dst, t, e))
            return lrcnn_fail(LRCNN_EINVAL, "internal: strip rows not in the band window");
          if ((st = strip_copy(batch, segs, dst, strip, t, e, v, "strip store")) != LRCNN_OK)
            return st;
        }
      }
      if (fp && (st = pipe_record(v)) != LRCNN_OK) return st;
    }
    return flush_copies(segs, "strip store");
  }

  Rows band_rows(int r, int v) const {
    if (sched == S_LAYERWISE) return Rows{0, P.shp[v].h, 0, P.shp[v].h};
    return P.rows[r][v];
  }

  // Error window of node u for band r: its view, and, in CARRY mode, the
  // rows [t, b) whose error band r+1 carried (returns false if none).
  // carry buffer of node u written by band `band` (and read by band - 1):
  // a node with two buffers alternates them by band parity
  char *carry_ptr(int u, int band) const {
    return ws + ((band & 1) && L.carry2[u] ? L.carry2[u] : L.carry[u]);
  }

  bool delta_view(int r, int u, View &cv, int &t) {
    const Rows q = band_rows(r, u);
    const Shape &s = P.shp[u];
    dlt[u] = win(L.delta[u], u, L.win_cap[u], q.lo);
    if (sched == S_CARRY && r + 1 < P.nb) {
      t = P.tail[r][u];
      if (q.b > t) {
        cv = View{carry_ptr(u, r + 1), (long long)L.carry_cap[u] * s.w * s.c, t, s.w, s.c,
                  L.carry_cap[u]};
        return true;
      }
    }
    return false;
  }

  // When v's backward launch (rows [y0, y1) of u) completes u's error and v
  // is u's only consumer, the launch forms u's error operand and carried
  // rows itself (eo). With two carry buffers (band parity) it writes the
  // carried-out rows into this band's buffer while it reads the rows carried
  // in from the other; with one, they are staged in u's error window and
  // moved to `stage` (u's carry buffer) after the launch, which reads the
  // rows carried in from that buffer. stage_a = 0 when nothing is staged.
  int fuse_err(int r, int v, int u, int y0, int y1, ErrOut &eo, View &stage, int &stage_a) {
    stage_a = 0;
    if (F.act[u] != v) return LRCNN_OK;
    const Rows qu = band_rows(r, u);
    const lrcnn_node &du = P.nodes[u];
    const Shape &sh = P.shp[u];
    if (qu.hi != qu.b || y0 != qu.lo || y1 != qu.b)
      return lrcnn_fail(LRCNN_EINVAL, "internal: fused error operand rows");
    const int oa = std::max(qu.a, qu.lo);
    eo.fact = 1;
    eo.fa = oa;
    eo.dc = View{ws + L.dc[u], (long long)(qu.b - oa) * sh.w * sh.c, oa, sh.w, sh.c, qu.b - oa};
    eo.z = act[u];
    eo.relu = du.relu;
    eo.scale = du.affine ? sc[u] : nullptr;
    if (oa < qu.b && !holds(act[u], oa, qu.b))
      return lrcnn_fail(LRCNN_EINVAL, "internal: activation rows not held");
    if (oa > qu.lo) {
      if (sched != S_CARRY || r == 0)
        return lrcnn_fail(LRCNN_EINVAL, "internal: rows below a band without carry");
      stage = View{carry_ptr(u, r), (long long)L.carry_cap[u] * sh.w * sh.c, qu.lo, sh.w, sh.c,
                   L.carry_cap[u]};
      if (L.carry2[u]) {
        // the rows carried in come from the other parity's buffer: the
        // launch writes the carried-out rows straight into this band's
        eo.carry = stage;
        if (!holds(eo.carry, qu.lo, oa))
          return lrcnn_fail(LRCNN_EINVAL, "internal: carry rows not held");
      } else {
        eo.carry = View{ws + L.delta[u], (long long)L.carry_cap[u] * sh.w * sh.c, qu.lo, sh.w,
                        sh.c, L.carry_cap[u]};
        if (!holds(eo.carry, qu.lo, oa) || !holds(stage, qu.lo, oa))
          return lrcnn_fail(LRCNN_EINVAL, "internal: carry rows not held");
        stage_a = oa;
      }
    }
    act_done[u] = 1;
    return LRCNN_OK;
  }
  int unstage(int r, int u, const ErrOut &eo, const View &stage, int stage_a) {
    if (!stage_a) return LRCNN_OK;
    const Shape &sh = P.shp[u];
    const Rows qu = band_rows(r, u);
    LAUNCH(launch_rows_copy(DT_F32, DT_F32, eo.carry, stage, 0, P.cfg.batch, qu.lo, stage_a,
                            sh.w, sh.c, stream),
           "carry store");
    return LRCNN_OK;
  }

  // The backward launch of v (a conv's input gradient, a max-pool's
  // backward) initializes u's error window itself (no zeroing pass) when it
  // writes every row of the window this band uses.
  bool init_by_dgrad(int r, int v, int u, bool want_dx) const {
    const lrcnn_node &d = P.nodes[v];
    if (u == 0 && !want_dx) return false;
    if (d.op == LRCNN_OP_ADD) {
      // the add's backward writes its own rows of each input (not when both
      // inputs are the same node: the second side adds to the first), and
      // the initial value of the window rows above them (a consumer with
      // later own rows, such as the next block's first conv, reaches them)
      const Rows qv = band_rows(r, v), qu = band_rows(r, u);
      return d.in0 != d.in1 && qv.b > qv.a && qv.a == qu.lo && qv.b <= qu.hi;
    }
    if (d.op != LRCNN_OP_CONV && d.op != LRCNN_OP_MAXPOOL) return false;
    const Rows qv = band_rows(r, v), qu = band_rows(r, u);
    if (qv.b <= qv.a) return false;
    const int y0 = std::max(0, qv.a * d.sh - d.ph);
    const int y1 = std::min(P.shp[u].h, (qv.b - 1) * d.sh - d.ph + d.kh);
    return y0 == qu.lo && y1 == qu.hi;
  }

  // Zero node u's error window for band r and bring in the error carried
  // from band r+1 (CARRY).
  int init_delta(int r, int u) {
    const Rows q = band_rows(r, u);
    const Shape &s = P.shp[u];
    dlt[u] = win(L.delta[u], u, L.win_cap[u], q.lo);
    if (sched == S_CARRY && r + 1 < P.nb) {
      const int t = P.tail[r][u];
      if (q.b > t) {
        // zero rows [lo, t), carried rows [t, b): one launch
        View cv = View{carry_ptr(u, r + 1), (long long)L.carry_cap[u] * s.w * s.c, t, s.w, s.c,
                       L.carry_cap[u]};
        if (!holds(cv, t, q.b) || !holds(dlt[u], q.lo, q.b) || q.b != q.hi)
          return lrcnn_fail(LRCNN_EINVAL, "internal: carry rows not held");
        LAUNCH(launch_rows_init(dlt[u], &cv, t, P.cfg.batch, q.lo, q.b, s.w, s.c, stream),
               "error window with carry");
        return LRCNN_OK;
      }
    }
    LAUNCH(launch_rows_zero(dlt[u], P.cfg.batch, q.lo, q.hi, s.w, s.c, stream), "zero error");
    return LRCNN_OK;
  }

  // Back-propagate node v's finished error rows [a, b) (Algorithm 1,
  // Get_error and g^l += Gradient).
  int node_bwd(int r, int v, float *const *dw, bool want_dx) {
    const Rows q = band_rows(r, v);
    const int a = q.a, b = q.b;
    if (b <= a) return LRCNN_OK;
    const lrcnn_node &d = P.nodes[v];
    const Shape &sv = P.shp[v];
    const int B = P.cfg.batch;
    const int u = d.in0;
    const Shape &su = P.shp[u];
    {
      int r0, r1;
      in_rows(d, su.h, a, b, r0, r1);
      bool ok = holds(act[v], a, b) && (fused(v) || holds(dlt[v], a, b)) &&
                holds(act[u], r0, r1) && (fused(u) || holds(dlt[u], r0, r1));
      if (d.op == LRCNN_OP_ADD)
        ok = ok && holds(act[d.in1], r0, r1) && (fused(d.in1) || holds(dlt[d.in1], r0, r1));
      if (!ok)
        return lrcnn_fail(LRCNN_EINVAL, "internal: backward rows of node " + std::to_string(v) +
                                            " not held by its buffers");
    }
    if (d.op == LRCNN_OP_CONV) {
      void *dc = ws + L.dc[v];
      // the rows carried to the previous band leave in the same launch
      View cv{};
      const bool carries = sched == S_CARRY && r > 0 && q.a > q.lo;
      if (carries) {
        cv = View{carry_ptr(v, r), (long long)L.carry_cap[v] * sv.w * sv.c, q.lo, sv.w, sv.c,
                  L.carry_cap[v]};
        if (!holds(cv, q.lo, q.a)) return lrcnn_fail(LRCNN_EINVAL, "internal: carry rows not held");
      }
      if (fused(v)) {
        // the add's backward already wrote this conv's error operand
        if (carries) return lrcnn_fail(LRCNN_EINVAL, "internal: fused conv carries rows");
      } else if (act_done[v]) {
        // the consumer's input gradient formed the error operand and carry
        act_done[v] = 0;
      } else {
        LAUNCH(launch_act_bwd(dt, dlt[v], act[v], d.affine ? sc[v] : nullptr, d.relu, dc, B, a,
                              b, sv.w, sv.c, stream, carries ? &cv : nullptr, q.lo, q.a),
               "error operand");
      }
      WgradArgs g{};
      g.dc = dc;
      g.src = act[u];
      float *wdst = dw[v];
      const bool padded = L.cpad && u == 0;
      if (padded) {
        // input rows of the band in channel-padded form
        const int r0 = std::max(0, a * d.sh - d.ph);
        const int r1 = std::min(su.h, (b - 1) * d.sh - d.ph + d.kh);
        if (r1 - r0 > L.xpad_cap) return lrcnn_fail(LRCNN_EINVAL, "internal: padded input rows");
        g.src = View{ws + L.xpad, (long long)L.xpad_cap * su.w * L.cpad, r0, su.w, L.cpad,
                     L.xpad_cap};
        LAUNCH(launch_pad_channels(dt, act[0], g.src, su.c, L.cpad, B, r0, r1, su.w, stream),
               "pad input channels");
        wdst = (float *)(ws + L.dwpad[v]);
      }
      g.out = (float *)(ws + L.wpart[v]);
      g.part_bytes = L.wpart_bytes[v];
      g.B = B;
      g.y0 = a;
      g.y1 = b;
      g.Wv = sv.w;
      g.Co = sv.c;
      g.Ci = padded ? L.cpad : su.c;
      g.Hs = su.h;
      g.Ws = su.w;
      g.kh = d.kh, g.kw = d.kw, g.sh = d.sh, g.sw = d.sw, g.ph = d.ph, g.pw = d.pw;
      g.overwrite = dw_set[v] ? 0 : 1;
      dw_set[v] = 1;
      if (side) {
        LAUNCH(hipEventRecord((hipEvent_t)P.ev_act, (hipStream_t)stream), "event record");
        LAUNCH(hipStreamWaitEvent(side, (hipEvent_t)P.ev_act, 0), "stream wait");
        LAUNCH(launch_wgrad(dt, g, wdst, side), "weight gradient");
        LAUNCH(hipEventRecord((hipEvent_t)P.ev_wg, side), "event record");
        wg_pending = true;
      } else {
        LAUNCH(launch_wgrad(dt, g, wdst, stream), "weight gradient");
      }
      if (u != 0 || want_dx) {
        ConvArgs c{};
        View stage{};  // carry buffer the staged carried-out rows go to
        int stage_a = 0;
        c.src = View{dc, (long long)(b - a) * sv.w * sv.c, a, sv.w, sv.c, b - a};
        c.dst = dlt[u];
        c.w = w[v];
        c.B = B;
        c.y0 = std::max(0, a * d.sh - d.ph);
        c.y1 = std::min(su.h, (b - 1) * d.sh - d.ph + d.kh);
        c.Wd = su.w;
        c.N = su.c;
        c.KC = sv.c;
        c.Hs = sv.h;
        c.Ws = sv.w;
        c.sy0 = a;
        c.sy1 = b;
        c.kh = d.kh, c.kw = d.kw, c.sh = d.sh, c.sw = d.sw, c.ph = d.ph, c.pw = d.pw;
        c.part = (float *)(ws + L.part);
        c.part_bytes = L.part_bytes;
        if (dinit[u]) {
          // this launch writes every row of u's window: no zeroing pass
          c.dst_init = 1;
          if (dinit_carry[u]) {
            if (!holds(dinit_cv[u], dinit_t[u], band_rows(r, u).b))
              return lrcnn_fail(LRCNN_EINVAL, "internal: carry rows not held");
            c.cinit = dinit_cv[u];
            c.cinit_t = dinit_t[u];
          }
          dinit[u] = 0;
          // the launch completes u's error: it forms u's error operand and
          // carry itself when v is u's only consumer
          if (int e = fuse_err(r, v, u, c.y0, c.y1, c.eo, stage, stage_a)) return e;
        }
        LAUNCH(launch_conv(dt, 1, c, stream), "input gradient");
        if (int e = unstage(r, u, c.eo, stage, stage_a)) return e;
      }
    } else if (d.op == LRCNN_OP_MAXPOOL) {
      PoolBwdArgs p{};
      p.dv = dlt[v];
      p.du = dlt[u];
      p.am = (const uint8_t *)(ws + L.argmax[v]);
      p.B = B;
      p.y0 = a;
      p.y1 = b;
      p.Wv = sv.w;
      p.C = sv.c;
      p.ua = std::max(0, a * d.sh - d.ph);
      p.ub = std::min(su.h, (b - 1) * d.sh - d.ph + d.kh);
      p.Wu = su.w;
      p.kh = d.kh, p.kw = d.kw, p.sh = d.sh, p.sw = d.sw, p.ph = d.ph, p.pw = d.pw;
      View stage{};
      int stage_a = 0;
      if (dinit[u]) {
        // this launch writes every row of u's window: no zeroing pass
        p.dst_init = 1;
        if (dinit_carry[u]) {
          if (!holds(dinit_cv[u], dinit_t[u], band_rows(r, u).b))
            return lrcnn_fail(LRCNN_EINVAL, "internal: carry rows not held");
          p.cinit = dinit_cv[u];
          p.cinit_t = dinit_t[u];
        }
        dinit[u] = 0;
        if (int e = fuse_err(r, v, u, p.ua, p.ub, p.eo, stage, stage_a)) return e;
      }
      LAUNCH(launch_pool_bwd(dt, p, stream), "max-pool backward");
      if (int e = unstage(r, u, p.eo, stage, stage_a)) return e;
    } else {
      AddSide side_in[2];
      const int in_ids[2] = {d.in0, d.in1};
      for (int k = 0; k < 2; ++k) {
        const int x = in_ids[k];
        AddSide &sd = side_in[k];
        sd = AddSide{dlt[x], nullptr, nullptr, sv.c, 0, View{}, 0, 0};
        if (dinit[x]) {
          // this launch writes every row of x's window: no zeroing pass
          const Rows qx = band_rows(r, x);
          sd.init = 1;
          sd.init_hi = qx.hi;
          if (dinit_carry[x]) {
            if ((qx.hi > b && qx.b != qx.hi) || !holds(dinit_cv[x], dinit_t[x], qx.b))
              return lrcnn_fail(LRCNN_EINVAL, "internal: carry rows not held");
            sd.cinit = dinit_cv[x];
            sd.cinit_t = dinit_t[x];
          }
          dinit[x] = 0;
        }
        if (fused(x)) {
          // own rows of the conv input equal the add's rows (1 x 1 window)
          const Rows qx = band_rows(r, x);
          if (qx.a != a || qx.b != b)
            return lrcnn_fail(LRCNN_EINVAL, "internal: fused conv rows differ from the add's");
          sd.dc = ws + L.dc[x];
          sd.scale = P.nodes[x].affine ? sc[x] : nullptr;
        }
      }
      LAUNCH(launch_add_bwd(dt, dlt[v], act[v], side_in[0], side_in[1], d.relu, B, a, b, sv.w,
                            sv.c, stream),
             "add backward");
    }
    return LRCNN_OK;
  }

  // a conv whose error operand the add's backward writes (no error window)
  bool fused(int u) const {
    return u > 0 && u < (int)F.add.size() && F.add[u] != 0;
  }

  // BP of band r after its feature maps are in place.
  int band_bwd(int r, const void *dy, float *const *dw, void *dx, float *dxacc) {
    const int n = P.n, B = P.cfg.batch;
    const bool want_dx = dx != nullptr;
    std::fill(act_done.begin(), act_done.end(), 0);
    // seed: the band's own rows of dL/dy
    {
      const Rows q = band_rows(r, n - 1);
      int st = init_delta(r, n - 1);
      if (st != LRCNN_OK) return st;
      const Shape &s = P.shp[n - 1];
      LAUNCH(launch_rows_copy(P.dy_f32 ? DT_F32 : dt, DT_F32, full(const_cast<void *>(dy), n - 1),
                              dlt[n - 1], 0, B, q.a, q.b, s.w, s.c, stream),
             "seed error");
    }
    for (int v = n - 1; v >= 1; --v) {
      const lrcnn_node &d = P.nodes[v];
      // a conv's step starts by joining the previous weight gradient: its
      // error operand and partial sums live in arena space this step reuses
      if (side && wg_pending && d.op == LRCNN_OP_CONV) {
        LAUNCH(hipStreamWaitEvent((hipStream_t)stream, (hipEvent_t)P.ev_wg, 0), "stream join");
        wg_pending = false;
      }
      int ins[2] = {d.in0, d.op == LRCNN_OP_ADD ? d.in1 : -1};
      for (int u : ins)
        if (u >= 0 && first_consumer[u] == v && !fused(u)) {
          if (u == 0 && !want_dx && P.nodes[v].op == LRCNN_OP_CONV) {
            // nothing reads the input's error: only its view is needed
            View cv;
            int t = 0;
            delta_view(r, u, cv, t);
            continue;
          }
          if (init_by_dgrad(r, v, u, want_dx)) {
            dinit[u] = 1;
            dinit_carry[u] = delta_view(r, u, dinit_cv[u], dinit_t[u]) ? 1 : 0;
            continue;
          }
          if (F.act[u] == v) {
            // v's input gradient forms u's error operand; a band without
            // rows of v holds nothing of u (the planner checked), and u's
            // error window has no memory of its own
            const Rows qu = band_rows(r, u);
            if (qu.b > qu.a || qu.lo != qu.a)
              return lrcnn_fail(LRCNN_EINVAL, "internal: fused error operand without launch");
            View cv;
            int t = 0;
            delta_view(r, u, cv, t);
            continue;
          }
          int st = init_delta(r, u);
          if (st != LRCNN_OK) return st;
        }
      int st = node_bwd(r, v, dw, want_dx);
      if (st != LRCNN_OK) return st;
      // a conv's carried rows left with its error operand, unless the band
      // owns none of its rows (node_bwd then launches nothing)
      const Rows qv = band_rows(r, v);
      if (sched == S_CARRY && r > 0 && (d.op != LRCNN_OP_CONV || qv.b <= qv.a) &&
          !act_done[v]) {
        const Rows q = band_rows(r, v);
        if (q.a > q.lo) {
          const Shape &s = P.shp[v];
          View cv{carry_ptr(v, r), (long long)L.carry_cap[v] * s.w * s.c, q.lo, s.w, s.c,
                  L.carry_cap[v]};
          if (!holds(cv, q.lo, q.a)) return lrcnn_fail(LRCNN_EINVAL, "internal: carry rows not held");
          LAUNCH(launch_rows_copy(DT_F32, DT_F32, dlt[v], cv, 0, B, q.lo, q.a, s.w, s.c, stream),
                 "carry store");
        }
      }
    }
    // the next band's recompute overwrites the windows the weight
    // gradients read
    if (side && wg_pending) {
      LAUNCH(hipStreamWaitEvent((hipStream_t)stream, (hipEvent_t)P.ev_wg, 0), "stream join");
      wg_pending = false;
    }
    // input gradient rows
    if (want_dx) {
      const Rows q = band_rows(r, 0);
      const Shape &s = P.shp[0];
      if (sched == S_RECOMPUTE) {
        View acc = dxacc ? full(dxacc, 0) : full(dx, 0);
        LAUNCH(launch_rows_copy(DT_F32, DT_F32, dlt[0], acc, 1, B, q.lo, q.hi, s.w, s.c, stream),
               "input gradient accumulate");
      } else {
        LAUNCH(launch_rows_copy(DT_F32, dx_f32 ? DT_F32 : dt, dlt[0], full(dx, 0), 0, B, q.a, q.b,
                                s.w, s.c, stream),
               "input gradient store");
        if (sched == S_CARRY && r > 0 && q.a > q.lo) {
          View cv{carry_ptr(0, r), (long long)L.carry_cap[0] * s.w * s.c, q.lo, s.w, s.c,
                  L.carry_cap[0]};
          if (!holds(cv, q.lo, q.a)) return lrcnn_fail(LRCNN_EINVAL, "internal: carry rows not held");
          LAUNCH(launch_rows_copy(DT_F32, DT_F32, dlt[0], cv, 0, B, q.lo, q.a, s.w, s.c, stream),
                 "carry store");
        }
      }
    }
    return LRCNN_OK;
  }

  // The first band that computes a conv's weight gradient writes it, later
  // bands add to it (Algorithm 1 resets g before the BP loop), so no
  // separate zeroing pass is needed.
  int begin_dw() {
    dw_set.assign(P.n, 0);
    return LRCNN_OK;
  }

  // first-layer weight gradients accumulated in channel-padded form
  int finish_dw(float *const *dw) {
    if (!L.cpad) return LRCNN_OK;
    if (side && wg_pending) {
      LAUNCH(hipStreamWaitEvent((hipStream_t)stream, (hipEvent_t)P.ev_wg, 0), "stream join");
      wg_pending = false;
    }
    for (int v = 1; v < P.n; ++v)
      if (P.nodes[v].op == LRCNN_OP_CONV && P.nodes[v].in0 == 0) {
        const lrcnn_node &d = P.nodes[v];
        const long long cnt = (long long)d.c_out * d.kh * d.kw * P.shp[0].c;
        LAUNCH(launch_compact_dw((const float *)(ws + L.dwpad[v]), dw[v], P.shp[0].c, L.cpad,
                                 cnt, stream),
               "first-layer dW");
      }
    return LRCNN_OK;
  }
};

bool misaligned(const void *p) { return ((uintptr_t)p & 15u) != 0; }

int check_params(const Plan &P, const void *x, const void *const *w, const float *const *sc,
                 const float *const *sf) {
  if (!x) return lrcnn_fail(LRCNN_EINVAL, "x is null");
  if (misaligned(x)) return lrcnn_fail(LRCNN_EINVAL, "x is not 16-byte aligned");
  if (!w) return lrcnn_fail(LRCNN_EINVAL, "weight array is null");
  for (int v = 1; v < P.n; ++v) {
    const lrcnn_node &d = P.nodes[v];
    if (d.op != LRCNN_OP_CONV) continue;
    if (!w[v] || misaligned(w[v]))
      return lrcnn_fail(LRCNN_EINVAL, "weights of node " + std::to_string(v) + " null or misaligned");
    if (d.affine && (!sc || !sf || !sc[v] || !sf[v]))
      return lrcnn_fail(LRCNN_EINVAL, "affine node " + std::to_string(v) + " needs scale and shift");
  }
  return LRCNN_OK;
}

int check_ws_bytes(size_t need, void *ws, size_t bytes) {
  if (!ws) return lrcnn_fail(LRCNN_EINVAL, "workspace is null");
  if (misaligned(ws)) return lrcnn_fail(LRCNN_EINVAL, "workspace is not 16-byte aligned");
  if (bytes < need)
    return lrcnn_fail(LRCNN_EWORKSPACE, "workspace needs " + std::to_string(need) +
                                            " bytes, got " + std::to_string(bytes));
  return LRCNN_OK;
}

int check_ws(const Layout &L, void *ws, size_t bytes) { return check_ws_bytes(L.total, ws, bytes); }

int check_dw(const Plan &P, float *const *dw) {
  if (!dw) return lrcnn_fail(LRCNN_EINVAL, "dw array is null");
  for (int v = 1; v < P.n; ++v)
    if (P.nodes[v].op == LRCNN_OP_CONV && (!dw[v] || misaligned(dw[v])))
      return lrcnn_fail(LRCNN_EINVAL, "dw of node " + std::to_string(v) + " null or misaligned");
  return LRCNN_OK;
}

uint64_t g_epoch = 0;

}  // namespace

void release_side(Plan &P) {
  for (void *e : P.ev_fp)
    if (e) (void)hipEventDestroy((hipEvent_t)e);
  P.ev_fp.clear();
  if (P.ev_fork) (void)hipEventDestroy((hipEvent_t)P.ev_fork);
  P.ev_fork = nullptr;
  if (P.ev_act) (void)hipEventDestroy((hipEvent_t)P.ev_act);
  if (P.ev_wg) (void)hipEventDestroy((hipEvent_t)P.ev_wg);
  if (P.side_stream) (void)hipStreamDestroy((hipStream_t)P.side_stream);
  P.ev_act = P.ev_wg = P.side_stream = nullptr;
  P.side_dev = -1;
}

namespace {

// Hybrid depth (2PS-H / OverL-H): the row-centric part writes the
// checkpoint map at full size; the layer-wise part reads it as its input.
int hybrid_forward(Plan &P, const void *x, const void *const *w, const float *const *sc,
                   const float *const *sf, void *y, char *ws, void *const *mask_out,
                   void *stream) {
  const int c = P.hyb - 1;
  P.fwd_workspace = nullptr;
  int st = lrcnn_forward_rows(reinterpret_cast<lrcnn_plan_t *>(P.row), x, w, sc, sf,
                              ws + P.h_ck, ws, P.h_ck, mask_out, stream);
  if (st != LRCNN_OK) return st;
  Plan &C = *P.col;
  Run run(C, C.lw, S_LAYERWISE, ws + P.h_col, ws + P.h_ck, w + c, sc ? sc + c : nullptr,
          sf ? sf + c : nullptr, stream);
  // the output map stays in the layer-wise part's window for the backward
  if ((st = run.band_fwd(0, y, mask_out ? mask_out + c : nullptr, true, true)) != LRCNN_OK)
    return st;
  P.fwd_workspace = ws;
  return LRCNN_OK;
}

// The layer-wise part's backward (its maps are still in place) gives the
// checkpoint's float32 error, which seeds the row-centric part's backward.
int hybrid_backward(Plan &P, const void *x, const void *const *w, const float *const *sc,
                    const float *const *sf, const void *dy, float *const *dw, void *dx,
                    char *ws, void *stream) {
  const int c = P.hyb - 1;
  if (P.fwd_workspace != ws)
    return lrcnn_fail(LRCNN_ESTATE,
                      "hybrid backward needs a preceding lrcnn_forward_rows on this plan and "
                      "workspace");
  Plan &C = *P.col;
  Run run(C, C.lw, S_LAYERWISE, ws + P.h_col, ws + P.h_ck, w + c, sc ? sc + c : nullptr,
          sf ? sf + c : nullptr, stream);
  run.dx_f32 = true;
  if (!g_dry && !g_serial_wg && ensure_side(C)) run.side = (hipStream_t)C.side_stream;
  int st;
  if ((st = run.band_fwd(0, nullptr, nullptr, true, false, true)) != LRCNN_OK) return st;
  if ((st = run.begin_dw()) != LRCNN_OK) return st;
  if ((st = run.band_bwd(0, dy, dw + c, ws + P.h_dck, nullptr)) != LRCNN_OK) return st;
  if ((st = run.finish_dw(dw + c)) != LRCNN_OK) return st;
  return lrcnn_backward_rows(reinterpret_cast<lrcnn_plan_t *>(P.row), x, w, sc, sf,
                             ws + P.h_dck, dw, dx, ws, P.h_ck, stream);
}

}  // namespace
}  // namespace lrcnn

using namespace lrcnn;

extern "C" int lrcnn_forward_rows(lrcnn_plan_t *plan, const void *x, const void *const *w,
                                  const float *const *aff_scale, const float *const *aff_shift,
                                  void *y, void *workspace, size_t ws_bytes,
                                  void *const *mask_out, void *stream) {
  if (!plan) return lrcnn_fail(LRCNN_EINVAL, "plan is null");
  Plan &P = *reinterpret_cast<Plan *>(plan);
  int st = check_params(P, x, w, aff_scale, aff_shift);
  if (st != LRCNN_OK) return st;
  if (!y || misaligned(y)) return lrcnn_fail(LRCNN_EINVAL, "y null or misaligned");
  if (P.hyb) {
    if ((st = check_ws_bytes(P.h_total, workspace, ws_bytes)) != LRCNN_OK) return st;
    return hybrid_forward(P, x, w, aff_scale, aff_shift, y, (char *)workspace, mask_out, stream);
  }
  if ((st = check_ws(P.rc, workspace, ws_bytes)) != LRCNN_OK) return st;
  Run run(P, P.rc, P.cfg.mode == LRCNN_CARRY ? S_CARRY : S_RECOMPUTE, workspace, x, w, aff_scale,
          aff_shift, stream);
  P.fwd_workspace = nullptr;
  P.last_band_kept = false;
  // the last band's maps can serve the BP only when both passes use the
  // same partition
  const bool keep = P.refine == 1 && !P.no_keep;
  // bands on alternating streams (the backward's side stream is idle here),
  // the second one with its partial sums in the idle backward arena
  // (a dry run walks the same schedule with placeholder events)
  std::vector<void *> dry_ev;
  const bool pipe = P.cfg.mode == LRCNN_CARRY && P.nb_fp > 1 && !P.rc.fp_packed &&
                    P.rc.arena_bytes >= P.rc.part_bytes && !g_no_fp_pipe &&
                    (g_dry || (ensure_side(P) && ensure_fp_events(P)));
  if (pipe && g_dry) dry_ev.assign(2 * P.n, nullptr);
  void **evs = g_dry ? dry_ev.data() : P.ev_fp.data();
  hipStream_t sides[2] = {(hipStream_t)stream, pipe ? (hipStream_t)P.side_stream : nullptr};
  if (pipe) {
    LAUNCH(hipEventRecord((hipEvent_t)P.ev_fork, sides[0]), "event record");
    if (!sides[1] && !g_dry) return lrcnn_fail(LRCNN_EHIP, "side stream");
    LAUNCH(hipStreamWaitEvent(sides[1], (hipEvent_t)P.ev_fork, 0), "stream fork");
    run.pipe = true;
  }
  for (int r = 0; r < P.nb_fp; ++r) {
    if (pipe) {
      run.stream = sides[r & 1];
      run.part_off = r & 1 ? P.rc.arena : P.rc.part;
      run.ev_cur = (hipEvent_t *)evs + (r & 1) * P.n;
      run.ev_prev = r ? (hipEvent_t *)evs + ((r + 1) & 1) * P.n : nullptr;
    }
    if ((st = run.band_fwd(r, y, mask_out, false, keep && r == P.nb_fp - 1)) != LRCNN_OK)
      return st;
  }
  if (pipe) {
    // the caller's stream joins the side stream's last band
    const int rs = (P.nb_fp - 1) & 1 ? P.nb_fp - 1 : P.nb_fp - 2;
    LAUNCH(hipStreamWaitEvent(sides[0], (hipEvent_t)evs[(rs & 1) * P.n + P.n - 1], 0),
           "stream join");
  }
  P.fwd_workspace = workspace;
  P.last_band_kept = keep;
  P.fwd_epoch = ++g_epoch;
  return LRCNN_OK;
}

extern "C" int lrcnn_backward_rows(lrcnn_plan_t *plan, const void *x, const void *const *w,
                                   const float *const *aff_scale, const float *const *aff_shift,
                                   const void *dy, float *const *dw, void *dx, void *workspace,
                                   size_t ws_bytes, void *stream) {
  if (!plan) return lrcnn_fail(LRCNN_EINVAL, "plan is null");
  Plan &P = *reinterpret_cast<Plan *>(plan);
  int st = check_params(P, x, w, aff_scale, aff_shift);
  if (st != LRCNN_OK) return st;
  if (!dy || misaligned(dy)) return lrcnn_fail(LRCNN_EINVAL, "dy null or misaligned");
  if (dx && misaligned(dx)) return lrcnn_fail(LRCNN_EINVAL, "dx misaligned");
  if ((st = check_dw(P, dw)) != LRCNN_OK) return st;
  if (P.hyb) {
    if ((st = check_ws_bytes(P.h_total, workspace, ws_bytes)) != LRCNN_OK) return st;
    return hybrid_backward(P, x, w, aff_scale, aff_shift, dy, dw, dx, (char *)workspace, stream);
  }
  if ((st = check_ws(P.rc, workspace, ws_bytes)) != LRCNN_OK) return st;
  const bool carry = P.cfg.mode == LRCNN_CARRY;
  if (carry && P.fwd_workspace != workspace)
    return lrcnn_fail(LRCNN_ESTATE,
                      "CARRY backward needs a preceding lrcnn_forward_rows on this plan and workspace");
  Run run(P, P.rc, carry ? S_CARRY : S_RECOMPUTE, workspace, x, w, aff_scale, aff_shift, stream);
  if (!g_dry && !g_serial_wg && ensure_side(P)) run.side = (hipStream_t)P.side_stream;
  if ((st = run.begin_dw()) != LRCNN_OK) return st;
  float *dxacc = nullptr;
  if (!carry && dx) {
    const Shape &s = P.shp[0];
    size_t cnt = (size_t)P.cfg.batch * s.h * s.w * s.c;
    dxacc = P.cfg.dtype == LRCNN_BF16 ? (float *)((char *)workspace + P.rc.dxacc) : (float *)dx;
    int e = g_dry ? 0 : launch_zero_f32(dxacc, cnt, stream);
    if (e) return lrcnn_fail(LRCNN_EHIP, "zero dX");
  }
  // the last band's maps are still in place after lrcnn_forward_rows on this
  // workspace, so BP starts without recomputing it
  const bool kept = P.last_band_kept && P.fwd_workspace == workspace;
  P.last_band_kept = false;
  for (int r = P.nb - 1; r >= 0; --r) {
    const bool skip = kept && r == P.nb - 1;
    if ((st = run.band_fwd(r, nullptr, nullptr, true, false, skip)) != LRCNN_OK) return st;
    if ((st = run.band_bwd(r, dy, dw, dx, dxacc)) != LRCNN_OK) return st;
  }
  if ((st = run.finish_dw(dw)) != LRCNN_OK) return st;
  if (!carry && dx && P.cfg.dtype == LRCNN_BF16 && !g_dry) {
    const Shape &s = P.shp[0];
    int e = launch_rows_copy(DT_F32, DT_BF16, run.full(dxacc, 0), run.full(dx, 0), 0,
                             P.cfg.batch, 0, s.h, s.w, s.c, stream);
    if (e) return lrcnn_fail(LRCNN_EHIP, "store dX");
  }
  return LRCNN_OK;
}

extern "C" int lrcnn_layerwise_reference_gpu(lrcnn_plan_t *plan, const void *x,
                                             const void *const *w,
                                             const float *const *aff_scale,
                                             const float *const *aff_shift, const void *dy,
                                             void *y, float *const *dw, void *dx,
                                             void *workspace, size_t ws_bytes,
                                             void *const *mask_out, void *stream) {
  if (!plan) return lrcnn_fail(LRCNN_EINVAL, "plan is null");
  Plan &P = *reinterpret_cast<Plan *>(plan);
  int st = check_params(P, x, w, aff_scale, aff_shift);
  if (st != LRCNN_OK) return st;
  if (!y || misaligned(y)) return lrcnn_fail(LRCNN_EINVAL, "y null or misaligned");
  if (!dy || misaligned(dy)) return lrcnn_fail(LRCNN_EINVAL, "dy null or misaligned");
  if (dx && misaligned(dx)) return lrcnn_fail(LRCNN_EINVAL, "dx misaligned");
  if ((st = check_dw(P, dw)) != LRCNN_OK) return st;
  if ((st = check_ws(P.lw, workspace, ws_bytes)) != LRCNN_OK) return st;
  Run run(P, P.lw, S_LAYERWISE, workspace, x, w, aff_scale, aff_shift, stream);
  if (!g_dry && !g_serial_wg && ensure_side(P)) run.side = (hipStream_t)P.side_stream;
  // FP keeps every node's full map; BP reads them without recomputing.
  // The pool argmax is produced in FP (bp = true selects its buffer).
  if ((st = run.band_fwd(0, y, mask_out, true)) != LRCNN_OK) return st;
  if ((st = run.begin_dw()) != LRCNN_OK) return st;
  if ((st = run.band_bwd(0, dy, dw, dx, nullptr)) != LRCNN_OK) return st;
  return run.finish_dw(dw);
}

extern "C" int lrcnn_debug_layerwise_map(const lrcnn_plan_t *plan, int32_t node,
                                         size_t *offset) {
  if (!plan || !offset) return lrcnn_fail(LRCNN_EINVAL, "null argument");
  const Plan &P = *reinterpret_cast<const Plan *>(plan);
  if (node <= 0 || node >= P.n) return lrcnn_fail(LRCNN_EINVAL, "node out of range or input");
  if (node == P.n - 1 && !P.lw_keep_out)
    return lrcnn_fail(LRCNN_EINVAL, "the output node's map is y");
  if (P.fz_lw.fwd[node]) return lrcnn_fail(LRCNN_EINVAL, "map consumed by a fused add");
  *offset = P.lw.win[node];
  return LRCNN_OK;
}

extern "C" void lrcnn_debug_dry_run(int on) { lrcnn::g_dry = on != 0; }
extern "C" void lrcnn_debug_act_fusion(int on) { lrcnn::g_no_act_fusion = on == 0; }
extern "C" void lrcnn_debug_fp_pipeline(int on) { lrcnn::g_no_fp_pipe = on == 0; }
extern "C" void lrcnn_debug_serial_wgrad(int on) { lrcnn::g_serial_wg = on != 0; }
extern "C" void lrcnn_debug_dgrad_phases(int mode) { lrcnn::set_dgrad_phases(mode); }

extern "C" void lrcnn_debug_profile(int on) { lrcnn::profile_enable(on); }
extern "C" int lrcnn_debug_profile_collect(void) { return lrcnn::profile_collect(); }
extern "C" int lrcnn_debug_profile_entry(int32_t i, const char **name, int64_t *launches,
                                         double *ms, double *flops) {
  return lrcnn::profile_entry(i, name, launches, ms, flops);
}
extern "C" int lrcnn_debug_profile_roofline(int32_t i, double *bytes, double *roofline_ms) {
  if (!bytes || !roofline_ms) return -1;
  return lrcnn::profile_entry_roofline(i, bytes, roofline_ms);
}
