// CPU check of the executor's stream schedule as a HIP graph capture would
// see it. Reads cases (same line format as the sanitizer dry run, plus a
// final pipeline flag), runs lrcnn_forward_rows then lrcnn_backward_rows on
// one origin stream with the launchers and HIP stream calls stubbed
// (trace_stubs.cpp), and checks the recorded trace:
//  * a stream other than the origin joins the capture only by waiting for
//    an event recorded in it, and issues nothing before that;
//  * every waited-for event was recorded earlier in the same capture;
//  * at the end every stream's last operation happens before the origin
//    stream's last operation (all forked work is joined back);
//  * no two forward launches on different streams that the streams and
//    events leave unordered touch the same bytes with one of them writing
//    (the stubs record each forward launch's rows of every buffer).
// A case's final flag: bit 0 pipelines the forward over two streams, bit 1
// checks the forward alone.
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <map>
#include <set>
#include <vector>

#include "lrcnn.h"
#include "lrcnn_testing.h"
#include "trace.hpp"

static int check(const std::vector<TraceOp> &t, uintptr_t origin, int ncase) {
  int bad = 0;
  std::vector<std::vector<int>> preds;  // op graph: node per trace op
  std::map<uintptr_t, int> last;        // stream -> last node (-1: none yet)
  std::map<uintptr_t, int> ev;          // event -> node of its record
  std::set<uintptr_t> joined{origin};
  std::map<uintptr_t, int> nops;
  last[origin] = -1;
  for (size_t i = 0; i < t.size(); ++i) {
    const TraceOp &o = t[i];
    ++nops[o.stream];
    std::vector<int> p;
    if (!joined.count(o.stream)) {
      if (o.kind != 'W') {
        std::printf("case %d: op %zu (%s) on stream %#lx before it joined the capture\n", ncase,
                    i, o.what, (unsigned long)o.stream);
        ++bad;
      }
      last[o.stream] = -1;
    }
    if (last[o.stream] >= 0) p.push_back(last[o.stream]);
    if (o.kind == 'W') {
      auto it = ev.find(o.event);
      if (it == ev.end()) {
        std::printf("case %d: op %zu waits for event %#lx not recorded in the capture\n", ncase,
                    i, (unsigned long)o.event);
        ++bad;
      } else if (it->second >= 0) {
        p.push_back(it->second);
      }
      joined.insert(o.stream);
    }
    preds.push_back(p);
    const int node = (int)preds.size() - 1;
    if (o.kind == 'R') ev[o.event] = last[o.stream];  // the stream's work so far
    else last[o.stream] = node;
    if (o.kind == 'R' && last[o.stream] < 0) ev[o.event] = -1;  // capture start
  }
  // ancestors of the origin stream's last node
  std::vector<char> anc(preds.size(), 0);
  std::vector<int> stack;
  if (last[origin] >= 0) stack.push_back(last[origin]);
  while (!stack.empty()) {
    const int n = stack.back();
    stack.pop_back();
    if (anc[n]) continue;
    anc[n] = 1;
    for (int q : preds[n]) stack.push_back(q);
  }
  for (auto &kv : last)
    if (kv.first != origin && kv.second >= 0 && !anc[kv.second]) {
      std::printf("case %d: stream %#lx has work after its last join (op %d, %s)\n", ncase,
                  (unsigned long)kv.first, kv.second, t[kv.second].what);
      ++bad;
    }
  // separate error-window initialisation launches (zeroing, carry copy-in)
  int inits = 0;
  for (const TraceOp &o : t)
    if (o.kind == 'K' && (!std::strcmp(o.what, "rows_init") || !std::strcmp(o.what, "rows_zero")))
      ++inits;
  std::printf("case %d: ops %zu streams %zu", ncase, t.size(), nops.size());
  for (auto &kv : nops) std::printf(" [%s %d]", kv.first == origin ? "origin" : "side", kv.second);
  std::printf(" inits %d violations %d\n", inits, bad);
  return bad;
}

// Unordered conflicting accesses among the launches trace[0, end): two
// launches on different streams, neither ordered before the other by the
// streams and events, that touch overlapping bytes, one of them writing.
// (lim: byte size of the buffer in each 2^40 range, 0 = unchecked)
static int races(const std::vector<TraceOp> &t, size_t end, int ncase,
                 const std::map<uint64_t, uint64_t> &lim) {
  std::map<uintptr_t, int> sid;
  for (size_t i = 0; i < end; ++i) sid.emplace(t[i].stream, (int)sid.size());
  const int S = (int)sid.size();
  std::vector<std::vector<int>> clock(S, std::vector<int>(S, 0)), vc(end);
  std::map<uintptr_t, std::vector<int>> evc;
  int unknown = 0;
  for (size_t i = 0; i < end; ++i) {
    const int s = sid[t[i].stream];
    if (t[i].kind == 'K') {
      ++clock[s][s];
      vc[i] = clock[s];
      if (!t[i].known) ++unknown;
    } else if (t[i].kind == 'R') {
      evc[t[i].event] = clock[s];
    } else {
      auto it = evc.find(t[i].event);
      if (it != evc.end())
        for (int k = 0; k < S; ++k) clock[s][k] = std::max(clock[s][k], it->second[k]);
    }
  }
  auto hb = [&](size_t a, size_t b) {  // launch a happens before launch b
    const int s = sid[t[a].stream];
    return vc[a][s] <= vc[b][s];
  };
  struct Iv {
    uintptr_t lo, hi;
    size_t op;
    bool w;
  };
  std::vector<Iv> iv;
  int oob = 0;
  for (size_t i = 0; i < end; ++i)
    if (t[i].kind == 'K')
      for (const Span &sp : t[i].spans) {
        iv.push_back(Iv{sp.lo, sp.hi, i, sp.write});
        const uint64_t k = (uint64_t)sp.lo >> 40;
        auto it = lim.find(k);
        if (it != lim.end() && (sp.hi > ((k << 40) + it->second) || (uint64_t)sp.hi >> 40 != k)) {
          if (oob < 8)
            std::printf("case %d: op %zu (%s) touches bytes [%#lx, %#lx) past its buffer's %lu "
                        "bytes\n", ncase, i, t[i].what, (unsigned long)(sp.lo - (k << 40)),
                        (unsigned long)(sp.hi - (k << 40)), (unsigned long)it->second);
          ++oob;
        }
      }
  std::sort(iv.begin(), iv.end(), [](const Iv &a, const Iv &b) { return a.lo < b.lo; });
  std::vector<Iv> act;
  int found = 0;
  for (const Iv &x : iv) {
    size_t k = 0;
    for (size_t j = 0; j < act.size(); ++j)
      if (act[j].hi > x.lo) act[k++] = act[j];
    act.resize(k);
    for (const Iv &a : act) {
      if (!(a.w || x.w) || t[a.op].stream == t[x.op].stream || a.op == x.op) continue;
      if (hb(a.op, x.op) || hb(x.op, a.op)) continue;
      if (found < 8)
        std::printf("case %d: race: op %zu (%s%s) and op %zu (%s%s) on different streams share "
                    "bytes [%#lx, %#lx)\n", ncase, a.op, t[a.op].what, a.w ? " write" : " read",
                    x.op, t[x.op].what, x.w ? " write" : " read", (unsigned long)x.lo,
                    (unsigned long)std::min(a.hi, x.hi));
      ++found;
    }
    act.push_back(x);
  }
  std::printf("case %d: forward launches %zu on %d stream(s), footprint unknown %d, races %d, "
              "out of bounds %d\n", ncase, end, S, unknown, found, oob);
  return found + unknown + oob;
}

int main() {
  int ncase = 0, fails = 0, n;
  while (std::scanf("%d", &n) == 1) {
    ++ncase;
    std::vector<lrcnn_node> nodes(n);
    for (auto &d : nodes)
      if (std::scanf("%d %d %d %d %d %d %d %d %d %d %d %d", &d.op, &d.in0, &d.in1, &d.c_out,
                     &d.kh, &d.kw, &d.sh, &d.sw, &d.ph, &d.pw, &d.affine, &d.relu) != 12)
        return 2;
    lrcnn_config c{};
    int nbounds = 0, pipe = 0;
    if (std::scanf("%d %d %d %d %d %d %d %d %d %d %d %d", &c.batch, &c.in_c, &c.in_h, &c.in_w,
                   &c.dtype, &c.mode, &c.n_bands, &c.policy, &c.bp_refine, &c.hybrid_from,
                   &c.first_rows, &nbounds) != 12)
      return 2;
    std::vector<int32_t> bounds(nbounds);
    for (auto &b : bounds)
      if (std::scanf("%d", &b) != 1) return 2;
    if (std::scanf("%d", &pipe) != 1) return 2;
    c.bounds = nbounds ? bounds.data() : nullptr;
    lrcnn_plan_t *p = nullptr;
    if (lrcnn_plan(nodes.data(), n, &c, &p) != LRCNN_OK) {
      std::printf("case %d: plan failed: %s\n", ncase, lrcnn_last_error());
      ++fails;
      continue;
    }
    lrcnn_plan_info info{};
    lrcnn_plan_query(p, &info);
    lrcnn_debug_fp_pipeline(pipe & 1);
    // placeholder device pointers, never dereferenced (the launchers are
    // stubs), each buffer in its own 2^40-byte range so that footprints of
    // distinct buffers never overlap
    auto fake = [](uint64_t k) { return (void *)(uintptr_t)(k << 40); };
    std::vector<const void *> cptr(n);
    std::vector<const float *> fptr(n);
    std::vector<float *> dwp(n);
    std::vector<void *> masks(n);
    for (int v = 0; v < n; ++v) {
      cptr[v] = fake(16 + v);
      fptr[v] = (const float *)fake(16 + n + v);
      dwp[v] = (float *)fake(16 + 2 * n + v);
      masks[v] = fake(16 + 3 * n + v);
    }
    void *x = fake(1), *y = fake(2), *dy = fake(3), *dx = fake(4), *ws = fake(5);
    const uintptr_t origin = 0x10;
    for (int rep = 0; rep < 2; ++rep) {  // a second step reuses the plan's streams and events
      g_trace.clear();
      int st = lrcnn_forward_rows(p, x, cptr.data(), fptr.data(), fptr.data(), y, ws,
                                  info.workspace_bytes, masks.data(), (void *)origin);
      const size_t fwd_end = g_trace.size();
      if (st == LRCNN_OK && rep == 0) {
        // buffer sizes: workspace, y and every node's mask
        std::map<uint64_t, uint64_t> lim;
        const uint64_t es = c.dtype == LRCNN_BF16 ? 2 : 4;
        lim[5] = info.workspace_bytes;
        lim[2] = (uint64_t)c.batch * info.out_h * info.out_w * info.out_c * es;
        for (int v = 1; v < n; ++v) {
          int32_t sh[3];
          if (lrcnn_plan_node_shape(p, v, sh) == LRCNN_OK)
            lim[16 + 3 * n + v] = (uint64_t)c.batch * sh[0] * sh[1] * sh[2];
        }
        fails += races(g_trace, fwd_end, ncase, lim) != 0;
      }
      if (st == LRCNN_OK && (pipe & 2)) {
        fails += check(g_trace, origin, ncase) != 0;  // forward only
        continue;
      }
      if (st == LRCNN_OK)
        st = lrcnn_backward_rows(p, x, cptr.data(), fptr.data(), fptr.data(), dy, dwp.data(), dx,
                                 ws, info.workspace_bytes, (void *)origin);
      if (st != LRCNN_OK) {
        std::printf("case %d: step failed: %s\n", ncase, lrcnn_last_error());
        ++fails;
        break;
      }
      fails += check(g_trace, origin, ncase) != 0;
    }
    lrcnn_debug_fp_pipeline(0);
    lrcnn_plan_destroy(p);
  }
  std::printf("cases %d failures %d\n", ncase, fails);
  return fails != 0;
}
