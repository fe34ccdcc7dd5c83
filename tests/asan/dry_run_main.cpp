// Host driver of the planner and the band executor's dry run, built with
// AddressSanitizer and UndefinedBehaviorSanitizer (tests/test_asan_dry_run.py).
// Reads cases from stdin, one per line:
//   n_nodes <12 ints per node> batch in_c in_h in_w dtype mode n_bands policy
//   bp_refine hybrid_from first_rows n_bounds <bounds> expect
// expect = 0: the plan must succeed and every entry point must walk its
// whole schedule in dry-run mode; expect < 0: lrcnn_plan must fail with
// that status. Device pointers are placeholders: a dry run never touches
// them (the launchers are stubs that fail if reached).
#include <cstdint>
#include <cstdio>
#include <vector>

#include "lrcnn.h"
#include "lrcnn_testing.h"

static int fails = 0;
#define EXPECT(c, msg)                                                             \
  do {                                                                             \
    if (!(c)) {                                                                    \
      ++fails;                                                                     \
      std::printf("case %d: %s failed: %s (%s)\n", ncase, msg, #c, lrcnn_last_error()); \
    }                                                                              \
  } while (0)

int main() {
  lrcnn_debug_dry_run(1);
  int ncase = 0;
  int n;
  while (std::scanf("%d", &n) == 1) {
    ++ncase;
    std::vector<lrcnn_node> nodes(n);
    for (auto &d : nodes)
      if (std::scanf("%d %d %d %d %d %d %d %d %d %d %d %d", &d.op, &d.in0, &d.in1, &d.c_out,
                     &d.kh, &d.kw, &d.sh, &d.sw, &d.ph, &d.pw, &d.affine, &d.relu) != 12)
        return 2;
    lrcnn_config c{};
    int nbounds = 0, expect = 0;
    if (std::scanf("%d %d %d %d %d %d %d %d %d %d %d %d", &c.batch, &c.in_c, &c.in_h, &c.in_w,
                   &c.dtype, &c.mode, &c.n_bands, &c.policy, &c.bp_refine, &c.hybrid_from,
                   &c.first_rows, &nbounds) != 12)
      return 2;
    std::vector<int32_t> bounds(nbounds);
    for (auto &b : bounds)
      if (std::scanf("%d", &b) != 1) return 2;
    if (std::scanf("%d", &expect) != 1) return 2;
    c.bounds = nbounds ? bounds.data() : nullptr;
    lrcnn_plan_t *p = nullptr;
    const int st = lrcnn_plan(nodes.data(), n, &c, &p);
    if (expect < 0) {
      EXPECT(st == expect && p == nullptr, "expected planning error");
      continue;
    }
    EXPECT(st == LRCNN_OK, "plan");
    if (st != LRCNN_OK) continue;
    lrcnn_plan_info info{};
    EXPECT(lrcnn_plan_query(p, &info) == LRCNN_OK, "query");
    for (int ph = 0; ph < 2; ++ph)
      for (int b = 0; b < (ph ? info.bp_bands : info.n_bands); ++b)
        for (int v = 0; v < n; ++v) {
          int32_t rows[4];
          EXPECT(lrcnn_plan_band_rows(p, ph, b, v, rows) == LRCNN_OK, "band rows");
        }
    // placeholder device pointers (16-byte aligned, never dereferenced)
    std::vector<void *> ptr(n, (void *)0x100000);
    std::vector<const void *> cptr(n, (const void *)0x100000);
    std::vector<const float *> fptr(n, (const float *)0x100000);
    std::vector<float *> dwp(n, (float *)0x100000);
    std::vector<void *> masks(n, (void *)0x200000);
    void *x = (void *)0x300000, *y = (void *)0x400000, *dy = (void *)0x500000,
         *dx = (void *)0x600000, *ws = (void *)0x700000;
    EXPECT(lrcnn_forward_rows(p, x, cptr.data(), fptr.data(), fptr.data(), y, ws,
                              info.workspace_bytes, masks.data(), nullptr) == LRCNN_OK,
           "forward");
    EXPECT(lrcnn_backward_rows(p, x, cptr.data(), fptr.data(), fptr.data(), dy, dwp.data(), dx,
                               ws, info.workspace_bytes, nullptr) == LRCNN_OK,
           "backward");
    EXPECT(lrcnn_backward_rows(p, x, cptr.data(), fptr.data(), fptr.data(), dy, dwp.data(),
                               nullptr, ws, info.workspace_bytes, nullptr) == LRCNN_OK,
           "backward without dx");
    EXPECT(lrcnn_layerwise_reference_gpu(p, x, cptr.data(), fptr.data(), fptr.data(), dy, y,
                                         dwp.data(), dx, ws, info.layerwise_workspace_bytes,
                                         masks.data(), nullptr) == LRCNN_OK,
           "layer-wise");
    // a workspace one byte short is refused
    EXPECT(lrcnn_forward_rows(p, x, cptr.data(), fptr.data(), fptr.data(), y, ws,
                              info.workspace_bytes - 1, nullptr, nullptr) == LRCNN_EWORKSPACE,
           "short workspace");
    size_t sb = 0;
    EXPECT(lrcnn_plan_step_bytes(p, 0, 1, &sb) == LRCNN_OK && sb > info.workspace_bytes,
           "step bytes");
    lrcnn_plan_destroy(p);
    if (c.policy != LRCNN_EXPLICIT && c.hybrid_from == 0) {
      // the budget of this plan's step: the search must return a plan
      // whose step fits it, or report that none does
      lrcnn_budget bud{sb, info.bp_bands, c.bp_refine > 1 ? c.bp_refine : 1, 1};
      lrcnn_plan_t *q = nullptr;
      const int bs = lrcnn_plan_for_budget(nodes.data(), n, &c, &bud, &q);
      size_t qb = 0;
      EXPECT(bs == LRCNN_EINFEASIBLE ||
                 (bs == LRCNN_OK && lrcnn_plan_step_bytes(q, 0, 1, &qb) == LRCNN_OK && qb <= sb),
             "budget plan");
      lrcnn_plan_destroy(q);
      int32_t mb = 0;
      const int ms = lrcnn_max_batch(nodes.data(), n, &c, 0, &bud, &mb);
      EXPECT(ms == LRCNN_EINFEASIBLE || (ms == LRCNN_OK && mb >= 1), "max batch");
    }
  }
  std::printf("cases %d failures %d\n", ncase, fails);
  return fails != 0;
}
