// Host stand-ins for the HIP runtime calls and GPU launchers used by the
// band executor, for a CPU check of its stream / event schedule: every
// launch, event record and stream wait is appended to a trace (no device
// work); streams and events are fake handles.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <vector>

#include "kernels.hpp"
#include "trace.hpp"

using lrcnn::View;

std::vector<TraceOp> g_trace;
static uintptr_t g_next_stream = 0x1000, g_next_event = 0x2000;

static int push(char kind, const void *s, const void *e, const char *what) {
  g_trace.push_back(TraceOp{kind, (uintptr_t)s, (uintptr_t)e, what, false, {}});
  return 0;
}
// A launch with its footprint: rows [r0, r1) of a view for every image.
struct Foot {
  std::vector<Span> spans;
  void rows(const View &v, int es, int B, int r0, int r1, bool w) {
    if (!v.p || r1 <= r0) return;
    const long long row = (long long)v.W * v.C;
    for (int b = 0; b < B; ++b) {
      const uintptr_t base = (uintptr_t)v.p + (uintptr_t)((b * v.bs + (r0 - v.row0) * row) * es);
      spans.push_back(Span{base, base + (uintptr_t)((r1 - r0) * row * es), w});
    }
  }
  void bytes(const void *p, size_t n, bool w) {
    if (p && n) spans.push_back(Span{(uintptr_t)p, (uintptr_t)p + n, w});
  }
  // rows [y0, y1) of a full-size [B][H][W][C] byte mask
  void mask(const uint8_t *m, int B, int H, int y0, int y1, int W, int C) {
    if (!m) return;
    for (int b = 0; b < B; ++b)
      bytes(m + ((size_t)b * H + y0) * W * C, (size_t)(y1 - y0) * W * C, true);
  }
};
static int launch(const void *s, const char *what, Foot &f) {
  g_trace.push_back(TraceOp{'K', (uintptr_t)s, 0, what, true, std::move(f.spans)});
  return 0;
}
static int es_of(int dt) { return dt == 0 ? 4 : 2; }

hipError_t hipGetDevice(int *d) {
  *d = 0;
  return hipSuccess;
}
hipError_t hipStreamCreateWithFlags(hipStream_t *s, unsigned int) {
  *s = (hipStream_t)(g_next_stream += 0x10);
  return hipSuccess;
}
hipError_t hipStreamDestroy(hipStream_t) { return hipSuccess; }
hipError_t hipEventCreateWithFlags(hipEvent_t *e, unsigned) {
  *e = (hipEvent_t)(g_next_event += 0x10);
  return hipSuccess;
}
hipError_t hipEventDestroy(hipEvent_t) { return hipSuccess; }
hipError_t hipEventRecord(hipEvent_t e, hipStream_t s) {
  push('R', s, e, "record");
  return hipSuccess;
}
hipError_t hipStreamWaitEvent(hipStream_t s, hipEvent_t e, unsigned int) {
  push('W', s, e, "wait");
  return hipSuccess;
}
const char *hipGetErrorString(hipError_t) { return "stub"; }

namespace lrcnn {
int launch_conv(int dt, int dgrad, const ConvArgs &a, void *s) {
  if (dgrad) return push('K', s, nullptr, "conv_dgrad");
  Foot f;
  const int es = es_of(dt);
  f.rows(a.src, es, a.B, std::max(a.sy0, a.y0 * a.sh - a.ph),
         std::min(a.sy1, (a.y1 - 1) * a.sh - a.ph + a.kh), false);
  f.rows(a.dst, es, a.B, a.y0, a.y1, true);
  if (a.res.p) f.rows(a.res, es, a.B, a.y0, a.y1, false);
  f.mask(a.mask, a.B, a.mask_h, a.y0, a.y1, a.Wd, a.N);
  if (a.splits > 1)
    f.bytes(a.part, (size_t)a.splits * a.B * (a.y1 - a.y0) * a.Wd * a.N * 4, true);
  return launch(s, "conv", f);
}
void set_dgrad_phases(int) {}
int launch_wgrad(int, const WgradArgs &, float *, void *s) { return push('K', s, nullptr, "wgrad"); }
int launch_pool_fwd(int dt, const PoolArgs &a, void *s) {
  Foot f;
  const int es = es_of(dt);
  f.rows(a.src, es, a.B, std::max(0, a.y0 * a.sh - a.ph),
         std::min(a.Hs, (a.y1 - 1) * a.sh - a.ph + a.kh), false);
  f.rows(a.dst, es, a.B, a.y0, a.y1, true);
  f.bytes(a.am, (size_t)a.B * (a.y1 - a.y0) * a.Wd * a.C, true);
  f.mask(a.mask, a.B, a.mask_h, a.y0, a.y1, a.Wd, a.C);
  return launch(s, "pool_fwd", f);
}
int launch_pool_bwd(int, const PoolBwdArgs &, void *s) { return push('K', s, nullptr, "pool_bwd"); }
int launch_add_fwd(int dt, View a, View b, View z, int, uint8_t *mask, int mask_h, int B, int y0,
                   int y1, int W, int C, void *s) {
  Foot f;
  const int es = es_of(dt);
  f.rows(a, es, B, y0, y1, false);
  f.rows(b, es, B, y0, y1, false);
  f.rows(z, es, B, y0, y1, true);
  f.mask(mask, B, mask_h, y0, y1, W, C);
  return launch(s, "add_fwd", f);
}
int launch_add_bwd(int, View, View, const AddSide &, const AddSide &, int, int, int, int, int, int,
                   void *s) {
  return push('K', s, nullptr, "add_bwd");
}
int launch_act_bwd(int, View, View, const float *, int, void *, int, int, int, int, int, void *s,
                   const View *, int, int) {
  return push('K', s, nullptr, "act_bwd");
}
int launch_rows_copy(int st, int dtt, View src, View dst, int acc, int B, int r0, int r1, int,
                     int, void *s) {
  Foot f;
  f.rows(src, es_of(st), B, r0, r1, false);
  f.rows(dst, es_of(dtt), B, r0, r1, true);
  if (acc) f.rows(dst, es_of(dtt), B, r0, r1, false);
  return launch(s, "rows_copy", f);
}
int launch_rows_copy_batch(int dt, const CopySeg *segs, int n, void *s) {
  Foot f;
  for (int i = 0; i < n; ++i) {
    f.rows(segs[i].src, es_of(dt), segs[i].B, segs[i].r0, segs[i].r1, false);
    f.rows(segs[i].dst, es_of(dt), segs[i].B, segs[i].r0, segs[i].r1, true);
  }
  return launch(s, "rows_copy_batch", f);
}
int launch_rows_init(View, const View *, int, int, int, int, int, int, void *s) {
  return push('K', s, nullptr, "rows_init");
}
int launch_rows_zero(View, int, int, int, int, int, void *s) { return push('K', s, nullptr, "rows_zero"); }
int launch_zero_f32(float *, size_t, void *s) { return push('K', s, nullptr, "zero_f32"); }
int launch_pad_channels(int, View, View, int, int, int, int, int, int, void *s) {
  return push('K', s, nullptr, "pad_channels");
}
int launch_compact_dw(const float *, float *, int, int, long long, void *s) {
  return push('K', s, nullptr, "compact_dw");
}
void profile_enable(int) {}
int profile_collect() { return 0; }
int profile_entry(int, const char **, int64_t *, double *, double *) { return -1; }
int profile_entry_roofline(int, double *, double *) { return -1; }
}  // namespace lrcnn
