// Allocation-free row-centric forward pass: lrcnn_forward_rows with a
// workspace that the library holds in a file-scope device array.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "lrcnn.h"
#include "plan.hpp"

// One copy per device, resident from the code object's load until the
// process ends; every call on a device uses (and overwrites) that device's
// copy.
static __device__ __align__(256) unsigned char scratch[LRCNN_STATIC_WORKSPACE_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void *g_scratch[kMaxDevices] = {};

// Device address of the current device's copy of `scratch`, looked up once
// per device (host code may not pass the array's own name to a kernel: on
// the host it is only a stand-in for the symbol).
int scratch_address(void **out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return lrcnn_fail(LRCNN_EHIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return lrcnn_fail(LRCNN_EHIP, "device index " + std::to_string(dev) + " out of range");
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return lrcnn_fail(LRCNN_EHIP, std::string("hipGetSymbolAddress(scratch): ") +
                                        hipGetErrorString(e));
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return LRCNN_OK;
}

}  // namespace

extern "C" int lrcnn_forward_rows_static(lrcnn_plan_t *plan, const void *x,
                                         const void *const *w, const float *const *aff_scale,
                                         const float *const *aff_shift, void *y,
                                         void *const *mask_out, void *stream) {
  if (!plan) return lrcnn_fail(LRCNN_EINVAL, "plan is null");
  lrcnn_plan_info info;
  int st = lrcnn_plan_query(plan, &info);
  if (st != LRCNN_OK) return st;
  if (info.workspace_bytes > (size_t)LRCNN_STATIC_WORKSPACE_BYTES)
    return lrcnn_fail(LRCNN_EWORKSPACE,
                      "plan needs " + std::to_string(info.workspace_bytes) +
                          " bytes of workspace; the static workspace holds " +
                          std::to_string((size_t)LRCNN_STATIC_WORKSPACE_BYTES));
  void *ws = nullptr;
  if ((st = scratch_address(&ws)) != LRCNN_OK) return st;
  return lrcnn_forward_rows(plan, x, w, aff_scale, aff_shift, y, ws,
                            (size_t)LRCNN_STATIC_WORKSPACE_BYTES, mask_out, stream);
}
