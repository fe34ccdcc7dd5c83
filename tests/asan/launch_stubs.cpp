// Stand-ins for the GPU launchers in the sanitizer build of the planner and
// executor: a dry run must never reach them, so each fails loudly.
#include <cstdio>
#include <cstdlib>

#include "kernels.hpp"

namespace lrcnn {
[[noreturn]] static void reached(const char *f) {
  std::fprintf(stderr, "dry run reached the GPU launcher %s\n", f);
  std::abort();
}
int launch_conv(int, int, const ConvArgs &, void *) { reached("launch_conv"); }
void set_dgrad_phases(int) {}
int launch_wgrad(int, const WgradArgs &, float *, void *) { reached("launch_wgrad"); }
int launch_pool_fwd(int, const PoolArgs &, void *) { reached("launch_pool_fwd"); }
int launch_pool_bwd(int, const PoolBwdArgs &, void *) { reached("launch_pool_bwd"); }
int launch_add_fwd(int, View, View, View, int, uint8_t *, int, int, int, int, int, int, void *) {
  reached("launch_add_fwd");
}
int launch_add_bwd(int, View, View, const AddSide &, const AddSide &, int, int, int, int, int, int,
                   void *) {
  reached("launch_add_bwd");
}
int launch_act_bwd(int, View, View, const float *, int, void *, int, int, int, int, int, void *,
                   const View *, int, int) {
  reached("launch_act_bwd");
}
int launch_rows_copy(int, int, View, View, int, int, int, int, int, int, void *) {
  reached("launch_rows_copy");
}
int launch_rows_copy_batch(int, const CopySeg *, int, void *) { reached("launch_rows_copy_batch"); }
int launch_rows_init(View, const View *, int, int, int, int, int, int, void *) {
  reached("launch_rows_init");
}
int launch_rows_zero(View, int, int, int, int, int, void *) { reached("launch_rows_zero"); }
int launch_zero_f32(float *, size_t, void *) { reached("launch_zero_f32"); }
int launch_pad_channels(int, View, View, int, int, int, int, int, int, void *) {
  reached("launch_pad_channels");
}
int launch_compact_dw(const float *, float *, int, int, long long, void *) {
  reached("launch_compact_dw");
}
void profile_enable(int) {}
int profile_collect() { return 0; }
int profile_entry(int, const char **, int64_t *, double *, double *) { return -1; }
int profile_entry_roofline(int, double *, double *) { return -1; }
}  // namespace lrcnn
