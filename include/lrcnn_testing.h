/*
 * lrcnn_testing.h -- test hooks of liblrcnn.so (not needed by users).
 */
#ifndef LRCNN_TESTING_H
#define LRCNN_TESTING_H

#include <stddef.h>
#include <stdint.h>

#include "lrcnn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* on != 0: on the calling thread, lrcnn_forward_rows, lrcnn_backward_rows
 * and lrcnn_layerwise_reference_gpu walk their whole band schedule and run
 * every host-side check (argument checks and the check that each kernel's
 * row ranges lie inside the buffers it touches) but enqueue no GPU work and
 * never dereference a device pointer. Lets the executor's bookkeeping be
 * tested on a machine without a GPU. on == 0 restores normal operation. */
void lrcnn_debug_dry_run(int on);

/* on == 0: plans created on the calling thread form every convolution's
 * error operand by its own activation-backward pass; on != 0 (default) the
 * input gradient of a convolution's only consumer, which completes the
 * convolution's error, forms the error operand and carried rows itself
 * (CARRY plans). Both do the same arithmetic, so results are bitwise equal. */
void lrcnn_debug_act_fusion(int on);

/* on != 0: on the calling thread, lrcnn_forward_rows of CARRY plans with
 * more than one band runs consecutive bands on two streams, each step of a
 * band waiting only until the previous band no longer reads the windows it
 * writes (split-K partial sums of the second stream in the idle backward
 * arena); on == 0 (default) the bands run one after another on the
 * caller's stream. Results are bitwise equal. */
void lrcnn_debug_fp_pipeline(int on);

/* on != 0: on the calling thread, the backward launches every weight
 * gradient on the caller's stream, just before the input gradient it would
 * otherwise overlap, so that a profile times each kernel with the GPU to
 * itself; on == 0 (default) the weight gradients run on the plan's side
 * stream. Results are bitwise equal. */
void lrcnn_debug_serial_wgrad(int on);

/* On the calling thread, the input gradient of a strided convolution
 * (stride s in both directions) is computed as s^2 launches, one per phase
 * of producer rows and columns ((y + pad) mod s), each with only the taps
 * that reach it: mode 0 = when estimated faster than one launch over all
 * taps (default), 1 = always, 2 = never. Results agree to rounding. */
void lrcnn_debug_dgrad_phases(int mode);

/* on != 0: clear and start timing every matrix-core kernel launch
 * (convolution forward, input gradient, weight gradient) and split
 * reduction: the launch goes through hipExtLaunchKernelGGL with a start and
 * a stop event attached to the dispatch, so the interval is the kernel's
 * execution; each launch's algorithmic FLOPs are recorded with it. on == 0
 * stops. Timing only: results are unchanged. Launches made while timing is
 * on cannot be captured in a graph (the events belong to the dispatch). */
void lrcnn_debug_profile(int on);

/* After the recorded streams are synchronised: aggregate the records per
 * kernel instantiation. Returns the number of kernels, or -1 on a HIP
 * error. */
int lrcnn_debug_profile_collect(void);

/* Entry i of the aggregate: kernel name (valid until the next collect),
 * launch count, summed launch durations in milliseconds and summed
 * algorithmic FLOPs. Returns 0, or -1 if i is out of range. */
int lrcnn_debug_profile_entry(int32_t i, const char **name, int64_t *launches,
                              double *ms, double *flops);

/* Entry i's summed algorithmic HBM bytes (operands read once, outputs and
 * split partial sums written once, read-modify-writes counted twice) and
 * summed roofline times in milliseconds: per launch the larger of its FLOPs
 * at MI355X's dense matrix-core peak for its storage type (bf16 2.5
 * PFLOP/s, fp32 157.3 TFLOP/s) and its bytes at 8 TB/s. Returns 0, or -1 if
 * i is out of range or a pointer is null. */
int lrcnn_debug_profile_roofline(int32_t i, double *bytes, double *roofline_ms);

/* Byte offset in the layer-wise workspace of node `node`'s full feature map
 * ([B][H][W][C], dense, the plan's storage dtype) as
 * lrcnn_layerwise_reference_gpu leaves it: its forward, which equals
 * lrcnn_forward_rows of the same plan bit for bit, keeps every map there
 * for the backward and the maps are unchanged when the call returns.
 * Errors: EINVAL for a null argument, a node out of range, the input
 * (node 0, which is x), the output node (which is y) and a convolution
 * whose value the residual add's forward consumes directly (never
 * stored). */
int lrcnn_debug_layerwise_map(const lrcnn_plan_t *plan, int32_t node, size_t *offset);

#ifdef __cplusplus
}
#endif
#endif /* LRCNN_TESTING_H */
