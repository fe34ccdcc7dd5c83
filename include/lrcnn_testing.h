/*
 * lrcnn_testing.h -- test hooks of liblrcnn.so (not needed by users).
 */
#ifndef LRCNN_TESTING_H
#define LRCNN_TESTING_H

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

#ifdef __cplusplus
}
#endif
#endif /* LRCNN_TESTING_H */
