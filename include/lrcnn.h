/*
 * lrcnn.h -- row-centric CNN training (LR-CNN, arXiv 2401.11471) on one
 * AMD Instinct MI355X (gfx950).
 *
 * The paper re-orders the training of a convolution stack from layer order
 * ("column") to row order (Section III-A, Eqs. (4)-(5), Algorithm 1): the
 * input is split into horizontal row bands, every band is pushed through all
 * layers before the next one starts, and the feature maps of a band are
 * dropped as soon as the band is done. Backward propagation walks the bands
 * in reverse, recomputes each band's feature maps (Algorithm 1, BP loop) and
 * accumulates the weight gradients g^l over bands. Convolution windows that
 * straddle two bands (the "weak dependency", Section III-B) are handled in
 * one of two ways:
 *   LRCNN_CARRY      two-phase sharing (Section IV-A): rows of a feature map
 *                    that a later band still needs are kept when the band
 *                    that computed them finishes, and reused in FP and BP;
 *                    in BP the error that a band sends to rows owned by an
 *                    earlier band is carried to that band in float32.
 *   LRCNN_RECOMPUTE  overlapping partitioning (Section IV-B): the last layer
 *                    is split evenly and every band recomputes its whole
 *                    receptive cone; each band back-propagates only its own
 *                    rows of the upstream gradient and the partial gradients
 *                    are summed (exact, by linearity).
 * Padding is "semi-closed" (Section III-B): only the true image top and
 * bottom are padded; band edges always see real rows.
 *
 * Results equal ordinary layer-by-layer training up to float rounding.
 *
 * Conventions for every entry point:
 *  - Return value: LRCNN_OK (0) or a negative lrcnn_status; the message of the
 *    last error on the calling thread is returned by lrcnn_last_error().
 *  - Device pointers are caller-owned device memory (hipMalloc or a torch
 *    tensor); the library never allocates or frees device memory and never
 *    synchronises: all work is enqueued on `stream` (a hipStream_t; NULL is
 *    the default stream).
 *  - Tensors are dense NHWC: x is [B][H][W][C_in], y / dy are the last node's
 *    output [B][H_L][W_L][C_L]. Weights are [C_out][kh][kw][C_in].
 *    Storage type is the plan's dtype (float32 or bfloat16) for x, y, dy, dx
 *    and weights; affine scale/shift and weight gradients are float32.
 *  - Per-node arrays (w, aff_scale, aff_shift, dw, mask_out) are HOST arrays
 *    of n_nodes device pointers indexed by node id; entries of nodes they do
 *    not apply to are ignored and may be NULL.
 *  - Device pointers must be 16-byte aligned.
 *  - A plan must not be used from two streams or threads at once.
 */
#ifndef LRCNN_H
#define LRCNN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  LRCNN_OK = 0,
  LRCNN_EINVAL = -1,      /* null pointer, bad enum, misaligned pointer      */
  LRCNN_ESHAPE = -2,      /* inconsistent graph or a layer with no output    */
  LRCNN_EPARTITION = -3,  /* band bounds not monotone / out of range         */
  LRCNN_EWORKSPACE = -4,  /* workspace smaller than the plan requires        */
  LRCNN_ESTATE = -5,      /* backward_rows without a matching forward_rows   */
  LRCNN_EDTYPE = -6,      /* unsupported dtype                               */
  LRCNN_EHIP = -7,        /* a HIP launch failed                             */
  LRCNN_EINFEASIBLE = -8  /* no band count fits the memory budget            */
} lrcnn_status;

/* Node kinds. Nodes are given in topological order; node 0 is the input. */
enum {
  LRCNN_OP_INPUT = 0,
  LRCNN_OP_CONV = 1,    /* bias-free cross-correlation, Eq. (1); optional  */
                        /* per-channel affine (fixed BatchNorm) and ReLU    */
  LRCNN_OP_MAXPOOL = 2, /* kh x kw window, stride, -inf padding             */
  LRCNN_OP_ADD = 3      /* elementwise in0 + in1 (residual), optional ReLU */
};

typedef struct {
  int32_t op;
  int32_t in0, in1;          /* producer node ids (in1 only for ADD), else -1 */
  int32_t c_out;             /* CONV output channels (ignored otherwise)      */
  int32_t kh, kw, sh, sw, ph, pw;
  int32_t affine;            /* CONV: out = scale[c] * conv + shift[c]       */
  int32_t relu;              /* CONV / ADD: ReLU after affine / sum           */
} lrcnn_node;

enum { LRCNN_F32 = 0, LRCNN_BF16 = 1 };
enum { LRCNN_CARRY = 0, LRCNN_RECOMPUTE = 1 };
/* Band placement. CARRY bands are ranges of input rows (Algorithm 1 splits
 * the input); RECOMPUTE bands are ranges of the last node's rows (the paper
 * divides the last layer evenly, Section IV-B).
 *   EVEN       r * H / N boundaries
 *   BALANCED   CARRY only: boundaries that minimise the peak workspace of
 *              the step (the skew of Section IV-A)
 *   EXPLICIT   the caller's `bounds` (n_bands + 1 non-decreasing values from
 *              0 to the partitioned height; empty bands are allowed)
 *   PAPER_2PS  CARRY only: the greedy partition of two-phase sharing
 *              (Section IV-A, Eqs. (11), (13), (14)). Band r must complete
 *              t_r rows of the last node: t_1 = first_rows (H_1^L; 0 reads
 *              as ceil(H_L / N_BP)), the remaining H_L - t_1 rows are split
 *              evenly over bands 2..N_BP. A band's end is the smallest input
 *              row count from which the frontier of the last node reaches
 *              t_r -- for a chain of layers exactly the input height that
 *              Eq. (11) (first band) and Eq. (13) (middle bands) give by
 *              inverting the layers from the last one; the last band takes
 *              the remaining input rows (Eq. (14)). The partition is made
 *              for the backward bands (N_BP = n_bands * bp_refine, as the
 *              paper sizes it for BP); the forward bands are every
 *              bp_refine-th of them. */
enum { LRCNN_EVEN = 0, LRCNN_BALANCED = 1, LRCNN_EXPLICIT = 2, LRCNN_PAPER_2PS = 3 };
enum { LRCNN_HYBRID_AUTO = -1 };

typedef struct {
  int32_t batch, in_c, in_h, in_w;
  int32_t dtype;             /* LRCNN_F32 | LRCNN_BF16                        */
  int32_t mode;              /* LRCNN_CARRY | LRCNN_RECOMPUTE                 */
  int32_t n_bands;           /* N >= 1: bands of the forward pass             */
  int32_t policy;            /* LRCNN_EVEN | BALANCED | EXPLICIT | PAPER_2PS  */
  const int32_t *bounds;     /* host array, used when policy == EXPLICIT      */
  int32_t bp_refine;         /* >= 1 (0 reads as 1): the backward pass splits */
                             /* every forward band evenly into bp_refine      */
                             /* bands, N_BP = N * bp_refine (the paper's finer */
                             /* BP granularity, Section III-C)                */
  int32_t hybrid_from;       /* 0: every node row-centric. k in [2, n-1]: the  */
                             /* hybrid variants (2PS-H / OverL-H, checkpoints  */
                             /* integrated with row partitioning, Sections     */
                             /* IV-A and IV-B): nodes 0..k-1 are row-centric,  */
                             /* node k-1 is a checkpoint kept at full size,   */
                             /* nodes k..n-1 run layer-wise over whole maps.  */
                             /* No node >= k may read a node below k-1.        */
                             /* LRCNN_HYBRID_AUTO (-1): the planner takes the  */
                             /* valid k with the smallest workspace (0 if no   */
                             /* checkpoint beats the all-row-centric plan).    */
  int32_t first_rows;        /* PAPER_2PS: H_1^L, rows of the last node that  */
                             /* the first band completes (0: ceil(H_L/N_BP)); */
                             /* ignored by the other policies                 */
} lrcnn_config;

/* Opaque plan handle (host memory only). */
typedef struct lrcnn_plan_s lrcnn_plan_t;

/* Analytic figures of a plan. Byte counts include the batch. */
typedef struct {
  int32_t n_nodes, n_bands, mode, dtype;  /* n_bands: forward bands          */
  int32_t out_h, out_w, out_c;
  size_t workspace_bytes;          /* forward_rows + backward_rows          */
  size_t layerwise_workspace_bytes;/* lrcnn_layerwise_reference_gpu         */
  size_t strip_bytes;              /* CARRY: shared rows kept FP -> BP      */
  size_t band_cache_bytes;         /* largest band's cached feature maps    */
  size_t delta_bytes;              /* float32 error windows (peak)          */
  size_t carry_bytes;              /* CARRY: float32 error carried to r-1   */
  size_t partial_bytes;            /* weight-gradient partial sums          */
  double omega_bytes;              /* Eq. (3): all node outputs, full size  */
  double omega_fp_bytes;           /* Eq. (7) analogue: peak of FP          */
  double omega_bp_bytes;           /* Eq. (8) analogue: peak of BP          */
  double flops_tau;                /* tau (Section IV-B): forward convs     */
  double flops_rows;               /* FLOPs of forward_rows+backward_rows   */
  double flops_layerwise;          /* 3 tau                                 */
  int64_t shared_rows;             /* CARRY: sum of kept rows over bands    */
  int64_t halo_rows;               /* RECOMPUTE: rows computed by more than */
                                   /* one band, summed over nodes and bands */
  int32_t bp_bands;                /* backward bands (n_bands * bp_refine)  */
  size_t fp_window_bytes;          /* forward windows (lifetime-packed when */
                                   /* bp_refine > 1, else the band cache)   */
  int32_t hybrid_from;             /* the checkpoint in use (0: none); the  */
                                   /* planner's choice for LRCNN_HYBRID_AUTO */
} lrcnn_plan_info;

/* Build a plan: shapes of every node, per-band row intervals, workspace
 * layout, analytic memory (Eqs. (3), (7), (8), (12)) and FLOPs (tau,
 * Section IV-B). Pure host code; needs no GPU. `nodes`, `cfg` and
 * `cfg->bounds` are read during the call only. On success *out owns a plan
 * that the caller releases with lrcnn_plan_destroy.
 * Errors: EINVAL (null pointer, bad enum, a hybrid checkpoint that an edge
 * crosses), ESHAPE (bad ids, channel or size mismatch, a layer with empty
 * output), EPARTITION (bad bounds). */
int lrcnn_plan(const lrcnn_node *nodes, int32_t n_nodes,
               const lrcnn_config *cfg, lrcnn_plan_t **out);

/* Fill *info. Errors: EINVAL on null. */
int lrcnn_plan_query(const lrcnn_plan_t *plan, lrcnn_plan_info *info);

/* Output shape of node `node`: shape = {H, W, C}. Errors: EINVAL. */
int lrcnn_plan_node_shape(const lrcnn_plan_t *plan, int32_t node,
                          int32_t shape[3]);

/* Rows of node `node` in band `band` (0-based) of the forward (phase 0) or
 * backward (phase 1) partition: rows[0..1] = the rows the band computes and
 * owns [a, b); rows[2..3] = the rows it holds [lo, hi) (CARRY: own rows plus
 * the rows shared from earlier bands; RECOMPUTE: the band's receptive cone).
 * Errors: EINVAL. */
int lrcnn_plan_band_rows(const lrcnn_plan_t *plan, int32_t phase, int32_t band,
                         int32_t node, int32_t rows[4]);

void lrcnn_plan_destroy(lrcnn_plan_t *plan);

/* Device bytes of one training step under `plan`: the workspace
 * (row-centric, or layer-wise when layerwise != 0) plus the xi of
 * Eqs. (9)-(10) -- every other buffer the step touches: x, y, dy (storage
 * dtype), the weights (storage dtype), their float32 gradients, the float32
 * affine scale and shift, and dx when want_dx != 0. Each buffer is counted
 * at the 256-byte granularity the library uses; a caller's allocator may
 * round further. Errors: EINVAL on null. */
int lrcnn_plan_step_bytes(const lrcnn_plan_t *plan, int32_t layerwise,
                          int32_t want_dx, size_t *bytes);

/* Memory budget of the budget-driven planner and the batch search. */
typedef struct {
  size_t budget_bytes;  /* M: device bytes the step may use               */
  int32_t max_bands;    /* largest N_BP tried; 0: min(256, partitioned   */
                        /* height: input rows in CARRY, output rows in    */
                        /* RECOMPUTE)                                     */
  int32_t max_refine;   /* largest N_BP / N_FP tried (0 reads as 1)       */
  int32_t want_dx;      /* count dx in xi                                 */
} lrcnn_budget;

/* Budget-driven row granularity (Section III-C, Eqs. (9)-(10); the memory
 * bound of 2PS, Eq. (12), and of OverL, Section IV-B): the plan with the
 * smallest backward band count N_BP = N whose step fits the budget
 * (lrcnn_plan_step_bytes(plan, 0, want_dx) <= budget_bytes), and for that
 * N_BP the smallest forward band count N_FP (a divisor of N_BP with
 * N_BP / N_FP <= max_refine). Small N is preferred because it gives the
 * kernels the most parallel work (the paper's second principle). The exact
 * workspace of each candidate plan stands in for the paper's analytic
 * Omega, so the strips, error windows and split-K buffers are counted too.
 * cfg->n_bands and cfg->bp_refine are ignored; cfg->policy must be EVEN,
 * BALANCED or PAPER_2PS. Candidates are tried in increasing (N_BP, N_FP)
 * order, each a full host-side plan (milliseconds). With PAPER_2PS each
 * (N_BP, N_FP) also tries H_1^L from H_L down to ceil(H_L / N_BP) and takes
 * the largest that fits (Eq. (12): the largest first band, the fewest
 * bands); cfg->first_rows is ignored.
 * Errors: EINVAL (null, EXPLICIT policy, bad budget), the errors of
 * lrcnn_plan, EINFEASIBLE (no candidate up to max_bands fits). */
int lrcnn_plan_for_budget(const lrcnn_node *nodes, int32_t n_nodes,
                          const lrcnn_config *cfg, const lrcnn_budget *budget,
                          lrcnn_plan_t **out);

/* Largest batch whose step fits the budget: the largest B with
 * lrcnn_plan_step_bytes(plan(B), layerwise, want_dx) <= budget_bytes, for
 * the row-centric step of cfg (layerwise == 0) or the layer-wise baseline
 * (layerwise != 0) -- the paper's largest-batch comparison (Section V).
 * cfg->batch is ignored; budget->max_bands and max_refine are unused. The
 * search doubles B until the step no longer fits (at most 2^24), then
 * bisects; step bytes grow with B. On success *batch >= 1.
 * Errors: EINVAL (null), the errors of lrcnn_plan, EINFEASIBLE (B = 1 does
 * not fit). */
int lrcnn_max_batch(const lrcnn_node *nodes, int32_t n_nodes,
                    const lrcnn_config *cfg, int32_t layerwise,
                    const lrcnn_budget *budget, int32_t *batch);

/* Row-centric FP (Algorithm 1, FP loop): writes y. In CARRY mode the rows
 * shared between bands are left in `workspace` for lrcnn_backward_rows.
 * mask_out (nullable host array; entries nullable): per node a device
 * uint8 [B][H][W][C] buffer that receives the ReLU mask (1 where the output
 * is > 0) of CONV/ADD nodes with ReLU and the argmax (row-major index inside
 * the window) of MAXPOOL nodes.
 * Errors: EINVAL, EWORKSPACE (ws_bytes < workspace_bytes), EHIP. */
int lrcnn_forward_rows(lrcnn_plan_t *plan, const void *x,
                       const void *const *w,
                       const float *const *aff_scale,
                       const float *const *aff_shift,
                       void *y, void *workspace, size_t ws_bytes,
                       void *const *mask_out, void *stream);

/* Allocation-free lrcnn_forward_rows, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc). The workspace is the library's own
 * static device array of LRCNN_STATIC_WORKSPACE_BYTES (64 MiB), one per
 * device, held from the library's load until the process ends; its device
 * address is looked up once per device on the first call there. The call
 * allocates no device memory; the caller still owns x, w, aff_*, y and
 * mask_out, with the meaning, layout and results of lrcnn_forward_rows.
 * Every call on a device shares that device's array, which keeps the last
 * call's contents (the forward initialises every row it reads): calls that
 * overlap on one device (several streams or threads) race. A later
 * lrcnn_backward_rows cannot use this forward's shared rows (ESTATE).
 * Errors: as lrcnn_forward_rows; EWORKSPACE when the plan's workspace_bytes
 * exceed LRCNN_STATIC_WORKSPACE_BYTES; EHIP when the array's device address
 * cannot be obtained. */
#define LRCNN_STATIC_WORKSPACE_BYTES (64u << 20)
int lrcnn_forward_rows_static(lrcnn_plan_t *plan, const void *x,
                              const void *const *w,
                              const float *const *aff_scale,
                              const float *const *aff_shift, void *y,
                              void *const *mask_out, void *stream);

/* Row-centric BP (Algorithm 1, BP loop), bands in reverse: recompute each
 * band, propagate the error dy = dL/dy, overwrite dw[node] (float32,
 * [C_out][kh][kw][C_in]) with the weight gradient of every conv node and,
 * when dx != NULL, write dL/dx. CARRY mode needs the workspace of the
 * preceding lrcnn_forward_rows on this plan, unchanged.
 * Errors: EINVAL, EWORKSPACE, ESTATE (CARRY without a preceding forward on
 * this plan and workspace), EHIP. */
int lrcnn_backward_rows(lrcnn_plan_t *plan, const void *x,
                        const void *const *w,
                        const float *const *aff_scale,
                        const float *const *aff_shift,
                        const void *dy, float *const *dw, void *dx,
                        void *workspace, size_t ws_bytes, void *stream);

/* Layer-by-layer ("column", Eqs. (1)-(3)) training step on the GPU with the
 * same kernels: full-height feature maps of every node are kept from FP to
 * BP and nothing is recomputed. Writes y, dw and (if non-NULL) dx and
 * mask_out as above. Needs layerwise_workspace_bytes of workspace.
 * Errors: EINVAL, EWORKSPACE, EHIP. */
int lrcnn_layerwise_reference_gpu(lrcnn_plan_t *plan, const void *x,
                                  const void *const *w,
                                  const float *const *aff_scale,
                                  const float *const *aff_shift,
                                  const void *dy, void *y, float *const *dw,
                                  void *dx, void *workspace, size_t ws_bytes,
                                  void *const *mask_out, void *stream);

/* ---- Full training step: classifier head, loss, update (Algorithm 1:
 * fully connected FP, Loss, fully connected BP after the last band's FP, and
 * the parameter update once every band's BP is done). Readings: one fully
 * connected layer over the trunk output flattened per image in NHWC order
 * (K = H_L * W_L * C_L features), softmax cross-entropy averaged over the
 * batch, plain SGD; the fixed affine parameters are not trained. */

/* Device scratch bytes lrcnn_head_loss needs for n_classes classes (1..64).
 * Errors: EINVAL. */
int lrcnn_head_workspace_bytes(const lrcnn_plan_t *plan, int32_t n_classes,
                               size_t *bytes);

/* y: the trunk output written by lrcnn_forward_rows (plan dtype,
 * [B][H_L][W_L][C_L]); fc_w: float32 [n_classes][K]; fc_b: float32
 * [n_classes]; labels: int32 [B] in [0, n_classes). Writes logits (float32
 * [B][n_classes]), loss (one float32: the batch mean), dy = dL/dy (plan
 * dtype, shape of y: the upstream gradient for lrcnn_backward_rows),
 * d_fc_w and d_fc_b (float32, overwritten). head_ws: device scratch of
 * lrcnn_head_workspace_bytes. A label outside [0, n_classes) makes the loss
 * NaN (nothing is read out of bounds). All device pointers 16-byte aligned.
 * Errors: EINVAL, EWORKSPACE, EHIP. */
int lrcnn_head_loss(const lrcnn_plan_t *plan, const void *y, const float *fc_w,
                    const float *fc_b, const int32_t *labels, int32_t n_classes,
                    float *logits, float *loss, void *dy, float *d_fc_w,
                    float *d_fc_b, void *head_ws, size_t head_ws_bytes,
                    void *stream);

/* theta <- theta - lr * g for every conv node's weights w[v] (plan dtype,
 * updated in float32 and rounded to the storage dtype) with dw[v] (float32,
 * from lrcnn_backward_rows), and, when fc_w is not NULL, for the head
 * (fc_w, fc_b with d_fc_w, d_fc_b; n_classes classes). Errors: EINVAL,
 * EHIP. */
int lrcnn_sgd_update(const lrcnn_plan_t *plan, float lr, void *const *w,
                     float *const *dw, float *fc_w, const float *d_fc_w,
                     float *fc_b, const float *d_fc_b, int32_t n_classes,
                     void *stream);

/* Message of the last failed call on this thread ("" if none). */
const char *lrcnn_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* LRCNN_H */
