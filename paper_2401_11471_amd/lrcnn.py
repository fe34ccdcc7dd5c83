"""ctypes binding of liblrcnn.so (include/lrcnn.h): argument marshalling only.

Every step of row-centric training runs in the HIP library; this module
converts Python values and torch tensors into the C ABI's plain pointers and
sizes. Device memory comes from torch; streams are torch's current stream.
If the library has not been built, importing this module raises.
"""
from __future__ import annotations

import ctypes as C
import os

# torch first: it brings its own HIP runtime, and liblrcnn.so must bind to
# that same runtime (one HIP/HSA runtime per process). Loading the library
# first would load the system runtime and leave torch and the library on
# different ones.
import torch  # noqa: F401

HERE = os.path.dirname(os.path.abspath(__file__))
# (LRCNN_LIB_PATH: another build of the library, e.g. a variant under test)
LIB_PATH = os.environ.get("LRCNN_LIB_PATH") or os.path.join(HERE, "liblrcnn.so")

OP_INPUT, OP_CONV, OP_MAXPOOL, OP_ADD = 0, 1, 2, 3
F32, BF16 = 0, 1
CARRY, RECOMPUTE = 0, 1
EVEN, BALANCED, EXPLICIT, PAPER_2PS = 0, 1, 2, 3
HYBRID_AUTO = -1

STATUS = {0: "OK", -1: "EINVAL", -2: "ESHAPE", -3: "EPARTITION",
          -4: "EWORKSPACE", -5: "ESTATE", -6: "EDTYPE", -7: "EHIP",
          -8: "EINFEASIBLE"}


class LrcnnError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{STATUS.get(code, code)}: {msg}")
        self.code = code


class Node(C.Structure):
    _fields_ = [(f, C.c_int32) for f in ("op", "in0", "in1", "c_out", "kh", "kw",
                                         "sh", "sw", "ph", "pw", "affine", "relu")]


class Config(C.Structure):
    _fields_ = [("batch", C.c_int32), ("in_c", C.c_int32), ("in_h", C.c_int32),
                ("in_w", C.c_int32), ("dtype", C.c_int32), ("mode", C.c_int32),
                ("n_bands", C.c_int32), ("policy", C.c_int32),
                ("bounds", C.POINTER(C.c_int32)), ("bp_refine", C.c_int32),
                ("hybrid_from", C.c_int32), ("first_rows", C.c_int32)]


class PlanInfo(C.Structure):
    _fields_ = [("n_nodes", C.c_int32), ("n_bands", C.c_int32), ("mode", C.c_int32),
                ("dtype", C.c_int32), ("out_h", C.c_int32), ("out_w", C.c_int32),
                ("out_c", C.c_int32),
                ("workspace_bytes", C.c_size_t), ("layerwise_workspace_bytes", C.c_size_t),
                ("strip_bytes", C.c_size_t), ("band_cache_bytes", C.c_size_t),
                ("delta_bytes", C.c_size_t), ("carry_bytes", C.c_size_t),
                ("partial_bytes", C.c_size_t),
                ("omega_bytes", C.c_double), ("omega_fp_bytes", C.c_double),
                ("omega_bp_bytes", C.c_double), ("flops_tau", C.c_double),
                ("flops_rows", C.c_double), ("flops_layerwise", C.c_double),
                ("shared_rows", C.c_int64), ("halo_rows", C.c_int64),
                ("bp_bands", C.c_int32), ("fp_window_bytes", C.c_size_t),
                ("hybrid_from", C.c_int32)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


class Budget(C.Structure):
    _fields_ = [("budget_bytes", C.c_size_t), ("max_bands", C.c_int32),
                ("max_refine", C.c_int32), ("want_dx", C.c_int32)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build the HIP library first "
            "(python -c 'import __graft_entry__ as g; g.build()')")
    lib = C.CDLL(LIB_PATH)
    vp, sz, i32 = C.c_void_p, C.c_size_t, C.c_int32
    pp = C.POINTER(C.c_void_p)
    lib.lrcnn_plan.argtypes = [C.POINTER(Node), i32, C.POINTER(Config), C.POINTER(vp)]
    lib.lrcnn_plan_query.argtypes = [vp, C.POINTER(PlanInfo)]
    lib.lrcnn_plan_node_shape.argtypes = [vp, i32, C.POINTER(i32)]
    lib.lrcnn_plan_band_rows.argtypes = [vp, i32, i32, i32, C.POINTER(i32)]
    lib.lrcnn_plan_destroy.argtypes = [vp]
    lib.lrcnn_plan_step_bytes.argtypes = [vp, i32, i32, C.POINTER(sz)]
    lib.lrcnn_plan_for_budget.argtypes = [C.POINTER(Node), i32, C.POINTER(Config),
                                          C.POINTER(Budget), C.POINTER(vp)]
    lib.lrcnn_max_batch.argtypes = [C.POINTER(Node), i32, C.POINTER(Config), i32,
                                    C.POINTER(Budget), C.POINTER(i32)]
    lib.lrcnn_plan_destroy.restype = None
    lib.lrcnn_forward_rows.argtypes = [vp, vp, pp, pp, pp, vp, vp, sz, pp, vp]
    lib.lrcnn_forward_rows_static.argtypes = [vp, vp, pp, pp, pp, vp, pp, vp]
    lib.lrcnn_backward_rows.argtypes = [vp, vp, pp, pp, pp, vp, pp, vp, vp, sz, vp]
    lib.lrcnn_layerwise_reference_gpu.argtypes = [vp, vp, pp, pp, pp, vp, vp, pp, vp,
                                                  vp, sz, pp, vp]
    lib.lrcnn_head_workspace_bytes.argtypes = [vp, i32, C.POINTER(sz)]
    lib.lrcnn_head_loss.argtypes = [vp, vp, vp, vp, vp, i32, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.lrcnn_sgd_update.argtypes = [vp, C.c_float, pp, pp, vp, vp, vp, vp, i32, vp]
    lib.lrcnn_last_error.restype = C.c_char_p
    lib.lrcnn_debug_dry_run.argtypes = [C.c_int]
    lib.lrcnn_debug_dry_run.restype = None
    lib.lrcnn_debug_fp_pipeline.argtypes = [C.c_int]
    lib.lrcnn_debug_fp_pipeline.restype = None
    lib.lrcnn_debug_act_fusion.argtypes = [C.c_int]
    lib.lrcnn_debug_act_fusion.restype = None
    lib.lrcnn_debug_serial_wgrad.argtypes = [C.c_int]
    lib.lrcnn_debug_serial_wgrad.restype = None
    lib.lrcnn_debug_dgrad_phases.argtypes = [C.c_int]
    lib.lrcnn_debug_dgrad_phases.restype = None
    lib.lrcnn_debug_profile.argtypes = [C.c_int]
    lib.lrcnn_debug_profile.restype = None
    lib.lrcnn_debug_profile_collect.restype = C.c_int
    lib.lrcnn_debug_profile_entry.argtypes = [i32, C.POINTER(C.c_char_p),
                                              C.POINTER(C.c_int64),
                                              C.POINTER(C.c_double), C.POINTER(C.c_double)]
    lib.lrcnn_debug_profile_entry.restype = C.c_int
    lib.lrcnn_debug_profile_roofline.argtypes = [i32, C.POINTER(C.c_double),
                                                 C.POINTER(C.c_double)]
    lib.lrcnn_debug_profile_roofline.restype = C.c_int
    lib.lrcnn_debug_layerwise_map.argtypes = [vp, i32, C.POINTER(sz)]
    lib.lrcnn_debug_layerwise_map.restype = C.c_int
    for f in ("lrcnn_plan", "lrcnn_plan_query", "lrcnn_plan_node_shape",
              "lrcnn_plan_band_rows", "lrcnn_forward_rows", "lrcnn_forward_rows_static",
              "lrcnn_backward_rows",
              "lrcnn_layerwise_reference_gpu", "lrcnn_plan_step_bytes",
              "lrcnn_plan_for_budget", "lrcnn_max_batch", "lrcnn_head_workspace_bytes",
              "lrcnn_head_loss", "lrcnn_sgd_update"):
        getattr(lib, f).restype = C.c_int
    return lib


LIB = _load()

# Names the header declares (checked by the tests against the shared object).
EXPORTS = ("lrcnn_plan", "lrcnn_plan_query", "lrcnn_plan_node_shape",
           "lrcnn_plan_band_rows", "lrcnn_plan_destroy", "lrcnn_plan_step_bytes",
           "lrcnn_plan_for_budget", "lrcnn_max_batch", "lrcnn_head_workspace_bytes",
           "lrcnn_head_loss", "lrcnn_sgd_update", "lrcnn_forward_rows",
           "lrcnn_forward_rows_static",
           "lrcnn_backward_rows", "lrcnn_layerwise_reference_gpu", "lrcnn_last_error",
           "lrcnn_debug_dry_run", "lrcnn_debug_fp_pipeline", "lrcnn_debug_act_fusion",
           "lrcnn_debug_dgrad_phases", "lrcnn_debug_serial_wgrad",
           "lrcnn_debug_profile",
           "lrcnn_debug_profile_collect", "lrcnn_debug_profile_entry",
           "lrcnn_debug_profile_roofline",
           "lrcnn_debug_layerwise_map")


def _check(code):
    if code != 0:
        raise LrcnnError(code, LIB.lrcnn_last_error().decode())


class Plan:
    """Owns an lrcnn_plan_t handle."""

    def __init__(self, handle, nodes):
        self.handle = handle
        self.nodes = list(nodes)
        self.n = len(self.nodes)

    def __del__(self):
        if getattr(self, "handle", None) and LIB is not None:
            LIB.lrcnn_plan_destroy(self.handle)
            self.handle = None

    def info(self):
        inf = PlanInfo()
        _check(LIB.lrcnn_plan_query(self.handle, C.byref(inf)))
        return inf.as_dict()

    def node_shape(self, v):
        out = (C.c_int32 * 3)()
        _check(LIB.lrcnn_plan_node_shape(self.handle, v, out))
        return tuple(out)

    def step_bytes(self, layerwise=False, want_dx=False):
        """Workspace plus every other buffer of one step (the xi of
        Eqs. (9)-(10)), in bytes."""
        out = C.c_size_t()
        _check(LIB.lrcnn_plan_step_bytes(self.handle, 1 if layerwise else 0,
                                         1 if want_dx else 0, C.byref(out)))
        return out.value

    def band_rows(self, band, v, phase=1):
        """Rows (a, b, lo, hi) of node v in a backward (phase 1) or forward
        (phase 0) band."""
        out = (C.c_int32 * 4)()
        _check(LIB.lrcnn_plan_band_rows(self.handle, phase, band, v, out))
        return tuple(out)


def lrcnn_plan(nodes, batch, in_c, in_h, in_w, dtype=F32, mode=CARRY, n_bands=1,
               policy=EVEN, bounds=None, bp_refine=1, hybrid_from=0, first_rows=0):
    arr = (Node * len(nodes))(*[Node(*nd) for nd in nodes])
    cfg = Config(batch, in_c, in_h, in_w, dtype, mode, n_bands, policy, None, bp_refine,
                 hybrid_from, first_rows)
    keep = None
    if bounds is not None:
        keep = (C.c_int32 * len(bounds))(*bounds)
        cfg.bounds = C.cast(keep, C.POINTER(C.c_int32))
    h = C.c_void_p()
    _check(LIB.lrcnn_plan(arr, len(nodes), C.byref(cfg), C.byref(h)))
    return Plan(h, nodes)


def _node_cfg(nodes, batch, in_c, in_h, in_w, dtype, mode, n_bands, policy, bp_refine,
              hybrid_from, first_rows=0):
    arr = (Node * len(nodes))(*[Node(*nd) for nd in nodes])
    return arr, Config(batch, in_c, in_h, in_w, dtype, mode, n_bands, policy, None,
                       bp_refine, hybrid_from, first_rows)


def lrcnn_plan_for_budget(nodes, batch, in_c, in_h, in_w, budget_bytes, dtype=F32,
                          mode=CARRY, policy=EVEN, max_bands=0, max_refine=1,
                          want_dx=False, hybrid_from=0):
    """Smallest (N_BP, N_FP) whose step fits budget_bytes (Eqs. (9)-(10))."""
    arr, cfg = _node_cfg(nodes, batch, in_c, in_h, in_w, dtype, mode, 1, policy, 1,
                         hybrid_from)
    bud = Budget(int(budget_bytes), max_bands, max_refine, 1 if want_dx else 0)
    h = C.c_void_p()
    _check(LIB.lrcnn_plan_for_budget(arr, len(nodes), C.byref(cfg), C.byref(bud),
                                     C.byref(h)))
    return Plan(h, nodes)


def lrcnn_max_batch(nodes, in_c, in_h, in_w, budget_bytes, dtype=F32, mode=CARRY,
                    n_bands=1, policy=EVEN, bp_refine=1, hybrid_from=0, layerwise=False,
                    want_dx=False):
    """Largest batch whose row-centric (or layer-wise) step fits budget_bytes."""
    arr, cfg = _node_cfg(nodes, 1, in_c, in_h, in_w, dtype, mode, n_bands, policy,
                         bp_refine, hybrid_from)
    bud = Budget(int(budget_bytes), 0, 1, 1 if want_dx else 0)
    out = C.c_int32()
    _check(LIB.lrcnn_max_batch(arr, len(nodes), C.byref(cfg), 1 if layerwise else 0,
                               C.byref(bud), C.byref(out)))
    return out.value


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _ptr_array(ts):
    return (C.c_void_p * len(ts))(*[None if t is None else t.data_ptr() for t in ts])


def _stream(stream):
    if stream is not None:
        return C.c_void_p(stream)
    import torch
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def lrcnn_forward_rows(plan, x, weights, scales, shifts, y, workspace, masks=None,
                       stream=None):
    """weights/scales/shifts/masks: per-node lists (None where unused)."""
    _check(LIB.lrcnn_forward_rows(
        plan.handle, _ptr(x), _ptr_array(weights), _ptr_array(scales),
        _ptr_array(shifts), _ptr(y), _ptr(workspace), workspace.numel(),
        _ptr_array(masks) if masks is not None else None, _stream(stream)))


def lrcnn_forward_rows_static(plan, x, weights, scales, shifts, y, masks=None, stream=None):
    """lrcnn_forward_rows on the library's static device workspace (no
    workspace argument; the call allocates nothing)."""
    _check(LIB.lrcnn_forward_rows_static(
        plan.handle, _ptr(x), _ptr_array(weights), _ptr_array(scales),
        _ptr_array(shifts), _ptr(y),
        _ptr_array(masks) if masks is not None else None, _stream(stream)))


STATIC_WORKSPACE_BYTES = 64 << 20


def lrcnn_backward_rows(plan, x, weights, scales, shifts, dy, dws, dx, workspace,
                        stream=None):
    _check(LIB.lrcnn_backward_rows(
        plan.handle, _ptr(x), _ptr_array(weights), _ptr_array(scales),
        _ptr_array(shifts), _ptr(dy), _ptr_array(dws), _ptr(dx), _ptr(workspace),
        workspace.numel(), _stream(stream)))


def lrcnn_layerwise_reference_gpu(plan, x, weights, scales, shifts, dy, y, dws, dx,
                                  workspace, masks=None, stream=None):
    _check(LIB.lrcnn_layerwise_reference_gpu(
        plan.handle, _ptr(x), _ptr_array(weights), _ptr_array(scales),
        _ptr_array(shifts), _ptr(dy), _ptr(y), _ptr_array(dws), _ptr(dx),
        _ptr(workspace), workspace.numel(),
        _ptr_array(masks) if masks is not None else None, _stream(stream)))


def lrcnn_head_workspace_bytes(plan, n_classes):
    out = C.c_size_t()
    _check(LIB.lrcnn_head_workspace_bytes(plan.handle, n_classes, C.byref(out)))
    return out.value


def lrcnn_head_loss(plan, y, fc_w, fc_b, labels, logits, loss, dy, d_fc_w, d_fc_b, head_ws,
                    stream=None):
    """Classifier head + softmax cross-entropy: logits, loss, dL/dy, head
    gradients (all device tensors; n_classes = fc_w.shape[0])."""
    _check(LIB.lrcnn_head_loss(
        plan.handle, _ptr(y), _ptr(fc_w), _ptr(fc_b), _ptr(labels), fc_w.shape[0],
        _ptr(logits), _ptr(loss), _ptr(dy), _ptr(d_fc_w), _ptr(d_fc_b), _ptr(head_ws),
        head_ws.numel(), _stream(stream)))


def lrcnn_sgd_update(plan, lr, weights, dws, fc_w=None, d_fc_w=None, fc_b=None, d_fc_b=None,
                     stream=None):
    """theta -= lr * g for every conv weight and (when given) the head."""
    n_classes = fc_w.shape[0] if fc_w is not None else 0
    _check(LIB.lrcnn_sgd_update(
        plan.handle, C.c_float(lr), _ptr_array(weights), _ptr_array(dws), _ptr(fc_w),
        _ptr(d_fc_w), _ptr(fc_b), _ptr(d_fc_b), n_classes, _stream(stream)))


def lrcnn_debug_dry_run(on):
    """Test hook: walk schedules with all host checks but launch nothing."""
    LIB.lrcnn_debug_dry_run(1 if on else 0)


def lrcnn_debug_fp_pipeline(on):
    """Test hook: forward bands pipelined on two streams (on) or sequential (off,
    the default)."""
    LIB.lrcnn_debug_fp_pipeline(1 if on else 0)


def lrcnn_debug_serial_wgrad(on):
    """Test hook: weight gradients on the caller's stream (on) or on the plan's
    side stream beside the input gradients (off, the default)."""
    LIB.lrcnn_debug_serial_wgrad(1 if on else 0)


def lrcnn_debug_act_fusion(on):
    """Test hook: error operands formed by the consumer's input gradient (on) or
    by their own activation-backward pass (off)."""
    LIB.lrcnn_debug_act_fusion(1 if on else 0)


def lrcnn_debug_dgrad_phases(mode):
    """Test hook: strided input gradients by phase (0 estimate, 1 always, 2 never)."""
    LIB.lrcnn_debug_dgrad_phases(int(mode))


def lrcnn_debug_profile(on):
    """Test hook: time every matrix-core kernel launch with HIP events."""
    LIB.lrcnn_debug_profile(1 if on else 0)


def lrcnn_debug_profile_collect(roofline=False):
    """Per-kernel aggregate of the recorded launches (streams synchronised
    by the caller): {name: (launches, ms, flops)}, with roofline also the
    summed algorithmic bytes and roofline ms: (launches, ms, flops, bytes,
    roofline_ms)."""
    n = LIB.lrcnn_debug_profile_collect()
    if n < 0:
        raise LrcnnError(-7, "profile collection failed")
    out = {}
    for i in range(n):
        nm, la, ms, fl = C.c_char_p(), C.c_int64(), C.c_double(), C.c_double()
        LIB.lrcnn_debug_profile_entry(i, C.byref(nm), C.byref(la), C.byref(ms), C.byref(fl))
        if roofline:
            by, rf = C.c_double(), C.c_double()
            LIB.lrcnn_debug_profile_roofline(i, C.byref(by), C.byref(rf))
            out[nm.value.decode()] = (la.value, ms.value, fl.value, by.value, rf.value)
        else:
            out[nm.value.decode()] = (la.value, ms.value, fl.value)
    return out


def lrcnn_debug_layerwise_map(plan, node):
    """Test hook: byte offset of node's full map in the layer-wise workspace,
    or None where the map is not stored there (input, output, fused conv)."""
    out = C.c_size_t()
    code = LIB.lrcnn_debug_layerwise_map(plan.handle, node, C.byref(out))
    return out.value if code == 0 else None
