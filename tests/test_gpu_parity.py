"""GPU parity: the HIP library (through its C ABI) against the CPU oracle on
the same seeded inputs. Sizes span several 128-wide tiles with ragged tails,
channel counts on and off the 16-byte vector paths, strides, pooling,
residual adds, empty bands and every schedule (two-phase sharing,
overlapping recompute, layer-wise)."""
import numpy as np
import pytest
import torch

from gpu_harness import assert_parity, gpu_run, hybrid_cuts, rel
from paper_2401_11471_amd import lrcnn as L
from workloads import NetBuilder, Inputs, config_inputs, tiny_net, F32, BF16

pytestmark = pytest.mark.gpu


def vgg_like(c=(16, 24, 40)):
    nb = NetBuilder()
    v = nb.conv(0, c[0], 3, 1, 1)
    v = nb.conv(v, c[0], 3, 1, 1)
    v = nb.pool(v, 2, 2, 0)
    v = nb.conv(v, c[1], 3, 1, 1)
    v = nb.pool(v, 2, 2, 0)
    v = nb.conv(v, c[2], 3, 1, 1)
    return nb.nodes


def wide_chain():
    # N = 136 and 200 span two 128-wide tiles; C_in = 72 leaves a partial
    # 16/32-element K chunk
    nb = NetBuilder()
    v = nb.conv(0, 72, 3, 1, 1)
    v = nb.conv(v, 136, 3, 1, 1)
    v = nb.conv(v, 200, 1, 1, 0, affine=1, relu=0)
    return nb.nodes


def odd_chain():
    # channel counts off the vector paths, even windows, stride 3
    nb = NetBuilder()
    v = nb.conv(0, 5, 5, 2, 2)
    v = nb.conv(v, 6, 2, 1, 0)
    v = nb.pool(v, 3, 2, 1)
    v = nb.conv(v, 3, 4, 3, 1)
    nb.conv(v, 7, 1, 1, 0)
    return nb.nodes


def resnet_like():
    nb = NetBuilder()
    a = nb.conv(0, 16, 7, 2, 3, affine=1)
    b = nb.pool(a, 3, 2, 1)
    c1 = nb.conv(b, 16, 1, 1, 0, affine=1)
    c2 = nb.conv(c1, 16, 3, 2, 1, affine=1)
    c3 = nb.conv(c2, 64, 1, 1, 0, affine=1, relu=0)
    sc = nb.conv(b, 64, 1, 2, 0, affine=1, relu=0)
    s = nb.sum(c3, sc)
    d1 = nb.conv(s, 16, 1, 1, 0, affine=1)
    d2 = nb.conv(d1, 16, 3, 1, 1, affine=1)
    d3 = nb.conv(d2, 64, 1, 1, 0, affine=1, relu=0)
    nb.sum(d3, s)
    return nb.nodes


NETS = {"tiny": (tiny_net(), 32, 32), "vgg_like": (vgg_like(), 44, 37),
        "wide": (wide_chain(), 29, 23), "odd": (odd_chain(), 47, 41),
        "resnet_like": (resnet_like(), 61, 45)}


def _inputs(name, dtype, batch=2, seed=0):
    nodes, h, w = NETS[name]
    return nodes, Inputs(nodes, batch, h, w, 3, dtype, seed=seed + 17)


def test_config1_tiny_parity():
    nodes, inp = config_inputs(1)
    gpu = gpu_run(nodes, inp, L.CARRY, 4)
    errs, nbad = assert_parity(nodes, inp, gpu)
    assert nbad == 0, "config 1 ReLU masks must equal the oracle's"
    print("config1", {k: f"{e:.1e}" for k, e in errs.items()})


@pytest.mark.parametrize("dtype", [F32, BF16])
@pytest.mark.parametrize("name", list(NETS))
def test_carry_parity(name, dtype):
    nodes, inp = _inputs(name, dtype)
    gpu = gpu_run(nodes, inp, L.CARRY, 3)
    assert_parity(nodes, inp, gpu)


@pytest.mark.parametrize("dtype", [F32, BF16])
@pytest.mark.parametrize("name", ["vgg_like", "odd", "resnet_like"])
def test_carry_uneven_and_empty_bands(name, dtype):
    nodes, inp = _inputs(name, dtype, seed=3)
    h = inp.x.shape[1]
    bounds = [0, 0, 5, 5, 6, h // 2, h - 3, h, h]
    gpu = gpu_run(nodes, inp, L.CARRY, len(bounds) - 1, L.EXPLICIT, bounds)
    assert_parity(nodes, inp, gpu)


@pytest.mark.parametrize("dtype", [F32, BF16])
@pytest.mark.parametrize("name", list(NETS))
def test_recompute_parity(name, dtype):
    nodes, inp = _inputs(name, dtype, seed=5)
    gpu = gpu_run(nodes, inp, L.RECOMPUTE, 4)
    assert_parity(nodes, inp, gpu)


@pytest.mark.parametrize("dtype", [F32, BF16])
@pytest.mark.parametrize("name", ["vgg_like", "odd", "resnet_like"])
@pytest.mark.parametrize("mode", [L.CARRY, L.RECOMPUTE])
def test_finer_backward_partition_parity(name, dtype, mode):
    # Section III-C: BP bands refine the FP bands (N_BP = 3 N_FP here)
    nodes, inp = _inputs(name, dtype, seed=15)
    gpu = gpu_run(nodes, inp, mode, 3, bp_refine=3)
    assert_parity(nodes, inp, gpu)


@pytest.mark.parametrize("dtype", [F32, BF16])
@pytest.mark.parametrize("name", ["vgg_like", "odd", "resnet_like"])
@pytest.mark.parametrize("mode", [L.CARRY, L.RECOMPUTE])
@pytest.mark.parametrize("where", ["early", "late"])
def test_hybrid_depth_parity(name, dtype, mode, where):
    # 2PS-H / OverL-H: row-centric up to a checkpoint, layer-wise after it
    nodes, inp = _inputs(name, dtype, seed=17)
    cuts = hybrid_cuts(nodes)
    k = cuts[0] if where == "early" else cuts[-1]
    print(f"hybrid {name} dtype={dtype} mode={mode} hybrid_from={k}", flush=True)
    gpu = gpu_run(nodes, inp, mode, 3, hybrid_from=k)
    assert_parity(nodes, inp, gpu)


@pytest.mark.parametrize("name", ["vgg_like", "resnet_like"])
def test_hybrid_matches_row_centric_float32(name):
    # the checkpoint's error enters the row part in float32, so the hybrid
    # step equals the all-row-centric step to rounding
    nodes, inp = _inputs(name, F32, seed=19)
    ref = gpu_run(nodes, inp, L.CARRY, 4)
    for k in hybrid_cuts(nodes):
        hy = gpu_run(nodes, inp, L.CARRY, 4, hybrid_from=k)
        assert rel(hy["y"], ref["y"]) < 1e-5, k
        assert rel(hy["dx"], ref["dx"]) < 1e-4, k
        for v, (a, b) in enumerate(zip(hy["dw"], ref["dw"])):
            if b is not None:
                assert rel(a, b) < 1e-4, (k, v)


@pytest.mark.parametrize("dtype", [F32, BF16])
@pytest.mark.parametrize("name", list(NETS))
def test_layerwise_parity(name, dtype):
    nodes, inp = _inputs(name, dtype, seed=7)
    gpu = gpu_run(nodes, inp, layerwise=True)
    assert_parity(nodes, inp, gpu)


SCHEDULES = [("carry_even", dict(mode=L.CARRY, nb=5)),
             ("carry_balanced", dict(mode=L.CARRY, nb=4, policy=L.BALANCED)),
             ("carry_paper_2ps", dict(mode=L.CARRY, nb=3, policy=L.PAPER_2PS)),
             ("carry_refined", dict(mode=L.CARRY, nb=2, bp_refine=3)),
             ("recompute", dict(mode=L.RECOMPUTE, nb=3))]


@pytest.mark.parametrize("dtype", [F32, BF16])
@pytest.mark.parametrize("name", list(NETS))
def test_forward_bitwise_equals_layerwise(name, dtype):
    # a plan fixes every layer's split-K chunks for all its forward
    # launches, so the row-centric forward output and every ReLU / argmax
    # decision equal the same plan's layer-wise step bit for bit (gpu_run
    # checks this for every row-centric run); gradients agree with the
    # whole-map layer-wise step to rounding
    nodes, inp = _inputs(name, dtype, seed=9)
    lw = gpu_run(nodes, inp, layerwise=True)
    h = inp.x.shape[1]
    scheds = SCHEDULES + [("carry_empty_bands",
                           dict(mode=L.CARRY, nb=6, policy=L.EXPLICIT,
                                bounds=[0, 0, 5, h // 2, h // 2, h - 2, h])),
                          ("hybrid", dict(mode=L.CARRY, nb=3, hybrid_from=hybrid_cuts(nodes)[-1]))]
    gtol = 1e-5 if dtype == F32 else 2e-2
    for label, kw in scheds:
        print(f"{name} dtype={dtype} {label}", flush=True)
        rc = gpu_run(nodes, inp, **kw)
        for v in range(1, len(nodes)):
            if lw["dw"][v] is not None:
                assert rel(rc["dw"][v], lw["dw"][v]) < gtol, (label, v)
        assert rel(rc["dx"], lw["dx"]) < gtol, label
        assert rel(rc["y"], lw["y"]) < (1e-6 if dtype == F32 else 1e-2), label


@pytest.mark.parametrize("dtype", [F32, BF16])
@pytest.mark.parametrize("name", ["vgg_like", "odd", "resnet_like"])
@pytest.mark.parametrize("policy", [L.BALANCED, L.PAPER_2PS])
def test_partition_policy_parity(name, dtype, policy):
    # the peak-minimising and the paper's greedy placement (Section IV-A)
    nodes, inp = _inputs(name, dtype, seed=23)
    gpu = gpu_run(nodes, inp, L.CARRY, 4, policy)
    assert_parity(nodes, inp, gpu)


def test_weight_gradients_are_deterministic():
    nodes, inp = _inputs("resnet_like", F32, seed=11)
    gpu = gpu_run(nodes, inp, L.CARRY, 4, repeat_bwd=2)
    a, b = gpu["dw_runs"]
    for v in range(1, len(nodes)):
        if a[v] is not None:
            np.testing.assert_array_equal(a[v], b[v])


def test_no_input_gradient_requested():
    nodes, inp = _inputs("vgg_like", F32, seed=13)
    gpu = gpu_run(nodes, inp, L.CARRY, 3, want_dx=False)
    assert gpu["dx"] is None
    assert_parity(nodes, inp, gpu, check_dx=False)


def test_backward_without_forward_is_rejected():
    nodes, inp = _inputs("tiny", F32)
    b, h, w, c = inp.x.shape
    plan = L.lrcnn_plan(nodes, b, c, h, w, F32, L.CARRY, 2)
    from paper_2401_11471_amd.device import DeviceModel
    dm = DeviceModel.from_inputs(nodes, inp)
    ws = dm.workspace(plan.info()["workspace_bytes"])
    dy = dm.empty((b,) + plan.node_shape(len(nodes) - 1))
    with pytest.raises(L.LrcnnError) as e:
        L.lrcnn_backward_rows(plan, dm.x, dm.w, dm.sc, dm.sf, dy, dm.dw, None, ws)
    assert e.value.code == -5
    torch.cuda.synchronize()


@pytest.mark.parametrize("dtype", [F32, BF16])
def test_serial_weight_gradients_equal_overlapped(dtype):
    """Weight gradients on the caller's stream (the profiling schedule) give
    the same bits as the default schedule on the side stream."""
    nodes, inp = _inputs("resnet_like", dtype, seed=17)
    base = gpu_run(nodes, inp, L.CARRY, 4, twin=False)
    L.lrcnn_debug_serial_wgrad(True)
    try:
        ser = gpu_run(nodes, inp, L.CARRY, 4, twin=False)
    finally:
        L.lrcnn_debug_serial_wgrad(False)
    np.testing.assert_array_equal(base["dx"], ser["dx"])
    for v in range(1, len(nodes)):
        if base["dw"][v] is not None:
            np.testing.assert_array_equal(base["dw"][v], ser["dw"][v])


def test_profile_roofline_entries():
    """The profiling hook's per-kernel aggregates: every matrix-core kernel
    and reduction of a step carries algorithmic bytes and a roofline time,
    and the roofline time (per launch the larger of FLOPs at the matrix-core
    peak and bytes at the HBM peak) never exceeds the measured time."""
    from paper_2401_11471_amd.device import DeviceModel
    nodes, inp = _inputs("resnet_like", BF16, seed=19)
    b, h, w, c = inp.x.shape
    plan = L.lrcnn_plan(nodes, b, c, h, w, BF16, L.CARRY, 4)
    dm = DeviceModel.from_inputs(nodes, inp)
    oshape = (b,) + plan.node_shape(len(nodes) - 1)
    y = dm.empty(oshape)
    dy = dm.to_device(inp.grad(oshape))
    ws = dm.workspace(plan.info()["workspace_bytes"])
    L.lrcnn_debug_profile(True)
    try:
        L.lrcnn_forward_rows(plan, dm.x, dm.w, dm.sc, dm.sf, y, ws)
        L.lrcnn_backward_rows(plan, dm.x, dm.w, dm.sc, dm.sf, dy, dm.dw, None, ws)
        torch.cuda.synchronize()
    finally:
        L.lrcnn_debug_profile(False)
    kern = L.lrcnn_debug_profile_collect(roofline=True)
    assert any(k.startswith("wgrad_kernel") for k in kern)
    assert any(k.startswith("conv_gemm_kernel") for k in kern)
    for name, (n, ms, fl, by, rf) in kern.items():
        assert n > 0 and ms > 0 and by > 0 and rf > 0, name
        assert rf <= ms, (name, rf, ms)
