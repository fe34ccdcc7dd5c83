"""Parity at the five benchmark workloads' full sizes, in the launch
configuration bench.py times (batch, resolution, band count, two-phase
sharing).

* Workloads 1-3: the whole CPU oracle runs on the same inputs; gradients are
  compared with the GPU's ReLU / argmax decisions injected into the oracle
  and every differing decision must be a certified near-tie.
* Workloads 4-5 are too large for a float64 oracle of the whole batch:
  - sampled outputs: the oracle runs on input crops aligned to the network's
    total stride whose interior outputs have their whole receptive cone
    inside the crop, so their values are exact;
  - the row-centric step equals the layer-wise step of the same library
    (partition invariance) to rounding;
  - VGG-16 has no bias, only ReLU and max-pool, so the loss sum(y * G) is
    positively homogeneous of degree 1 in each layer's weights and in the
    input: <W_l, dL/dW_l> = <y, G> for every conv layer (Euler's theorem).
"""
import numpy as np
import pytest
import torch

from gpu_harness import assert_parity, gpu_run, oracle_run, rel, check_masks
from oracle import column as OC, rows as OR
from paper_2401_11471_amd import lrcnn as L
from paper_2401_11471_amd.device import DeviceModel
from workloads import CONFIGS, config_inputs, BF16, F32

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]


def _say(msg):
    print(msg, flush=True)


@pytest.mark.parametrize("cid", [2, 3])
def test_full_oracle_parity(cid):
    c = CONFIGS[cid]
    _say(f"workload {cid} {c['name']}: GPU row-centric step")
    nodes, inp = config_inputs(cid)
    gpu = gpu_run(nodes, inp, L.CARRY, c["bands"], want_dx=False)
    _say(f"workload {cid}: CPU oracle (float64) with the GPU's decisions")
    errs, nbad = assert_parity(nodes, inp, gpu, check_dx=False)
    _say(f"workload {cid}: max rel errors {max(errs.values()):.2e}, "
         f"differing near-tie decisions {nbad}")


def _crop_ref(nodes, inp, b, y0, x0, h, w, bf16):
    """Oracle outputs on an input crop, with a mask of the outputs whose
    receptive cone lies inside the crop (or meets only true image edges)."""
    H, W = inp.x.shape[1:3]
    x = inp.x[b:b + 1, y0:y0 + h, x0:x0 + w]
    acts, _ = OC.forward(nodes, x, inp.weights, inp.scales, inp.shifts, bf16=bf16)
    out = acts[-1][0]
    ok = np.zeros(out.shape[:2], bool)

    def inside(n_in, n_out, off, full):
        shp = OC.shapes(nodes, n_in, n_in, 3)
        res = np.zeros(n_out, bool)
        for o in range(n_out):
            (lo, hi), = OR.cone_intervals(nodes, shp, [o, o + 1])
            top_ok = lo[0] > 0 or off == 0
            bot_ok = hi[0] < n_in or off + n_in == full
            res[o] = top_ok and bot_ok
        return res
    rows_ok = inside(h, out.shape[0], y0, H)
    cols_ok = inside(w, out.shape[1], x0, W) if w != h or x0 != y0 else rows_ok
    ok = rows_ok[:, None] & cols_ok[None, :]
    return out, ok


def _fullsize_gpu(cid, layerwise, dtype=None):
    c = CONFIGS[cid]
    nodes, inp = config_inputs(cid)
    if dtype is not None and dtype != inp.dtype:
        from workloads import Inputs
        B, H, W, C = inp.x.shape
        inp = Inputs(nodes, B, H, W, C, dtype, seed=cid)
    B, H, W, C = inp.x.shape
    plan = L.lrcnn_plan(nodes, B, C, H, W, inp.dtype, L.CARRY, c["bands"])
    info = plan.info()
    dm = DeviceModel.from_inputs(nodes, inp)
    oshape = (B,) + plan.node_shape(len(nodes) - 1)
    g = inp.grad(oshape)
    dy = dm.to_device(g)
    y = dm.empty(oshape)
    ws = dm.workspace(info["workspace_bytes"])
    L.lrcnn_forward_rows(plan, dm.x, dm.w, dm.sc, dm.sf, y, ws)
    L.lrcnn_backward_rows(plan, dm.x, dm.w, dm.sc, dm.sf, dy, dm.dw, None, ws)
    torch.cuda.synchronize()
    res = {"y": y.float(), "dw": [None if t is None else t.clone() for t in dm.dw]}
    del ws
    torch.cuda.empty_cache()
    if layerwise:
        ylw = dm.empty(oshape)
        ws = dm.workspace(info["layerwise_workspace_bytes"])
        L.lrcnn_layerwise_reference_gpu(plan, dm.x, dm.w, dm.sc, dm.sf, dy, ylw, dm.dw,
                                        None, ws)
        torch.cuda.synchronize()
        res["y_lw"] = ylw.float()
        res["dw_lw"] = [None if t is None else t.clone() for t in dm.dw]
        del ws
        torch.cuda.empty_cache()
    return nodes, inp, dm, g, res


@pytest.mark.parametrize("cid", [4, 5])
def test_fullsize_sampled_outputs_and_partition_invariance(cid):
    c = CONFIGS[cid]
    bf16 = c["dtype"] == BF16
    _say(f"workload {cid} {c['name']}: GPU row-centric and layer-wise steps")
    nodes, inp, dm, g, res = _fullsize_gpu(cid, layerwise=True)
    tol = 2e-2 if bf16 else 1e-4
    # partition invariance: row-centric == layer-wise (same kernels). The
    # two group split reductions differently with the launch size, so the
    # forward agrees to rounding and a few ReLU / argmax decisions that sit
    # at a tie flip (about 2e2 of 2.7e9 at workload 4); a flipped decision
    # in a deep layer perturbs the error in its whole receptive cone, so
    # weight gradients are compared in relative Frobenius norm with a bound
    # that allows for those flips.
    # In bfloat16 a 1-ulp difference in a stored activation flips every
    # ReLU decision within that ulp of zero (about 3e-3 of them), so the two
    # schedules' weight gradients differ by ~sqrt(3e-3) in norm from flips
    # alone; the bfloat16 backward is pinned by workload 3 against the oracle
    # (with the GPU's decisions injected) and the banding machinery at this
    # size by the float32 run of the same network below.
    yr, yl = res["y"].cpu().numpy(), res["y_lw"].cpu().numpy()
    assert rel(yr, yl) < (2e-2 if bf16 else 1e-5)
    if not bf16:
        _check_dw_partition(cid, nodes, res)
    # sampled outputs against the oracle on crops
    crop = 448 if c["net"] == "vgg16" else 768
    B, H, W = inp.x.shape[:3]
    checked = 0
    for b, fy, fx in ((0, 0.5, 0.5), (B - 1, 0.0, 1.0), (B // 2, 1.0, 0.25)):
        y0 = int((H - crop) * fy) // 32 * 32
        x0 = int((W - crop) * fx) // 32 * 32
        _say(f"workload {cid}: oracle on crop image {b} rows {y0}+{crop} cols {x0}+{crop}")
        out, ok = _crop_ref(nodes, inp, b, y0, x0, crop, crop, bf16)
        oy, ox = y0 // 32, x0 // 32
        got = yr[b, oy:oy + out.shape[0], ox:ox + out.shape[1]]
        assert ok.sum() >= 4
        ref = out[ok]
        e = np.abs(got[ok] - ref).max() / np.abs(ref).max()
        assert e < tol, e
        checked += ok.sum()
    _say(f"workload {cid}: {checked} sampled output positions match")


def _check_dw_partition(cid, nodes, res):
    worst = 0.0
    for v in range(1, len(nodes)):
        if res["dw"][v] is not None:
            a, b = res["dw"][v].double(), res["dw_lw"][v].double()
            e = float((a - b).norm() / b.norm())
            worst = max(worst, e)
            assert e < 2e-2, (v, e)
    _say(f"workload {cid}: row-centric vs layer-wise dW, worst relative norm {worst:.2e}")


def test_resnet_fullsize_partition_invariance_float32():
    # workload 5's network, batch, resolution and 32 bands, stored in float32
    _say("workload 5 shapes in float32: GPU row-centric and layer-wise steps")
    nodes, inp, dm, g, res = _fullsize_gpu(5, layerwise=True, dtype=F32)
    assert rel(res["y"].cpu().numpy(), res["y_lw"].cpu().numpy()) < 1e-4
    _check_dw_partition(5, nodes, res)


@pytest.mark.parametrize("cid", [2, 4])
def test_vgg_euler_identity_at_full_size(cid):
    # homogeneity of degree 1: <W_l, dW_l> = <y, G> for every conv layer,
    # for the row-centric step and for the layer-wise step
    _say(f"workload {cid}: Euler identity of every VGG-16 conv layer")
    nodes, inp, dm, g, res = _fullsize_gpu(cid, layerwise=True)
    gd = torch.from_numpy(g).double().to(res["y"].device)
    for yk, dk in (("y", "dw"), ("y_lw", "dw_lw")):
        lhs = float((res[yk].double() * gd).sum())
        for v in range(1, len(nodes)):
            if res[dk][v] is None:
                continue
            rhs = float((dm.w[v].double() * res[dk][v].double()).sum())
            assert abs(rhs - lhs) <= 1e-4 * abs(lhs), (dk, v, rhs, lhs)
