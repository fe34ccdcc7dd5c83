"""Parity at the five benchmark workloads' full sizes, in the launch
configuration bench.py times (resolution, band count, two-phase sharing).

* Every workload's row-centric step is compared with the float64 oracle:
  the output, every weight gradient and the input gradient, with the GPU's
  ReLU / argmax decisions injected into the oracle's backward, and every
  decision that differs from the oracle's certified per site
  (``oracle.bounds``). Workloads 4 and 5 run the oracle one image at a time
  (the loss is a sum over images, so dW is the sum of the images' dW);
  workload 5 runs at batch 2 instead of 8 so that the float64 oracle of its
  2400 x 3600 images finishes within the test's time limit.
* The row-centric forward equals the layer-wise step's bit for bit at
  workloads 4 and 5 (every forward launch of a layer sums the same K
  chunks).
* VGG-16 has no bias, only ReLU and max-pool, so the loss sum(y * G) is
  positively homogeneous of degree 1 in each layer's weights:
  <W_l, dL/dW_l> = <y, G> for every conv layer (Euler's theorem).
"""
import numpy as np
import pytest
import torch

from gpu_harness import assert_parity, assert_parity_per_image, gpu_run, rel
from paper_2401_11471_amd import lrcnn as L
from paper_2401_11471_amd.device import DeviceModel
from workloads import CONFIGS, config_inputs, BF16

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]


def _say(msg):
    print(msg, flush=True)


@pytest.mark.parametrize("cid", [2, 3])
def test_full_oracle_parity(cid):
    c = CONFIGS[cid]
    _say(f"workload {cid} {c['name']}: GPU row-centric step")
    nodes, inp = config_inputs(cid)
    gpu = gpu_run(nodes, inp, L.CARRY, c["bands"], want_dx=True)
    _say(f"workload {cid}: CPU oracle (float64) with the GPU's decisions")
    errs, nflip = assert_parity(nodes, inp, gpu)
    _say(f"workload {cid}: max rel errors {max(errs.values()):.2e} "
         f"(dx {errs['dx']:.2e}), differing certified decisions {nflip}")


@pytest.mark.parametrize("cid,batch", [(4, None), (5, 2)])
def test_fullsize_gradients_match_oracle(cid, batch):
    c = CONFIGS[cid]
    nodes, inp = config_inputs(cid, batch=batch)
    B = inp.x.shape[0]
    _say(f"workload {cid} {c['name']} at batch {B}: GPU row-centric step, "
         f"{c['bands']} bands, decisions exported")
    gpu = gpu_run(nodes, inp, L.CARRY, c["bands"], want_dx=True)
    torch.cuda.empty_cache()
    errs, nflip = assert_parity_per_image(nodes, inp, gpu, say=_say)
    _say(f"workload {cid}: max rel errors y {errs['y']:.2e}, dx {errs['dx']:.2e}, dW "
         f"{max(e for k, e in errs.items() if k.startswith('dw')):.2e}; "
         f"differing certified decisions {nflip}")


def _fullsize_gpu(cid, layerwise):
    c = CONFIGS[cid]
    nodes, inp = config_inputs(cid)
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
def test_fullsize_forward_bitwise_equals_layerwise(cid):
    c = CONFIGS[cid]
    _say(f"workload {cid} {c['name']}: GPU row-centric and layer-wise steps")
    nodes, inp, dm, g, res = _fullsize_gpu(cid, layerwise=True)
    assert torch.equal(res["y"], res["y_lw"])
    gtol = 2e-2 if c["dtype"] == BF16 else 1e-4
    worst = 0.0
    for v in range(1, len(nodes)):
        if res["dw"][v] is not None:
            e = rel(res["dw"][v].cpu().numpy(), res["dw_lw"][v].cpu().numpy())
            worst = max(worst, e)
            assert e < gtol, (v, e)
    _say(f"workload {cid}: forward bitwise equal; dW worst max rel difference {worst:.2e}")


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
