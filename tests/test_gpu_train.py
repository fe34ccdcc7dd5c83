"""Full training step on the GPU (Algorithm 1: head, loss and update around
the row-centric FP and BP) against the float64 oracle of column training.

* the head alone: logits, loss, dL/dy and head gradients against the oracle
  on the trunk output the GPU produced;
* a few SGD steps: the loss before every update and the final parameters
  against the oracle's own training loop from the same initial values;
* row-centric against layer-wise training on the GPU: the loss curves agree
  to rounding (the paper's convergence claim, without a dataset).
"""
import numpy as np
import pytest
import torch

from oracle import head as OH
from paper_2401_11471_amd import lrcnn as L
from paper_2401_11471_amd.device import DeviceModel
from paper_2401_11471_amd.train import Trainer
from test_gpu_parity import NETS, _inputs
from workloads import F32, BF16

pytestmark = pytest.mark.gpu


def rel(a, r):
    a = np.asarray(a, np.float64)
    r = np.asarray(r, np.float64)
    return float(np.abs(a - r).max() / max(np.abs(r).max(), 1e-30))


def _head_params(plan, n_classes, seed):
    oh, ow, oc = plan.node_shape(plan.n - 1)
    g = np.random.default_rng(seed)
    fw = (g.standard_normal((n_classes, oh * ow * oc)) / np.sqrt(oh * ow * oc)).astype(np.float32)
    fb = (g.standard_normal(n_classes) * 0.1).astype(np.float32)
    return fw, fb


@pytest.mark.parametrize("dtype", [F32, BF16])
@pytest.mark.parametrize("name", ["vgg_like", "resnet_like"])
def test_head_matches_oracle(name, dtype):
    nodes, inp = _inputs(name, dtype, batch=3, seed=31)
    b, h, w, c = inp.x.shape
    plan = L.lrcnn_plan(nodes, b, c, h, w, dtype, L.CARRY, 3)
    dm = DeviceModel.from_inputs(nodes, inp)
    fw, fb = _head_params(plan, 10, 5)
    labels = np.array([1, 7, 4])
    tr = Trainer(plan, dm, fw, fb, labels)
    L.lrcnn_forward_rows(plan, dm.x, dm.w, dm.sc, dm.sf, tr.y, tr.ws)
    L.lrcnn_head_loss(plan, tr.y, tr.fc_w, tr.fc_b, tr.labels, tr.logits, tr.loss, tr.dy,
                      tr.d_fc_w, tr.d_fc_b, tr.head_ws)
    torch.cuda.synchronize()
    y = tr.y.float().cpu().numpy()
    logits = OH.head_forward(y, fw, fb)
    loss, dlog = OH.softmax_xent(logits, labels)
    dy, dfw, dfb = OH.head_backward(y, fw, dlog)
    tol = 1e-5
    assert rel(tr.logits.cpu().numpy(), logits) < tol
    assert abs(tr.loss[0].item() - loss) <= tol * abs(loss)
    assert rel(tr.d_fc_w.cpu().numpy(), dfw) < tol
    assert rel(tr.d_fc_b.cpu().numpy(), dfb) < tol
    # dL/dy is stored in the plan's dtype
    assert rel(tr.dy.float().cpu().numpy(), dy) < (tol if dtype == F32 else 1e-2)


def test_invalid_label_gives_nan_loss():
    nodes, inp = _inputs("tiny", F32, batch=2, seed=3)
    b, h, w, c = inp.x.shape
    plan = L.lrcnn_plan(nodes, b, c, h, w, F32, L.CARRY, 2)
    dm = DeviceModel.from_inputs(nodes, inp)
    fw, fb = _head_params(plan, 4, 2)
    tr = Trainer(plan, dm, fw, fb, np.array([1, 9]))
    tr.step(0.0)
    torch.cuda.synchronize()
    assert np.isnan(tr.loss[0].item())


@pytest.mark.parametrize("mode,nb", [(L.CARRY, 4), (L.RECOMPUTE, 3)])
@pytest.mark.parametrize("name", ["tiny", "vgg_like", "resnet_like"])
def test_training_steps_match_oracle(name, mode, nb):
    nodes, inp = _inputs(name, F32, batch=2, seed=41)
    b, h, w, c = inp.x.shape
    plan = L.lrcnn_plan(nodes, b, c, h, w, F32, mode, nb)
    dm = DeviceModel.from_inputs(nodes, inp)
    fw, fb = _head_params(plan, 10, 9)
    labels = np.array([2, 5])
    lr, steps = 1e-4, 4
    tr = Trainer(plan, dm, fw, fb, labels)
    losses = []
    for _ in range(steps):
        losses.append(tr.step(lr).item())
    torch.cuda.synchronize()
    ref, wref, fwref, fbref = OH.train(nodes, inp.x, inp.weights, inp.scales, inp.shifts,
                                       fw, fb, labels, lr, steps)
    print(name, "losses", losses, "oracle", ref)
    np.testing.assert_allclose(losses, ref, rtol=2e-5, atol=0)
    assert ref[-1] < ref[0]
    for v in range(1, len(nodes)):
        if wref[v - 1] is not None:
            assert rel(dm.w[v].cpu().numpy(), wref[v - 1]) < 1e-5
    assert rel(tr.fc_w.cpu().numpy(), fwref) < 1e-5
    assert rel(tr.fc_b.cpu().numpy(), fbref) < 1e-5


@pytest.mark.parametrize("dtype", [F32, BF16])
def test_row_centric_and_layerwise_training_agree(dtype):
    nodes, inp = _inputs("vgg_like", dtype, batch=4, seed=51)
    b, h, w, c = inp.x.shape
    curves = {}
    for lw in (False, True):
        plan = L.lrcnn_plan(nodes, b, c, h, w, dtype, L.CARRY, 4)
        dm = DeviceModel.from_inputs(nodes, inp)
        fw, fb = _head_params(plan, 10, 13)
        tr = Trainer(plan, dm, fw, fb, np.array([0, 3, 3, 9]), layerwise=lw)
        curves[lw] = [tr.step(1e-4).item() for _ in range(8)]
    torch.cuda.synchronize()
    print("row-centric", curves[False], "layer-wise", curves[True])
    tol = 1e-4 if dtype == F32 else 2e-2
    np.testing.assert_allclose(curves[False], curves[True], rtol=tol)
    assert curves[False][-1] < curves[False][0]
