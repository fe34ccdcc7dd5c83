"""Budget-driven planning on the device (Section III-C, Eqs. (9)-(10)): the
plan lrcnn_plan_for_budget picks for a byte budget M runs with every buffer
of its step requested within M (the bytes requested from torch's
allocator, before its own rounding), the library allocates nothing during
the step, and the step matches the float64 oracle."""
import pytest
import torch

from gpu_harness import assert_parity, gpu_run
from paper_2401_11471_amd import lrcnn as L
from paper_2401_11471_amd.device import DeviceModel
from workloads import Inputs, net_nodes, F32, BF16

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("net,dtype,shape,policy",
                         [("vgg16", F32, (2, 96, 64), L.EVEN),
                          ("resnet50", BF16, (2, 128, 96), L.BALANCED),
                          ("vgg16", BF16, (2, 160, 64), L.PAPER_2PS)])
def test_budget_plan_fits_and_matches_oracle(net, dtype, shape, policy):
    nodes = net_nodes(net)
    B, H, W = shape
    inp = Inputs(nodes, B, H, W, 3, dtype, seed=31)
    one = L.lrcnn_plan(nodes, B, 3, H, W, dtype).step_bytes(False, True)
    # a budget that three bands of the policy meet and one band does not
    M = L.lrcnn_plan(nodes, B, 3, H, W, dtype, L.CARRY, 3, policy).step_bytes(False, True)
    assert M < one
    plan = L.lrcnn_plan_for_budget(nodes, B, 3, H, W, M, dtype, policy=policy, max_bands=32,
                                   max_refine=2, want_dx=True)
    info = plan.info()
    assert plan.step_bytes(False, True) <= M
    print(f"{net} budget {M} of {one}: {info['n_bands']} forward, {info['bp_bands']} "
          f"backward bands, step {plan.step_bytes(False, True)} bytes", flush=True)
    torch.cuda.synchronize()
    torch.cuda.empty_cache()

    def requested():
        return torch.cuda.memory_stats()["requested_bytes.all.current"]
    r0 = requested()
    dm = DeviceModel.from_inputs(nodes, inp)
    oshape = (B,) + plan.node_shape(len(nodes) - 1)
    y, dy, dx = dm.empty(oshape), dm.to_device(inp.grad(oshape)), dm.empty(inp.x.shape)
    ws = dm.workspace(info["workspace_bytes"])
    torch.cuda.synchronize()
    r1 = requested()
    # every buffer of the step, as requested from the allocator (which
    # rounds each request further), fits the budget
    assert r1 - r0 <= M
    torch.cuda.reset_peak_memory_stats()
    L.lrcnn_forward_rows(plan, dm.x, dm.w, dm.sc, dm.sf, y, ws)
    L.lrcnn_backward_rows(plan, dm.x, dm.w, dm.sc, dm.sf, dy, dm.dw, dx, ws)
    torch.cuda.synchronize()
    # the step itself allocates nothing
    assert torch.cuda.memory_stats()["requested_bytes.all.peak"] == r1
    del dm, y, dy, dx, ws
    torch.cuda.empty_cache()
    gpu = gpu_run(nodes, inp, plan=plan)
    assert_parity(nodes, inp, gpu)
