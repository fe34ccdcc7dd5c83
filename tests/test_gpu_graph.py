"""A row-centric training step (lrcnn_forward_rows + lrcnn_backward_rows,
including the backward's side stream) captured in a HIP graph: every replay
reproduces the eager step bitwise, with eager work that overwrites the
outputs and the workspace, and synchronisations, between replays."""
import numpy as np
import pytest
import torch

from paper_2401_11471_amd import lrcnn as L
from paper_2401_11471_amd.device import DeviceModel
from workloads import BF16, F32, Inputs, resnet50_net, vgg16_net

pytestmark = pytest.mark.gpu

CASES = [
    ("vgg", F32, L.CARRY, 4, 1),
    ("vgg", F32, L.CARRY, 4, 2),
    ("vgg", BF16, L.CARRY, 3, 1),
    ("vgg", F32, L.RECOMPUTE, 3, 1),
    ("resnet", BF16, L.CARRY, 4, 1),
]


def _snapshot(y, dws, dx):
    return (y.float().cpu().numpy().copy(),
            [None if t is None else t.cpu().numpy().copy() for t in dws],
            dx.float().cpu().numpy().copy())


@pytest.mark.parametrize("net,dtype,mode,nb,refine", CASES)
def test_graph_replay_matches_eager(net, dtype, mode, nb, refine):
    nodes = vgg16_net(with_pool5=True) if net == "vgg" else resnet50_net()
    B, H, W = 2, 64, 96
    print(f"graph case {net} dtype={dtype} mode={mode} bands={nb} refine={refine}", flush=True)
    inp = Inputs(nodes, B, H, W, 3, dtype, seed=11)
    plan = L.lrcnn_plan(nodes, B, 3, H, W, dtype, mode, nb, bp_refine=refine)
    info = plan.info()
    dm = DeviceModel.from_inputs(nodes, inp)
    oshape = (B,) + plan.node_shape(len(nodes) - 1)
    dy = dm.to_device(inp.grad(oshape))
    y = dm.empty(oshape)
    dx = dm.empty(tuple(inp.x.shape))
    ws = dm.workspace(info["workspace_bytes"])

    def step():
        L.lrcnn_forward_rows(plan, dm.x, dm.w, dm.sc, dm.sf, y, ws)
        L.lrcnn_backward_rows(plan, dm.x, dm.w, dm.sc, dm.sf, dy, dm.dw, dx, ws)

    step()
    torch.cuda.synchronize()
    ref = _snapshot(y, dm.dw, dx)

    # warm up on a side stream, then capture
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()

    for rep in range(3):
        # eager work between replays: overwrite everything the step writes
        y.fill_(7.0)
        dx.fill_(-3.0)
        for t in dm.dw:
            if t is not None:
                t.fill_(5.0)
        ws.fill_(0x5A)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = _snapshot(y, dm.dw, dx)
        assert np.array_equal(got[0], ref[0]), f"replay {rep}: y differs"
        for v, (a, b) in enumerate(zip(got[1], ref[1])):
            if b is not None:
                assert np.array_equal(a, b), f"replay {rep}: dW of node {v} differs"
        assert np.array_equal(got[2], ref[2]), f"replay {rep}: dX differs"
    del graph
