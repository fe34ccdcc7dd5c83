"""The allocation-free forward entry point, lrcnn_forward_rows_static,
against lrcnn_forward_rows on the same plan and inputs: output and ReLU /
argmax decisions equal bit for bit (the same kernels run on the same
plan), on two calls in a row, the second on a smaller input (the static
workspace then holds the first call's data); torch allocates nothing
during the call (its cumulative allocation count is unchanged); a plan whose workspace exceeds the static array is
refused before any device work."""
import pytest
import torch

from paper_2401_11471_amd import lrcnn as L
from workloads import NetBuilder, Inputs, F32, BF16


def _net():
    nb = NetBuilder()
    a = nb.conv(0, 16, 7, 2, 3, affine=1)
    b = nb.pool(a, 3, 2, 1)
    c1 = nb.conv(b, 24, 3, 1, 1, affine=1)
    c2 = nb.conv(c1, 64, 1, 1, 0, affine=1, relu=0)
    sc = nb.conv(b, 64, 1, 1, 0, affine=1, relu=0)
    s = nb.sum(c2, sc)
    d = nb.conv(s, 40, 3, 1, 1)
    nb.pool(d, 2, 2, 0)
    return nb.nodes


def _has_mask(nd):
    return (nd[0] in (L.OP_CONV, L.OP_ADD) and nd[11]) or nd[0] == L.OP_MAXPOOL


def test_static_forward_refuses_large_plans():
    # VGG-style 3x3 stack at 512 x 512, batch 4: far more than 64 MiB of
    # workspace; refused from the plan alone (no pointer is touched)
    nb = NetBuilder()
    v = 0
    for c in (64, 64, 128, 128):
        v = nb.conv(v, c, 3, 1, 1)
    plan = L.lrcnn_plan(nb.nodes, 4, 3, 512, 512, L.F32, L.CARRY, 2)
    assert plan.info()["workspace_bytes"] > L.STATIC_WORKSPACE_BYTES
    code = L.LIB.lrcnn_forward_rows_static(plan.handle, None, None, None, None, None,
                                           None, None)
    assert code == -4, code
    assert "static workspace" in L.LIB.lrcnn_last_error().decode()
    assert L.LIB.lrcnn_forward_rows_static(None, None, None, None, None, None, None,
                                           None) == -1


@pytest.mark.gpu
@pytest.mark.parametrize("dtype", [F32, BF16])
def test_static_forward_equals_forward_rows(dtype):
    from paper_2401_11471_amd.device import DeviceModel
    nodes = _net()
    n = len(nodes)
    # (batch, H, W, mode, bands); the second call is the smaller one
    cases = [(2, 83, 61, L.CARRY, 4), (1, 37, 29, L.RECOMPUTE, 3)]
    for i, (B, H, W, mode, nbands) in enumerate(cases):
        print(f"static forward: dtype={dtype} call {i} B={B} {H}x{W} mode={mode} "
              f"bands={nbands}", flush=True)
        inp = Inputs(nodes, B, H, W, 3, dtype, seed=31 + i)
        plan = L.lrcnn_plan(nodes, B, 3, H, W, dtype, mode, nbands)
        info = plan.info()
        assert 0 < info["workspace_bytes"] <= L.STATIC_WORKSPACE_BYTES
        dm = DeviceModel.from_inputs(nodes, inp)
        oshape = (B,) + plan.node_shape(n - 1)

        def masks():
            return [dm.empty((B,) + plan.node_shape(v), torch.uint8)
                    if v and _has_mask(nodes[v]) else None for v in range(n)]
        y_ref, m_ref = dm.empty(oshape), masks()
        ws = dm.workspace(info["workspace_bytes"])
        L.lrcnn_forward_rows(plan, dm.x, dm.w, dm.sc, dm.sf, y_ref, ws, m_ref)
        y, m = dm.empty(oshape), masks()
        torch.cuda.synchronize()
        # cumulative count of torch's device allocations (frees by Python's
        # garbage collector during the call do not change it)
        before = torch.cuda.memory_stats()["allocation.all.allocated"]
        L.lrcnn_forward_rows_static(plan, dm.x, dm.w, dm.sc, dm.sf, y, m)
        torch.cuda.synchronize()
        assert torch.cuda.memory_stats()["allocation.all.allocated"] == before
        assert torch.equal(y, y_ref)
        for v in range(n):
            if m[v] is not None:
                assert torch.equal(m[v], m_ref[v]), v
        if mode == L.CARRY:
            # the static forward's shared rows are not in the caller's workspace
            dy = dm.empty(oshape)
            with pytest.raises(L.LrcnnError) as e:
                L.lrcnn_backward_rows(plan, dm.x, dm.w, dm.sc, dm.sf, dy, dm.dw, None, ws)
            assert e.value.code == -5
        torch.cuda.synchronize()
