"""Helpers for GPU parity tests: run the HIP library through its C ABI and
the CPU oracle on the same seeded inputs, and compare them by the rules of
the parity protocol (max relative error per tensor; ReLU / argmax decisions
equal except at certified near-ties; gradients checked against the oracle
with the GPU's decisions injected)."""
from __future__ import annotations

import numpy as np
import torch

from oracle import column as OC
from paper_2401_11471_amd import lrcnn as L
from paper_2401_11471_amd.device import DeviceModel

TOL = {L.F32: 1e-4, L.BF16: 2e-2}
# a decision may differ only where the oracle's margin is within this
# fraction of the node's largest magnitude
TIE = {L.F32: 1e-5, L.BF16: 3e-2}


def has_mask(nd):
    return (nd[0] in (L.OP_CONV, L.OP_ADD) and nd[11]) or nd[0] == L.OP_MAXPOOL


def hybrid_cuts(nodes):
    """hybrid_from values whose checkpoint (node k - 1) no edge crosses."""
    n = len(nodes)
    return [k for k in range(2, n)
            if all(nodes[v][1] >= k - 1 and (nodes[v][0] != L.OP_ADD or nodes[v][2] >= k - 1)
                   for v in range(k, n))]


def rel(a, b):
    return float(np.max(np.abs(a - b)) / max(float(np.max(np.abs(b))), 1e-30))


def gpu_run(nodes, inp, mode=L.CARRY, nb=1, policy=L.EVEN, bounds=None,
            layerwise=False, want_dx=True, masks=True, repeat_bwd=1, bp_refine=1,
            hybrid_from=0):
    b, h, w, c = inp.x.shape
    plan = L.lrcnn_plan(nodes, b, c, h, w, inp.dtype, mode, nb, policy, bounds, bp_refine,
                        hybrid_from)
    info = plan.info()
    dm = DeviceModel.from_inputs(nodes, inp)
    out_shape = (b,) + plan.node_shape(len(nodes) - 1)
    g = inp.grad(out_shape)
    dy = dm.to_device(g)
    y = dm.empty(out_shape)
    dx = dm.empty(tuple(inp.x.shape)) if want_dx else None
    mk = None
    if masks:
        mk = [None] + [torch.full((b,) + plan.node_shape(v), 255, dtype=torch.uint8,
                                  device="cuda") if has_mask(nd) else None
                       for v, nd in enumerate(nodes[1:], 1)]
    dws_runs = []
    if layerwise:
        ws = dm.workspace(info["layerwise_workspace_bytes"])
        L.lrcnn_layerwise_reference_gpu(plan, dm.x, dm.w, dm.sc, dm.sf, dy, y, dm.dw,
                                        dx, ws, mk)
        torch.cuda.synchronize()
        dws_runs.append([None if t is None else t.cpu().numpy() for t in dm.dw])
    else:
        ws = dm.workspace(info["workspace_bytes"])
        L.lrcnn_forward_rows(plan, dm.x, dm.w, dm.sc, dm.sf, y, ws, mk)
        for _ in range(repeat_bwd):
            L.lrcnn_backward_rows(plan, dm.x, dm.w, dm.sc, dm.sf, dy, dm.dw, dx, ws)
            torch.cuda.synchronize()
            dws_runs.append([None if t is None else t.cpu().numpy() for t in dm.dw])
    out = dict(
        y=y.float().cpu().numpy(),
        dw=dws_runs[-1], dw_runs=dws_runs,
        dx=None if dx is None else dx.float().cpu().numpy(),
        masks=None if mk is None else {v: t.cpu().numpy() for v, t in enumerate(mk)
                                       if t is not None},
        g=g, info=info, plan=plan)
    return out


def oracle_run(nodes, inp, g, masks=None):
    bf = inp.dtype == L.BF16
    acts, am, pre = OC.forward(nodes, inp.x, inp.weights, inp.scales, inp.shifts,
                               bf16=bf, keep_pre=True)
    inj = None
    if masks is not None:
        inj = {}
        for v, m in masks.items():
            inj[v] = m if nodes[v][0] == L.OP_MAXPOOL else (m != 0)
    dws, dx = OC.backward(nodes, acts, am, inp.weights, inp.scales, g, bf16=bf,
                          masks=inj)
    return dict(acts=acts, argmax=am, pre=pre, dw=dws, dx=dx)


def check_masks(nodes, ref, masks, dtype, frac_limit):
    """Every differing ReLU / argmax decision must be a near-tie in the oracle.
    Returns the number of differing decisions."""
    tie = TIE[dtype]
    total_bad = 0
    for v, m in masks.items():
        nd = nodes[v]
        assert (m != 255).all(), f"node {v}: mask not fully written"
        if nd[0] == L.OP_MAXPOOL:
            ref_idx = ref["argmax"][v]
            diff = m != ref_idx
            if diff.any():
                x = ref["acts"][nd[1]]
                scale = np.abs(x).max()
                val = _window_values(x, nd, m)
                best = ref["acts"][v]
                gap = np.abs(best - val)[diff]
                assert (gap <= tie * scale).all(), f"node {v}: argmax differs off a tie"
        else:
            pre = ref["pre"][v]
            diff = (m != 0) != (pre > 0)
            if diff.any():
                scale = np.abs(pre).max()
                assert (np.abs(pre[diff]) <= tie * scale).all(), \
                    f"node {v}: ReLU decision differs off a tie"
        nbad = int(diff.sum())
        assert nbad <= frac_limit * diff.size + 0, f"node {v}: {nbad} differing decisions"
        total_bad += nbad
    return total_bad


def _window_values(x, nd, idx):
    """Oracle input value at window position idx of every pool output."""
    op, in0, in1, co, kh, kw, sh, sw, ph, pw, aff, rl = nd
    b, h, w, c = x.shape
    ho, wo = idx.shape[1:3]
    yy = np.arange(ho)[None, :, None, None] * sh - ph + idx // kw
    xx = np.arange(wo)[None, None, :, None] * sw - pw + idx % kw
    bb = np.arange(b)[:, None, None, None]
    cc = np.arange(c)[None, None, None, :]
    ok = (yy >= 0) & (yy < h) & (xx >= 0) & (xx < w)
    vals = np.where(ok, x[bb, np.clip(yy, 0, h - 1), np.clip(xx, 0, w - 1), cc], -np.inf)
    return vals


def assert_parity(nodes, inp, gpu, frac_limit=None, check_dx=True):
    dt = inp.dtype
    tol = TOL[dt]
    if frac_limit is None:
        frac_limit = 1e-5 if dt == L.F32 else 1e-2
    ref = oracle_run(nodes, inp, gpu["g"], masks=gpu["masks"])
    errs = {"y": rel(gpu["y"], ref["acts"][-1])}
    for v in range(1, len(nodes)):
        if ref["dw"][v] is not None:
            errs[f"dw{v}"] = rel(gpu["dw"][v], ref["dw"][v])
    if check_dx and gpu["dx"] is not None:
        errs["dx"] = rel(gpu["dx"], ref["dx"])
    bad = {k: e for k, e in errs.items() if not e <= tol}
    assert not bad, f"max relative errors above {tol}: {bad}"
    nbad = 0
    if gpu["masks"] is not None:
        nbad = check_masks(nodes, ref, gpu["masks"], dt, frac_limit)
    return errs, nbad
