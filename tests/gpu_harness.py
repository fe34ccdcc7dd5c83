"""Helpers for GPU parity tests: run the HIP library through its C ABI and
the CPU oracle on the same seeded inputs, and compare them by the rules of
the parity protocol (max relative error per tensor; ReLU / argmax decisions
equal except at certified near-ties; gradients checked against the oracle
with the GPU's decisions injected)."""
from __future__ import annotations

import numpy as np
import torch

from oracle import bounds as OB, column as OC
from paper_2401_11471_amd import lrcnn as L
from paper_2401_11471_amd.device import DeviceModel

TOL = {L.F32: 1e-4, L.BF16: 2e-2}
# most decisions of a node that may differ from the oracle's (each one must
# also be certified per site by oracle.bounds)
FLIP_CAP = {L.F32: 1e-5, L.BF16: 2e-3}


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
            hybrid_from=0, first_rows=0, plan=None):
    b, h, w, c = inp.x.shape
    if plan is None:
        plan = L.lrcnn_plan(nodes, b, c, h, w, inp.dtype, mode, nb, policy, bounds, bp_refine,
                            hybrid_from, first_rows)
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


def kappa_from_output(y_gpu, y_ref, dtype):
    """Largest deviation of the implementation's output from the oracle's,
    in units of the storage rounding of each value (at least 1): the bound
    the per-site certification assumes for every stored value a site reads
    (the output is the deepest node, where deviations have grown the most).
    Values within 1e-2 of the largest magnitude of zero are skipped."""
    u = OB.unit(dtype == L.BF16)
    yr = np.asarray(y_ref, np.float64)
    big = np.abs(yr) >= 1e-2 * np.abs(yr).max()
    if not big.any():
        return 1
    k = float(np.max(np.abs(np.asarray(y_gpu, np.float64)[big] - yr[big]) / (u * np.abs(yr[big]))))
    return max(1, int(np.ceil(k)))


def check_masks(nodes, inp, ref, masks, dtype, frac_limit, kappa, image=None):
    """Every ReLU / argmax decision that differs from the oracle's must be
    certified by ``oracle.bounds`` (the oracle's value lies within the
    implementation's possible deviation at that site, with stored inputs
    within kappa units of their rounding), and at most frac_limit of a
    node's decisions may differ. `image`: the oracle ran on this image only.
    Returns the number of differing decisions."""
    bf = dtype == L.BF16
    total_bad = 0
    for v, m in masks.items():
        nd = nodes[v]
        op, in0, in1, co, kh, kw, sh, sw, ph, pw, aff, rl = nd
        if image is not None:
            m = m[image:image + 1]
        assert (m != 255).all(), f"node {v}: mask not fully written"
        if op == L.OP_MAXPOOL:
            n, bad = OB.argmax_flips(nd, ref["acts"][in0], ref["argmax"][v], m, kappa, bf)
        else:
            t = ref["pre"][v]
            sites = OB.relu_flips(t, m)
            n = len(sites)
            bad = 0
            if n:
                ts = t[tuple(sites.T)]
                if op == L.OP_CONV:
                    K = kh * kw * ref["acts"][in0].shape[3]
                    S = OB.conv_abs_at(ref["acts"][in0], inp.weights[v - 1], sh, sw, ph, pw,
                                       sites)
                    Et = OB.conv_site_bound(S, K, ts, inp.scales[v - 1], inp.shifts[v - 1],
                                            sites[:, 3], kappa, bf)
                else:
                    za = ref["acts"][in0][tuple(sites.T)]
                    zb = ref["acts"][in1][tuple(sites.T)]
                    Et = OB.add_site_bound(za, zb, ts, kappa, bf)
                bad = int((np.abs(ts) > Et).sum())
        assert bad == 0, f"node {v}: {bad} of {n} differing decisions not certified"
        assert n <= frac_limit * m.size, f"node {v}: {n} differing decisions of {m.size}"
        total_bad += n
    return total_bad


def assert_parity(nodes, inp, gpu, frac_limit=None, check_dx=True):
    dt = inp.dtype
    tol = TOL[dt]
    if frac_limit is None:
        frac_limit = FLIP_CAP[dt]
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
        kappa = kappa_from_output(gpu["y"], ref["acts"][-1], dt)
        nbad = check_masks(nodes, inp, ref, gpu["masks"], dt, frac_limit, kappa)
    return errs, nbad


def assert_parity_per_image(nodes, inp, gpu, frac_limit=None, check_dx=True, say=print):
    """assert_parity with the oracle run one image at a time (the loss is a
    sum over images, so dW is the sum of the images' dW): for workloads
    whose float64 maps do not fit the host several images at once."""
    dt = inp.dtype
    bf = dt == L.BF16
    tol = TOL[dt]
    if frac_limit is None:
        frac_limit = FLIP_CAP[dt]
    B = inp.x.shape[0]
    g = gpu["g"]
    masks = gpu["masks"]
    dws, dx, yref = None, None, None
    nflip = 0
    for b in range(B):
        say(f"oracle image {b + 1} of {B}: forward")
        acts, am, pre = OC.forward(nodes, inp.x[b:b + 1], inp.weights, inp.scales, inp.shifts,
                                   bf16=bf, keep_pre=True)
        y_b = acts[-1]
        if yref is None:
            yref = np.empty((B,) + y_b.shape[1:])
        yref[b] = y_b[0]
        ref = dict(acts=acts, argmax=am, pre=pre)
        kappa = kappa_from_output(gpu["y"][b:b + 1], y_b, dt)
        nflip += check_masks(nodes, inp, ref, masks, dt, frac_limit, kappa, image=b)
        del pre, ref
        inj = {v: (m[b:b + 1] if nodes[v][0] == L.OP_MAXPOOL else (m[b:b + 1] != 0))
               for v, m in masks.items()}
        say(f"oracle image {b + 1} of {B}: backward with the GPU's decisions "
            f"(kappa {kappa})")
        dw_b, dx_b = OC.backward(nodes, acts, am, inp.weights, inp.scales, g[b:b + 1], bf16=bf,
                                 masks=inj, want_dx=check_dx)
        del acts, am, inj
        if dws is None:
            dws = dw_b
        else:
            dws = [None if a is None else a + c for a, c in zip(dws, dw_b)]
        if check_dx:
            if dx is None:
                dx = np.empty(inp.x.shape)
            dx[b] = dx_b[0]
    errs = {"y": rel(gpu["y"], yref)}
    for v in range(1, len(nodes)):
        if dws[v] is not None:
            errs[f"dw{v}"] = rel(gpu["dw"][v], dws[v])
    if check_dx and gpu["dx"] is not None:
        errs["dx"] = rel(gpu["dx"], dx)
    bad = {k: e for k, e in errs.items() if not e <= tol}
    assert not bad, f"max relative errors above {tol}: {bad}"
    return errs, nflip
