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
# Most decisions of a node that may differ from the oracle's; each one must
# also be certified per site (oracle.bounds). Estimate: stored inputs that
# differ from the oracle's by a relative r move a pre-activation (or a
# window value) of spread sigma by about r sigma, which flips the sites
# within that distance of zero (of the window's runner-up): a fraction of
# about (2 / pi) r for a zero-mean Gaussian-shaped density. In bfloat16 one
# unit of storage rounding is r = 2^-7, about 5e-3; in float32 the stored
# values differ from float64 by accumulation (r of order 1e-5 after a dozen
# layers, from the measured output errors), about 1e-5. The caps are about
# twice (bfloat16) and ten times (float32) these estimates.
FLIP_CAP = {L.F32: 1e-4, L.BF16: 1e-2}


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


def _map_reader(plan, nodes, inp, ws, y):
    """(node, image slice) -> the GPU's stored output map of that node for
    those images (float64 numpy), read from the layer-wise workspace the
    same plan's layer-wise step filled (None for a conv the residual add's
    forward consumes unstored). The two most recent maps are cached."""
    es = 2 if inp.dtype == L.BF16 else 4
    tdt = torch.bfloat16 if inp.dtype == L.BF16 else torch.float32
    b = inp.x.shape[0]
    cache = {}

    def read(v, sl=slice(None)):
        key = (v, sl.start, sl.stop)
        if key in cache:
            return cache[key]
        if v == 0:
            out = np.asarray(inp.x[sl], np.float64)
        elif v == len(nodes) - 1:
            out = y[sl].double().cpu().numpy()
        else:
            off = L.lrcnn_debug_layerwise_map(plan, v)
            if off is None:
                return None
            shape = (b,) + plan.node_shape(v)
            n = int(np.prod(shape))
            out = ws[off:off + n * es].view(tdt).reshape(shape)[sl].double().cpu().numpy()
        if len(cache) >= 2:
            cache.pop(next(iter(cache)))
        cache[key] = out
        return out
    return read


def gpu_run(nodes, inp, mode=L.CARRY, nb=1, policy=L.EVEN, bounds=None,
            layerwise=False, want_dx=True, masks=True, repeat_bwd=1, bp_refine=1,
            hybrid_from=0, first_rows=0, plan=None, twin=True):
    """One training step through the C ABI. Row-centric runs with `twin`
    also run the layer-wise step of the same plan, check that its forward
    output and every decision equal the row-centric ones bit for bit, and
    keep its workspace so that `maps(v)` returns the GPU's stored map of
    any node (for certifying decisions)."""
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

    def new_masks():
        return [None] + [torch.full((b,) + plan.node_shape(v), 255, dtype=torch.uint8,
                                    device="cuda") if has_mask(nd) else None
                         for v, nd in enumerate(nodes[1:], 1)]
    mk = new_masks() if masks else None
    dws_runs = []
    maps = None
    if layerwise:
        ws = dm.workspace(info["layerwise_workspace_bytes"])
        L.lrcnn_layerwise_reference_gpu(plan, dm.x, dm.w, dm.sc, dm.sf, dy, y, dm.dw,
                                        dx, ws, mk)
        torch.cuda.synchronize()
        dws_runs.append([None if t is None else t.cpu().numpy() for t in dm.dw])
        maps = _map_reader(plan, nodes, inp, ws, y)
    else:
        ws = dm.workspace(info["workspace_bytes"])
        L.lrcnn_forward_rows(plan, dm.x, dm.w, dm.sc, dm.sf, y, ws, mk)
        for _ in range(repeat_bwd):
            L.lrcnn_backward_rows(plan, dm.x, dm.w, dm.sc, dm.sf, dy, dm.dw, dx, ws)
            torch.cuda.synchronize()
            dws_runs.append([None if t is None else t.cpu().numpy() for t in dm.dw])
        if twin:
            del ws
            torch.cuda.empty_cache()
            lws = dm.workspace(info["layerwise_workspace_bytes"])
            ly = dm.empty(out_shape)
            lmk = new_masks() if masks else None
            ldw = [None if t is None else torch.empty_like(t) for t in dm.dw]
            L.lrcnn_layerwise_reference_gpu(plan, dm.x, dm.w, dm.sc, dm.sf, dy, ly, ldw,
                                            None, lws, lmk)
            torch.cuda.synchronize()
            assert torch.equal(ly, y), "row-centric forward differs from the layer-wise one"
            if masks:
                for v, (a, q) in enumerate(zip(mk, lmk)):
                    if a is not None:
                        assert torch.equal(a, q), f"node {v}: decisions differ from layer-wise"
            del ldw, lmk
            maps = _map_reader(plan, nodes, inp, lws, ly)
    out = dict(
        y=y.float().cpu().numpy(),
        dw=dws_runs[-1], dw_runs=dws_runs,
        dx=None if dx is None else dx.float().cpu().numpy(),
        masks=None if mk is None else {v: t.cpu().numpy() for v, t in enumerate(mk)
                                       if t is not None},
        g=g, info=info, plan=plan, maps=maps)
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


def check_masks(nodes, inp, ref, masks, dtype, frac_limit, maps, image=None):
    """Every ReLU / argmax decision that differs from the oracle's must be
    the one the GPU's own stored inputs imply up to the GPU's float32
    accumulation error at that site (``oracle.bounds``), every max-pool
    index must be the first maximum of the GPU's own window, and at most
    frac_limit of a node's decisions may differ from the oracle's.
    maps(v, slice): the GPU's stored map of node v; `image`: the oracle ran on
    this image only. Returns the number of differing decisions."""
    bf = dtype == L.BF16
    total = 0
    sl = slice(None) if image is None else slice(image, image + 1)
    for v, m in masks.items():
        nd = nodes[v]
        op, in0, in1, co, kh, kw, sh, sw, ph, pw, aff, rl = nd
        m = m[sl]
        assert (m != 255).all(), f"node {v}: mask not fully written"
        if op == L.OP_MAXPOOL:
            n = int((m != ref["argmax"][v]).sum())
            bad = OB.pool_first_max_violations(nd, maps(in0, sl), m)
            assert bad == 0, f"node {v}: {bad} indices are not the first maximum of the GPU's window"
        else:
            sites = np.argwhere((m != 0) != (ref["pre"][v] > 0))
            n = len(sites)
            if n:
                dec = m[tuple(sites.T)] != 0
                if op == L.OP_CONV:
                    t, E = OB.conv_site(maps(in0, sl), inp.weights[v - 1], inp.scales[v - 1],
                                        inp.shifts[v - 1], nd, sites)
                else:
                    t, E = np.zeros(n), np.zeros(n)
                    for u in (in0, in1):
                        z = maps(u, sl)
                        if z is not None:
                            t += z[tuple(sites.T)]
                            continue
                        # a conv the add consumes unstored: its rounded value
                        du = nodes[u]
                        tc, Ec = OB.conv_site(maps(du[1], sl), inp.weights[u - 1],
                                              inp.scales[u - 1], inp.shifts[u - 1], du, sites)
                        t += tc
                        E += OB.fused_conv_value_bound(tc, Ec, bf)
                    E = E + OB.U32 * (np.abs(t) + E)
                bad = int((~OB.relu_certified(t, E, dec)).sum())
                assert bad == 0, f"node {v}: {bad} of {n} differing decisions not certified"
        assert n <= frac_limit * m.size, f"node {v}: {n} differing decisions of {m.size}"
        total += n
    return total


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
        nbad = check_masks(nodes, inp, ref, gpu["masks"], dt, frac_limit, gpu["maps"])
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
        nflip += check_masks(nodes, inp, ref, masks, dt, frac_limit, gpu["maps"], image=b)
        del pre, ref
        inj = {v: (m[b:b + 1] if nodes[v][0] == L.OP_MAXPOOL else (m[b:b + 1] != 0))
               for v, m in masks.items()}
        say(f"oracle image {b + 1} of {B}: backward with the GPU's decisions")
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
