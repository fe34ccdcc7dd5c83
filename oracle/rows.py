"""Row-centric training on the CPU (Algorithm 1), with both ways the paper
handles the weak dependency between consecutive rows.

TEST INFRASTRUCTURE (see ``oracle/column.py``).

* CARRY = two-phase sharing, 2PS (Section IV-A): rows of a feature map that a
  later row band still needs are cached when band r computes them and reused
  by band r+1, both in FP and in BP. Bands are ranges of input rows
  (Algorithm 1 splits the input chi into chi_1..chi_N).
* RECOMPUTE = overlapping partitioning, OverL (Section IV-B): the last
  layer is split evenly (the paper's balancing advice) and every band
  recomputes its whole receptive cone, so bands share nothing. Instead of the
  paper's "record redundant times and average" step, each band
  back-propagates only its own slice of the upstream gradient and the
  partial gradients add up exactly (linearity).
* Semi-closed padding (Section III-B): zero (or -inf for pooling) padding
  is applied only at the true image top and bottom; rows at an internal band
  edge always come from real data.

This module carries its own interval arithmetic, written independently of
the HIP library's planner; the two are compared by the tests.
"""
from __future__ import annotations

import numpy as np

from . import column as C
from .bf16 import round_bf16

OP_INPUT, OP_CONV, OP_MAXPOOL, OP_ADD = C.OP_INPUT, C.OP_CONV, C.OP_MAXPOOL, C.OP_ADD


def _ksp(node):
    op, in0, in1, co, kh, kw, sh, sw, ph, pw, aff, rl = node
    if op == OP_ADD:
        return 1, 1, 0
    return kh, sh, ph


def consumers(nodes):
    cons = [[] for _ in nodes]
    for v, nd in enumerate(nodes):
        if v == 0:
            continue
        cons[nd[1]].append(v)
        if nd[0] == OP_ADD:
            cons[nd[2]].append(v)
    return cons


# ---------------------------------------------------------------- intervals
def frontier_step(f_in, h_in, h_out, k, s, p):
    """Rows of an op's output computable from input rows [0, f_in): output
    row y needs input rows [y*s-p, y*s-p+k) clipped to the image."""
    if f_in >= h_in:
        return h_out
    y_last = (f_in + p - k) // s  # last y with y*s-p+k <= f_in
    return max(0, min(h_out, y_last + 1))


def carry_intervals(nodes, shp, bounds):
    """F[r][v]: rows of node v finished after bands 1..r; T[r][v]: first row of
    v that a band after r may still read (the cached shared rows are
    [T[r][v], F[r][v]))."""
    n, nb = len(nodes), len(bounds) - 1
    cons = consumers(nodes)
    F = [[0] * n for _ in range(nb + 1)]
    T = [[0] * n for _ in range(nb + 1)]
    for r in range(1, nb + 1):
        F[r][0] = bounds[r]
        for v in range(1, n):
            nd = nodes[v]
            if nd[0] == OP_ADD:
                F[r][v] = min(F[r][nd[1]], F[r][nd[2]])
            else:
                k, s, p = _ksp(nd)
                F[r][v] = frontier_step(F[r][nd[1]], shp[nd[1]][0], shp[v][0],
                                        k, s, p)
    for r in range(1, nb + 1):
        for v in range(n):
            t = F[r][v]
            for c in cons[v]:
                k, s, p = _ksp(nodes[c])
                t = min(t, F[r][c] * s - p)
            T[r][v] = max(0, min(t, F[r][v]))
    return F, T


def cone_intervals(nodes, shp, out_bounds):
    """Per band, the receptive cone [lo, hi) of every node needed to produce
    the band's own output rows (Eq. (15) read as an interval recursion)."""
    n = len(nodes)
    cons = consumers(nodes)
    res = []
    for r in range(1, len(out_bounds)):
        lo = [0] * n
        hi = [0] * n
        lo[n - 1], hi[n - 1] = out_bounds[r - 1], out_bounds[r]
        for v in range(n - 2, -1, -1):
            a, b = None, None
            for c in cons[v]:
                if hi[c] <= lo[c]:
                    continue
                k, s, p = _ksp(nodes[c])
                ca = max(0, lo[c] * s - p)
                cb = min(shp[v][0], (hi[c] - 1) * s - p + k)
                a = ca if a is None else min(a, ca)
                b = cb if b is None else max(b, cb)
            if a is None or b <= a:
                lo[v] = hi[v] = 0
            else:
                lo[v], hi[v] = a, b
        res.append((lo, hi))
    return res


def even_bounds(h, nb):
    return [(r * h) // nb for r in range(nb + 1)]


# ------------------------------------------------------------ band kernels
class Window:
    """Rows [lo, lo + len(a)) of one node's feature map (all images)."""

    def __init__(self, lo, a):
        self.lo, self.a = lo, a

    @property
    def hi(self):
        return self.lo + self.a.shape[1]

    def rows(self, a, b, h, fill):
        """Rows [a, b) with semi-closed padding: rows outside [0, h) are
        ``fill``; every row inside the image must be held by the window."""
        bsz, _, w, c = self.a.shape
        out = np.full((bsz, max(0, b - a), w, c), fill, dtype=np.float64)
        for y in range(a, b):
            if 0 <= y < h:
                assert self.lo <= y < self.hi, (y, self.lo, self.hi)
                out[:, y - a] = self.a[:, y - self.lo]
        return out


def band_node_fwd(nodes, v, wins, shp, y0, y1, prm, bf16):
    """Rows [y0, y1) of node v from its inputs' windows. Returns (rows,
    argmax rows or None)."""
    nd = nodes[v]
    op, in0, in1, co, kh, kw, sh, sw, ph, pw, aff, rl = nd
    bsz = wins[in0].a.shape[0]
    if y1 <= y0:
        h, w, c = shp[v]
        return (np.zeros((bsz, 0, w, c)),
                np.zeros((bsz, 0, w, c), np.uint8) if op == OP_MAXPOOL else None)
    if op == OP_ADD:
        a = wins[in0].rows(y0, y1, shp[in0][0], 0.0)
        b = wins[in1].rows(y0, y1, shp[in1][0], 0.0)
        return C.apply_node(nd, [a, b], None, None, None, bf16)
    fill = -np.inf if op == OP_MAXPOOL else 0.0
    slab = wins[in0].rows(y0 * sh - ph, (y1 - 1) * sh - ph + kh,
                          shp[in0][0], fill)
    # rows are already padded; only the columns keep their padding
    nd_rows = (op, in0, in1, co, kh, kw, sh, sw, 0, pw, aff, rl)
    w, sc, sf = prm(v)
    return C.apply_node(nd_rows, [slab], w, sc, sf, bf16)


def band_node_bwd(nodes, v, wins, dwins, shp, y0, y1, d, z, idx, prm, bf16,
                  want_dx, dws):
    """Back-propagate the finished error rows [y0, y1) of node v into its
    inputs' error windows and add its weight gradient (Algorithm 1,
    Get_error and g^l += Gradient)."""
    if y1 <= y0:
        return
    nd = nodes[v]
    op, in0, in1, co, kh, kw, sh, sw, ph, pw, aff, rl = nd
    w, sc, sf = prm(v)
    if op == OP_ADD:
        if rl:
            d = d * (z > 0)
        for u in (in0, in1):
            _add_rows(dwins[u], y0, d, shp[u][0])
        return
    a = y0 * sh - ph
    b = (y1 - 1) * sh - ph + kh
    if op == OP_CONV:
        slab = wins[in0].rows(a, b, shp[in0][0], 0.0)
        dc = C.error_operand(nd, d, z, sc, bf16)
        dws[v] = dws[v] + C.conv_wgrad(dc, slab, kh, kw, sh, sw, 0, pw)
        if in0 == 0 and not want_dx:
            return
        ds = C.conv_dgrad(dc, w, slab.shape[1:3], sh, sw, 0, pw)
    else:
        ds = C.maxpool_bwd(d, idx, (b - a, shp[in0][1]), kh, kw, sh, sw, 0, pw)
    _add_rows(dwins[in0], a, ds, shp[in0][0])


def _add_rows(win, a, rows, h):
    for t in range(rows.shape[1]):
        y = a + t
        if 0 <= y < h:
            assert win.lo <= y < win.hi, (y, win.lo, win.hi)
            win.a[:, y - win.lo] += rows[:, t]


class _Params:
    def __init__(self, ws, scs, shs):
        self.ws, self.scs, self.shs = ws, scs, shs

    def __call__(self, v):
        return self.ws[v - 1], self.scs[v - 1], self.shs[v - 1]


# --------------------------------------------------------------- CARRY (2PS)
def carry_forward(nodes, x, ws, scs, shs, bounds, bf16=False):
    """Row-centric FP with shared rows cached across bands (Algorithm 1 FP
    loop + Section IV-A). Returns (y, strips) where strips[(r, v)] holds the
    rows [T[r][v], F[r][v]) kept for the next band and for BP."""
    x = np.asarray(x, np.float64)
    bsz, h, w, c = x.shape
    shp = C.shapes(nodes, h, w, c)
    F, T = carry_intervals(nodes, shp, bounds)
    prm = _Params(ws, scs, shs)
    n, nb = len(nodes), len(bounds) - 1
    last = n - 1
    y = np.zeros((bsz,) + shp[last], dtype=np.float64)
    strips = {(0, v): np.zeros((bsz, 0) + shp[v][1:]) for v in range(n)}
    for r in range(1, nb + 1):
        wins = _band_recompute(nodes, x, shp, F, T, strips, r, prm, bf16)[0]
        for v in range(n):
            win = wins[v]
            strips[(r, v)] = win.a[:, T[r][v] - win.lo:F[r][v] - win.lo].copy()
        y[:, F[r - 1][last]:F[r][last]] = \
            wins[last].a[:, F[r - 1][last] - wins[last].lo:]
    return y, strips


def _band_recompute(nodes, x, shp, F, T, strips, r, prm, bf16):
    n = len(nodes)
    wins = [None] * n
    argm = [None] * n
    wins[0] = Window(T[r - 1][0], x[:, T[r - 1][0]:F[r][0]])
    for v in range(1, n):
        rows, idx = band_node_fwd(nodes, v, wins, shp, F[r - 1][v], F[r][v],
                                  prm, bf16)
        head = strips[(r - 1, v)]
        wins[v] = Window(T[r - 1][v], np.concatenate([head, rows], axis=1))
        argm[v] = idx
    return wins, argm


def carry_backward(nodes, x, ws, scs, shs, g, bounds, strips, bf16=False,
                   want_dx=True):
    """Row-centric BP (Algorithm 1 BP loop): bands in reverse order, each
    first recomputing its rows from the cached shared rows, then propagating
    errors; the error that band r sends to rows owned by earlier bands is
    carried to them. Returns (dW per node, dX)."""
    x = np.asarray(x, np.float64)
    g = np.asarray(g, np.float64)
    bsz, h, w, c = x.shape
    shp = C.shapes(nodes, h, w, c)
    F, T = carry_intervals(nodes, shp, bounds)
    prm = _Params(ws, scs, shs)
    n, nb = len(nodes), len(bounds) - 1
    last = n - 1
    dws = [np.zeros(np.shape(ws[v - 1])) if nodes[v][0] == OP_CONV else None
           for v in range(n)]
    dx = np.zeros_like(x)
    carry = [np.zeros((bsz, 0) + shp[v][1:]) for v in range(n)]
    for r in range(nb, 0, -1):
        wins, argm = _band_recompute(nodes, x, shp, F, T, strips, r, prm, bf16)
        dwins = []
        for v in range(n):
            lo, hi = T[r - 1][v], F[r][v]
            a = np.zeros((bsz, hi - lo) + shp[v][1:])
            cr = carry[v]
            a[:, T[r][v] - lo:T[r][v] - lo + cr.shape[1]] += cr
            dwins.append(Window(lo, a))
        dwins[last].a[:, F[r - 1][last] - dwins[last].lo:] += \
            g[:, F[r - 1][last]:F[r][last]]
        for v in range(n - 1, 0, -1):
            y0, y1 = F[r - 1][v], F[r][v]
            lo = dwins[v].lo
            d = dwins[v].a[:, y0 - lo:y1 - lo]
            z = wins[v].a[:, y0 - wins[v].lo:y1 - wins[v].lo]
            band_node_bwd(nodes, v, wins, dwins, shp, y0, y1, d, z, argm[v],
                          prm, bf16, want_dx, dws)
            carry[v] = dwins[v].a[:, T[r - 1][v] - lo:F[r - 1][v] - lo].copy()
        lo = dwins[0].lo
        dx[:, F[r - 1][0]:F[r][0]] = dwins[0].a[:, F[r - 1][0] - lo:]
        carry[0] = dwins[0].a[:, T[r - 1][0] - lo:F[r - 1][0] - lo].copy()
    return dws, dx


# ----------------------------------------------------------- RECOMPUTE (OverL)
def _cone_band(nodes, x, shp, lo, hi, prm, bf16):
    n = len(nodes)
    wins = [None] * n
    argm = [None] * n
    wins[0] = Window(lo[0], x[:, lo[0]:hi[0]])
    for v in range(1, n):
        rows, idx = band_node_fwd(nodes, v, wins, shp, lo[v], hi[v], prm, bf16)
        wins[v] = Window(lo[v], rows)
        argm[v] = idx
    return wins, argm


def recompute_forward(nodes, x, ws, scs, shs, out_bounds, bf16=False):
    """OverL FP: each band computes its whole cone independently and writes
    only its own output rows."""
    x = np.asarray(x, np.float64)
    bsz, h, w, c = x.shape
    shp = C.shapes(nodes, h, w, c)
    prm = _Params(ws, scs, shs)
    last = len(nodes) - 1
    y = np.zeros((bsz,) + shp[last])
    for lo, hi in cone_intervals(nodes, shp, out_bounds):
        wins, _ = _cone_band(nodes, x, shp, lo, hi, prm, bf16)
        y[:, lo[last]:hi[last]] = wins[last].a
    return y


def recompute_backward(nodes, x, ws, scs, shs, g, out_bounds, bf16=False,
                       want_dx=True):
    """OverL BP: per band, recompute the cone, seed the error with the band's
    own rows of G only, back-propagate through the cone and add the partial
    weight and input gradients."""
    x = np.asarray(x, np.float64)
    g = np.asarray(g, np.float64)
    bsz, h, w, c = x.shape
    shp = C.shapes(nodes, h, w, c)
    prm = _Params(ws, scs, shs)
    n = len(nodes)
    last = n - 1
    dws = [np.zeros(np.shape(ws[v - 1])) if nodes[v][0] == OP_CONV else None
           for v in range(n)]
    dx = np.zeros_like(x)
    for lo, hi in cone_intervals(nodes, shp, out_bounds):
        wins, argm = _cone_band(nodes, x, shp, lo, hi, prm, bf16)
        dwins = [Window(lo[v], np.zeros((bsz, hi[v] - lo[v]) + shp[v][1:]))
                 for v in range(n)]
        dwins[last].a += g[:, lo[last]:hi[last]]
        for v in range(n - 1, 0, -1):
            band_node_bwd(nodes, v, wins, dwins, shp, lo[v], hi[v],
                          dwins[v].a, wins[v].a, argm[v], prm, bf16, want_dx,
                          dws)
        dx[:, lo[0]:hi[0]] += dwins[0].a
    return dws, dx


# ------------------------------------------------- no dependency handling
def independent_bands_forward(nodes, x, ws, scs, shs, bounds, bf16=False):
    """Each input band run through the network as if it were a whole image:
    no shared rows and zero padding at every band edge. This is the broken
    baseline of Section III-B (feature loss, padding redundancy); outputs are
    concatenated along the height."""
    outs = []
    for r in range(1, len(bounds)):
        xb = np.asarray(x, np.float64)[:, bounds[r - 1]:bounds[r]]
        acts, _ = C.forward(nodes, xb, ws, scs, shs, bf16)
        outs.append(acts[-1])
    return np.concatenate(outs, axis=1)
