"""Column (layer-by-layer) CNN training in float64: the plain definition that
row-centric training must reproduce exactly.

TEST INFRASTRUCTURE. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package. It shares no
code with the HIP library and never calls it.

The paper states that row-centric training reorders the computation without
changing the result (Abstract; Section I, contributions; Section III-A,
"An Example"), so the oracle is simply ordinary training:

* forward, Eq. (1): z^l = Conv(z^{l-1}, theta_l), with ReLU, a fixed
  per-channel affine in place of BatchNorm, max-pooling and residual adds
  (Section II-A);
* backward, Eq. (2): g^l = Gradient(delta^l, z^{l-1}), the error delta
  propagating from the last layer to the first (Algorithm 1, BP loop);
* loss L = sum(y * G), so dL/dy = G.

Numerics: float64 everywhere. With ``bf16=True`` the storage of a bfloat16
run is emulated by rounding (round-to-nearest-even) at exactly two kinds of
points: every stored node output, and the error operand that enters a
convolution's input- and weight-gradient (delta times ReLU mask times affine
scale). Everything else stays wide.

Readings where the paper is silent or garbled (each listed in the design
notes): output size floor((H+2p-k)/s)+1 (Section III-B prints a garbled
form); zero padding only at true image edges (semi-closed padding,
Section III-B); max-pool ties go to the first maximum in row-major window
order and -inf padding is never chosen; ReLU'(0) = 0; convolutions carry no
bias.
"""
from __future__ import annotations

import numpy as np

from .bf16 import round_bf16

OP_INPUT, OP_CONV, OP_MAXPOOL, OP_ADD = 0, 1, 2, 3


def out_size(n, k, s, p):
    """Output extent of a k-window with stride s and padding p over n cells
    (Section III-B, read as floor((n + 2p - k) / s) + 1)."""
    return (n + 2 * p - k) // s + 1


def _taps(kh, kw):
    return [(i, j) for i in range(kh) for j in range(kw)]


def _pad(x, ph, pw, value=0.0):
    b, h, w, c = x.shape
    xp = np.full((b, h + 2 * ph, w + 2 * pw, c), value, dtype=np.float64)
    xp[:, ph:ph + h, pw:pw + w, :] = x
    return xp


def conv_fwd(x, w, sh, sw, ph, pw):
    """Cross-correlation, Eq. (1): out[b,y,x,o] = sum_{i,j,c} w[o,i,j,c] *
    xpad[b, y*sh+i, x*sw+j, c]. x is (B,H,W,C), w is (Co,kh,kw,Ci)."""
    b, h, wd, c = x.shape
    co, kh, kw, ci = w.shape
    assert ci == c
    ho, wo = out_size(h, kh, sh, ph), out_size(wd, kw, sw, pw)
    xp = _pad(x, ph, pw)
    out = np.zeros((b, ho, wo, co), dtype=np.float64)
    for i, j in _taps(kh, kw):
        patch = xp[:, i:i + sh * (ho - 1) + 1:sh, j:j + sw * (wo - 1) + 1:sw, :]
        out += patch @ w[:, i, j, :].T.astype(np.float64)
    return out


def conv_dgrad(dy, w, in_hw, sh, sw, ph, pw):
    """Error propagated to a convolution's input (the "Get_error" step of
    Algorithm 1): the adjoint of ``conv_fwd`` in x."""
    b, ho, wo, co = dy.shape
    _, kh, kw, ci = w.shape
    h, wd = in_hw
    dxp = np.zeros((b, h + 2 * ph, wd + 2 * pw, ci), dtype=np.float64)
    for i, j in _taps(kh, kw):
        dxp[:, i:i + sh * (ho - 1) + 1:sh, j:j + sw * (wo - 1) + 1:sw, :] += \
            dy @ w[:, i, j, :].astype(np.float64)
    return dxp[:, ph:ph + h, pw:pw + wd, :]


def conv_wgrad(dy, x, kh, kw, sh, sw, ph, pw):
    """Weight gradient g = Gradient(delta, z^{l-1}), Eq. (2): the adjoint of
    ``conv_fwd`` in w, in the (Co,kh,kw,Ci) layout."""
    b, ho, wo, co = dy.shape
    ci = x.shape[3]
    xp = _pad(x, ph, pw)
    dw = np.zeros((co, kh, kw, ci), dtype=np.float64)
    for i, j in _taps(kh, kw):
        patch = xp[:, i:i + sh * (ho - 1) + 1:sh, j:j + sw * (wo - 1) + 1:sw, :]
        dw[:, i, j, :] = np.tensordot(dy, patch, axes=([0, 1, 2], [0, 1, 2]))
    return dw


def maxpool_fwd(x, kh, kw, sh, sw, ph, pw):
    """Max-pool (the "internal pooling layer" of Section II-A) with -inf
    padding. Returns (values, argmax) where argmax is the row-major index of
    the first maximum inside the window (uint8)."""
    b, h, wd, c = x.shape
    ho, wo = out_size(h, kh, sh, ph), out_size(wd, kw, sw, pw)
    xp = _pad(x, ph, pw, value=-np.inf)
    best = None
    idx = np.zeros((b, ho, wo, c), dtype=np.uint8)
    for t, (i, j) in enumerate(_taps(kh, kw)):
        v = xp[:, i:i + sh * (ho - 1) + 1:sh, j:j + sw * (wo - 1) + 1:sw, :]
        if best is None:
            best = v.copy()
        else:
            m = v > best
            best[m] = v[m]
            idx[m] = t
    return best, idx


def maxpool_bwd(dy, idx, in_hw, kh, kw, sh, sw, ph, pw):
    """Route each output error to its window's argmax."""
    b, ho, wo, c = dy.shape
    h, wd = in_hw
    dxp = np.zeros((b, h + 2 * ph, wd + 2 * pw, c), dtype=np.float64)
    for t, (i, j) in enumerate(_taps(kh, kw)):
        dxp[:, i:i + sh * (ho - 1) + 1:sh, j:j + sw * (wo - 1) + 1:sw, :] += \
            np.where(idx == t, dy, 0.0)
    return dxp[:, ph:ph + h, pw:pw + wd, :]


def relu(t):
    """max(t, 0) with ReLU'(0) = 0; returns +0.0 for every t <= 0."""
    return np.where(t > 0, t, 0.0)


def shapes(nodes, h, w, c):
    """(H, W, C) of every node's output."""
    out = [(h, w, c)]
    for (op, in0, in1, co, kh, kw, sh, sw, ph, pw, aff, rl) in nodes[1:]:
        hi, wi, ci = out[in0]
        if op == OP_CONV:
            out.append((out_size(hi, kh, sh, ph), out_size(wi, kw, sw, pw), co))
        elif op == OP_MAXPOOL:
            out.append((out_size(hi, kh, sh, ph), out_size(wi, kw, sw, pw), ci))
        elif op == OP_ADD:
            assert out[in1] == out[in0]
            out.append(out[in0])
        else:
            raise ValueError("bad op")
    return out


def apply_node(node, srcs, w, scale, shift, bf16, want_pre=False):
    """Forward of one node given its input tensors. Returns (out, argmax),
    plus the value before ReLU (None for pooling) when ``want_pre``."""
    op, in0, in1, co, kh, kw, sh, sw, ph, pw, aff, rl = node
    idx = None
    t = None
    if op == OP_CONV:
        t = conv_fwd(srcs[0], w, sh, sw, ph, pw)
        if aff:
            t = t * scale.astype(np.float64) + shift.astype(np.float64)
        out = relu(t) if rl else t
    elif op == OP_MAXPOOL:
        out, idx = maxpool_fwd(srcs[0], kh, kw, sh, sw, ph, pw)
    elif op == OP_ADD:
        t = srcs[0] + srcs[1]
        out = relu(t) if rl else t
    else:
        raise ValueError("bad op")
    if bf16:
        out = round_bf16(out)
    if want_pre:
        return out, idx, t
    return out, idx


def forward(nodes, x, weights, scales, shifts, bf16=False, keep_pre=False):
    """Column FP (Eq. (1) applied layer after layer). ``weights[v-1]`` etc.
    belong to node v. Returns (acts, argmax) with acts[0] = x; with
    ``keep_pre`` also the values before ReLU of every ReLU node (so a
    ReLU decision of another implementation can be judged a near-tie)."""
    acts = [np.asarray(x, dtype=np.float64)]
    argmax = [None]
    pre = [None]
    for v, node in enumerate(nodes[1:], start=1):
        srcs = [acts[node[1]]] + ([acts[node[2]]] if node[0] == OP_ADD else [])
        out, idx, t = apply_node(node, srcs, weights[v - 1], scales[v - 1],
                                 shifts[v - 1], bf16, want_pre=True)
        pre.append(t if (keep_pre and node[11]) else None)
        acts.append(out)
        argmax.append(idx)
    if keep_pre:
        return acts, argmax, pre
    return acts, argmax


def error_operand(node, d, z, scale, bf16, mask=None):
    """delta entering a conv's gradient kernels: delta * [z > 0] (ReLU) times
    the affine scale, rounded to bf16 when emulating bf16 storage."""
    op, in0, in1, co, kh, kw, sh, sw, ph, pw, aff, rl = node
    if rl:
        d = d * (mask if mask is not None else (z > 0))
    if aff:
        d = d * scale.astype(np.float64)
    return round_bf16(d) if bf16 else d


def backward(nodes, acts, argmax, weights, scales, g, bf16=False, masks=None,
             want_dx=True):
    """Column BP (Eq. (2); Algorithm 1's BP loop run over the whole map).
    ``masks`` optionally replaces the ReLU masks / pool argmax derived from
    ``acts`` (node index -> bool array or uint8 argmax), so a gradient can be
    checked against another implementation's ReLU/argmax decisions.
    Returns (dW per node or None, dX)."""
    n = len(nodes)
    delta = [None] * n
    delta[n - 1] = np.asarray(g, dtype=np.float64)
    dws = [None] * n
    masks = masks or {}

    def acc(u, t):
        delta[u] = t if delta[u] is None else delta[u] + t

    for v in range(n - 1, 0, -1):
        node = nodes[v]
        op, in0, in1, co, kh, kw, sh, sw, ph, pw, aff, rl = node
        d = delta[v]
        if d is None:
            d = np.zeros_like(acts[v])
        hu, wu = acts[in0].shape[1:3]
        if op == OP_CONV:
            dc = error_operand(node, d, acts[v], scales[v - 1], bf16,
                               masks.get(v))
            dws[v] = conv_wgrad(dc, acts[in0], kh, kw, sh, sw, ph, pw)
            if in0 != 0 or want_dx:
                acc(in0, conv_dgrad(dc, weights[v - 1], (hu, wu), sh, sw, ph, pw))
        elif op == OP_MAXPOOL:
            idx = masks.get(v, argmax[v])
            acc(in0, maxpool_bwd(d, idx, (hu, wu), kh, kw, sh, sw, ph, pw))
        elif op == OP_ADD:
            if rl:
                m = masks.get(v)
                d = d * (m if m is not None else (acts[v] > 0))
            acc(in0, d)
            acc(in1, d)
        delta[v] = None
    return dws, delta[0]


def relu_masks(nodes, acts):
    """ReLU masks [z > 0] of every ReLU site (node index -> bool array)."""
    return {v: acts[v] > 0 for v, nd in enumerate(nodes)
            if v > 0 and nd[11] and nd[0] in (OP_CONV, OP_ADD)}


def flops_forward(nodes, batch, h, w, c):
    """tau of Section IV-B: sum over conv layers of 2 k^2 B C^{l-1} C^l H^l W^l
    (generalised to kh*kw), counted from the output shapes."""
    shp = shapes(nodes, h, w, c)
    tot = 0
    for v, (op, in0, in1, co, kh, kw, *_r) in enumerate(nodes):
        if op == OP_CONV:
            ho, wo, _ = shp[v]
            tot += 2 * kh * kw * batch * shp[in0][2] * co * ho * wo
    return tot
