"""Certification of ReLU and max-pool decisions that differ from the oracle's.

TEST INFRASTRUCTURE (see ``oracle/column.py``): only ``tests/`` may use it.

The paper states no precision. An implementation that stores node outputs
in float32 (or bfloat16, rounded at the oracle's emulated points) and sums
each convolution's products in float32 in any order reaches its ReLU and
argmax decisions from its own stored inputs, which differ from the
oracle's by rounding; a decision can then legitimately differ from the
oracle's. Such a decision is certified when it is the one the
implementation's own stored inputs imply, up to the implementation's own
accumulation error at that site. The bound follows standard floating-point
error analysis (Higham, "Accuracy and Stability of Numerical Algorithms",
2nd ed., Section 3.1: a sum of n terms computed in floating point with unit
roundoff u, in any order, differs from the exact sum by at most gamma_n
times the sum of the terms' magnitudes, gamma_n = n u / (1 - n u)):

* convolution site with inputs x'_k (the implementation's stored values)
  and weights w_k, K = kh * kw * C_in products: the exact sum
  c = sum_k w_k x'_k is computed here in float64 and the implementation's
  value lies within gamma_{K+1} * sum_k |w_k| |x'_k| of it (gamma's "+1"
  covers the rounding of each product); a fixed affine a * c + b in float32
  adds two roundings;
* residual add of two stored values: their exact sum has the sign the
  float32 sum has, so the decision must match it exactly; when one input is
  a convolution whose value the add consumes without storing it, that
  value's accumulation error and its storage rounding are added;
* max-pool compares stored values without arithmetic, so the chosen index
  must be the first maximum of the implementation's own window.

A decision is certified when it equals the sign (ReLU) of the exact value
from the implementation's inputs or that value lies within the bound.
"""
from __future__ import annotations

import numpy as np

U32 = 2.0 ** -24   # unit roundoff of float32, round to nearest
UBF16 = 2.0 ** -8  # unit roundoff of bfloat16, round to nearest


def gamma(n, u=U32):
    """gamma_n = n u / (1 - n u) (Higham, Section 3.1)."""
    nu = n * u
    assert nu < 1
    return nu / (1.0 - nu)


def unit(bf16):
    """Unit roundoff of the storage type."""
    return UBF16 if bf16 else U32


def _taps_at(x, w, sh, sw, ph, pw, sites, absolute):
    sites = np.asarray(sites).reshape(-1, 4)
    out = np.zeros(len(sites))
    if len(sites) == 0:
        return out
    h, wd = x.shape[1:3]
    co, kh, kw, ci = w.shape
    b, y, xx, o = (sites[:, k] for k in range(4))
    ww = np.asarray(w, dtype=np.float64)
    if absolute:
        ww = np.abs(ww)
    for i in range(kh):
        for j in range(kw):
            sy, sx = y * sh - ph + i, xx * sw - pw + j
            ok = (sy >= 0) & (sy < h) & (sx >= 0) & (sx < wd)
            v = x[b, np.clip(sy, 0, h - 1), np.clip(sx, 0, wd - 1), :].astype(np.float64)
            if absolute:
                v = np.abs(v)
            out += np.where(ok, np.einsum("nc,nc->n", v, ww[o, i, j, :]), 0.0)
    return out


def conv_at(x, w, sh, sw, ph, pw, sites):
    """Exact (float64) sum_{i,j,c} w[o,i,j,c] x[b, y*sh - ph + i, x*sw - pw + j, c]
    at output sites (rows of (b, y, x, o)); outside the image nothing is
    added (zero padding)."""
    return _taps_at(x, w, sh, sw, ph, pw, sites, False)


def conv_abs_at(x, w, sh, sw, ph, pw, sites):
    """The same sum of |w| |x| (the magnitude the accumulation bound scales)."""
    return _taps_at(x, w, sh, sw, ph, pw, sites, True)


def conv_site(x, w, scale, shift, node, sites):
    """(t, E) at conv sites: t the exact pre-activation from inputs x (the
    affine applied in float64), E the bound on the implementation's float32
    accumulation and affine rounding."""
    op, in0, in1, co, kh, kw, sh, sw, ph, pw, aff, rl = node
    sites = np.asarray(sites).reshape(-1, 4)
    c = conv_at(x, w, sh, sw, ph, pw, sites)
    S = conv_abs_at(x, w, sh, sw, ph, pw, sites)
    E = gamma(kh * kw * x.shape[3] + 1) * S
    if not aff:
        return c, E
    o = sites[:, 3]
    a = np.asarray(scale, dtype=np.float64)[o]
    b = np.asarray(shift, dtype=np.float64)[o]
    t = a * c + b
    return t, np.abs(a) * E + 2.0 * U32 * (np.abs(a * c) + np.abs(a) * E + np.abs(b))


def fused_conv_value_bound(t, E, bf16):
    """Bound on |r' - t| for the stored (rounded) value r' of a conv whose
    exact value from the implementation's inputs is t, known within E."""
    return E + unit(bf16) * (np.abs(t) + E)


def relu_certified(t, E, decision):
    """Decisions (bool) at sites with exact values t and bounds E that are
    certified: equal to t > 0, or |t| <= E."""
    return (decision == (t > 0)) | (np.abs(t) <= E)


def pool_first_max_violations(node, z, idx):
    """Number of max-pool outputs whose index (row-major in the window) is
    not the first maximum of window values z (-inf padding)."""
    op, in0, in1, co, kh, kw, sh, sw, ph, pw, aff, rl = node
    b_, ho, wo, c_ = idx.shape
    h, w = z.shape[1:3]
    best = np.full(idx.shape, -np.inf)
    first = np.zeros(idx.shape, np.int64)
    for i in range(kh):
        for j in range(kw):
            yy = np.arange(ho)[None, :, None, None] * sh - ph + i
            xx = np.arange(wo)[None, None, :, None] * sw - pw + j
            ok = (yy >= 0) & (yy < h) & (xx >= 0) & (xx < w)
            v = np.where(ok, z[:, np.clip(yy[0, :, 0, 0], 0, h - 1)][:, :,
                                np.clip(xx[0, 0, :, 0], 0, w - 1)], -np.inf)
            better = v > best
            best = np.where(better, v, best)
            first = np.where(better, i * kw + j, first)
    return int((first != idx).sum())
