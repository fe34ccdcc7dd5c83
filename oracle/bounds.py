"""Per-site bounds that certify a differing ReLU or max-pool decision.

TEST INFRASTRUCTURE (see ``oracle/column.py``): only ``tests/`` may use it.

The paper states no precision. The parity protocol compares an
implementation that stores node outputs in float32, or in bfloat16 rounded
to nearest even at the oracle's emulated rounding points, and sums each
convolution's products in float32 in any order, with the float64 oracle.
Its ReLU and argmax decisions can then legitimately differ from the
oracle's where the oracle's pre-activation (or the gap between two window
values) lies within the implementation's possible deviation at that site.

The bound of one site assumes that the stored values the site reads differ
from the oracle's by at most kappa units of their storage rounding
(kappa * u * |value|, u = 2^-24 for float32, 2^-8 for bfloat16); the test
measures kappa on the network output, the deepest and largest deviation.
Given that, by standard floating-point error analysis (Higham, "Accuracy
and Stability of Numerical Algorithms", 2nd ed., Section 3.1: a sum of n
terms computed in floating point with unit roundoff u, in any order,
differs from the exact sum by at most gamma_n times the sum of the terms'
magnitudes, gamma_n = n u / (1 - n u)):

* convolution site, K = kh * kw * C_in products of weights w_k and inputs
  x_k: |conv' - conv| <= (kappa u_s + gamma_{K+1}(1 + kappa u_s)) S,
  S = sum_k |w_k| |x_k| (gamma's "+1" covers the rounding of each product);
* fixed affine a * c + b in float32: |a| times that, plus two roundings;
* residual add z_a + z_b in float32: kappa u_s (|z_a| + |z_b|) plus one
  rounding;
* max-pool: window values x_i, x_j each within kappa u_s of their own
  magnitude.

A ReLU decision may differ only where |t| <= E_t; an argmax may differ
only where the oracle's maximum x_i and the implementation's choice x_j
satisfy x_i - x_j <= kappa u_s (|x_i| + |x_j|).
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


def conv_abs_at(x, w, sh, sw, ph, pw, sites):
    """S = sum over taps and input channels of |w[o, i, j, c]| * |x[b, y*sh -
    ph + i, x*sw - pw + j, c]| at the given output sites (rows of
    (b, y, x, o)); positions outside the image contribute nothing."""
    sites = np.asarray(sites).reshape(-1, 4)
    b_, h, wd, c = x.shape
    co, kh, kw, ci = w.shape
    out = np.zeros(len(sites))
    if len(sites) == 0:
        return out
    b, y, xx, o = (sites[:, k] for k in range(4))
    aw = np.abs(np.asarray(w, dtype=np.float64))
    for i in range(kh):
        for j in range(kw):
            sy, sx = y * sh - ph + i, xx * sw - pw + j
            ok = (sy >= 0) & (sy < h) & (sx >= 0) & (sx < wd)
            v = np.abs(x[b, np.clip(sy, 0, h - 1), np.clip(sx, 0, wd - 1), :].astype(np.float64))
            out += np.where(ok, np.einsum("nc,nc->n", v, aw[o, i, j, :]), 0.0)
    return out


def conv_site_bound(S, K, t, scale, shift, o, kappa, bf16):
    """Bound E_t on |t' - t| at convolution sites with S (conv_abs_at), K
    products each, pre-activations t and output channels o."""
    us = unit(bf16)
    d = (kappa * us + gamma(K + 1) * (1.0 + kappa * us)) * S
    if scale is None:
        return d
    a = np.abs(np.asarray(scale, dtype=np.float64))[o]
    bb = np.abs(np.asarray(shift, dtype=np.float64))[o]
    ac = np.abs(t - np.asarray(shift, dtype=np.float64)[o])
    return a * d + 2.0 * U32 * (ac + a * d + bb)


def add_site_bound(za, zb, t, kappa, bf16):
    """Bound E_t on |t' - t| of a residual add t = z_a + z_b at its sites."""
    e = kappa * unit(bf16) * (np.abs(za) + np.abs(zb))
    return e + U32 * (np.abs(t) + e)


def relu_flips(t, gpu_mask):
    """Sites (b, y, x, c) where the implementation's ReLU decision
    (gpu_mask != 0) differs from the oracle's (t > 0)."""
    return np.argwhere((gpu_mask != 0) != (t > 0))


def argmax_flips(node, z_in, oracle_idx, gpu_idx, kappa, bf16):
    """(differing argmax decisions, of which not certified) of a max-pool
    node: the oracle's maximum x_i and the implementation's choice x_j may
    differ only where x_i - x_j <= kappa u_s (|x_i| + |x_j|)."""
    op, in0, in1, co, kh, kw, sh, sw, ph, pw, aff, rl = node
    diff = gpu_idx != oracle_idx
    if not diff.any():
        return 0, 0
    h, w = z_in.shape[1:3]
    bb, yy, xx, cc = np.nonzero(diff)

    def at(idx):
        iy = yy * sh - ph + idx[bb, yy, xx, cc] // kw
        ix = xx * sw - pw + idx[bb, yy, xx, cc] % kw
        ok = (iy >= 0) & (iy < h) & (ix >= 0) & (ix < w)
        v = z_in[bb, np.clip(iy, 0, h - 1), np.clip(ix, 0, w - 1), cc].astype(np.float64)
        return np.where(ok, v, -np.inf)

    xi, xj = at(oracle_idx), at(gpu_idx)
    with np.errstate(invalid="ignore"):
        bad = ~(xi - xj <= kappa * unit(bf16) * (np.abs(xi) + np.abs(xj)))
    return int(diff.sum()), int(bad.sum())
