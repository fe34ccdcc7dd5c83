"""Pins of ``oracle/bounds.py``, the per-site bounds that certify a
differing ReLU / argmax decision.

* ``conv_abs_at`` equals the oracle convolution of |x| with |w| at every
  site (brute-force agreement with ``column.conv_fwd``).
* The bounds hold for float32 implementations written here independently
  of the oracle: one convolution layer computed by torch's CPU float32
  convolution (its own summation order) and by a float32 tap loop in
  reverse tap order, on inputs perturbed by up to kappa units of their
  storage rounding, stays within E_t of the float64 pre-activation at
  every site; so does a float32 residual add; every ReLU or argmax
  decision such an implementation flips is certified.
* A planted mistake (one weight off by 2%) breaks the bound.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import bounds as OB, column as C
from oracle.bf16 import round_bf16

rng = np.random.default_rng(42)


def perturb(x, kappa, bf16):
    u = OB.unit(bf16)
    return x * (1 + rng.uniform(-kappa * u, kappa * u, x.shape))


def conv32(x, w, s, p, kind):
    x32, w32 = x.astype(np.float32), w.astype(np.float32)
    if kind == "torch":
        return F.conv2d(torch.from_numpy(x32).permute(0, 3, 1, 2),
                        torch.from_numpy(w32).permute(0, 3, 1, 2), stride=s,
                        padding=p).permute(0, 2, 3, 1).contiguous().numpy()
    b_, h, wd, c = x32.shape
    co, kh, kw, _ = w32.shape
    ho, wo = (h + 2 * p - kh) // s + 1, (wd + 2 * p - kw) // s + 1
    xp = np.zeros((b_, h + 2 * p, wd + 2 * p, c), np.float32)
    xp[:, p:p + h, p:p + wd] = x32
    out = np.zeros((b_, ho, wo, co), np.float32)
    for i in reversed(range(kh)):
        for j in reversed(range(kw)):
            patch = xp[:, i:i + s * (ho - 1) + 1:s, j:j + s * (wo - 1) + 1:s]
            out = (out + patch @ w32[:, i, j, :].T).astype(np.float32)
    return out


def all_sites(shape):
    return np.argwhere(np.ones(shape, bool))


def test_conv_abs_at_matches_convolution_of_magnitudes():
    x, w = rng.standard_normal((2, 9, 7, 5)), rng.standard_normal((4, 3, 3, 5))
    ref = C.conv_fwd(np.abs(x), np.abs(w), 2, 2, 1, 1)
    got = OB.conv_abs_at(x, w, 2, 2, 1, 1, all_sites(ref.shape)).reshape(ref.shape)
    np.testing.assert_allclose(got, ref, rtol=1e-13, atol=0)


@pytest.mark.parametrize("bf16", [False, True])
@pytest.mark.parametrize("kind", ["torch", "taps_reversed"])
@pytest.mark.parametrize("kappa", [1, 4])
def test_conv_site_bound_holds_for_float32_layers(bf16, kind, kappa):
    x = rng.standard_normal((2, 11, 9, 24))
    w = rng.standard_normal((16, 3, 3, 24)) * np.sqrt(2 / 216)
    if bf16:
        x, w = round_bf16(x), round_bf16(w)
    scale, shift = rng.uniform(0.5, 1, 16), rng.uniform(-0.1, 0.1, 16)
    t = C.conv_fwd(x, w, 1, 1, 1, 1) * scale + shift
    xp = perturb(x, kappa, bf16)
    t32 = (conv32(xp, w, 1, 1, kind) * scale.astype(np.float32)
           + shift.astype(np.float32)).astype(np.float32)
    sites = all_sites(t.shape)
    S = OB.conv_abs_at(x, w, 1, 1, 1, 1, sites).reshape(t.shape)
    o = np.broadcast_to(np.arange(16), t.shape)
    # (the float32 copy of a perturbed input adds one more rounding)
    Et = OB.conv_site_bound(S, 216, t, scale, shift, o, kappa + 1, bf16)
    assert (np.abs(t32 - t) <= Et).all()
    flips = OB.relu_flips(t, (t32 > 0).astype(np.uint8))
    for b, y, xx, c in flips:
        assert abs(t[b, y, xx, c]) <= Et[b, y, xx, c]
    # not vacuous: the bound is a small part of the values' spread
    assert np.median(Et) < 0.2 * np.std(t)


def test_planted_mistake_breaks_the_conv_bound():
    x = rng.standard_normal((1, 8, 8, 16))
    w = rng.standard_normal((8, 3, 3, 16)) * np.sqrt(2 / 144)
    t = C.conv_fwd(x, w, 1, 1, 1, 1)
    wbad = w.copy()
    wbad[0, 1, 1, 0] *= 1.02
    t32 = conv32(x, wbad, 1, 1, "torch")
    S = OB.conv_abs_at(x, w, 1, 1, 1, 1, all_sites(t.shape)).reshape(t.shape)
    o = np.broadcast_to(np.arange(8), t.shape)
    Et = OB.conv_site_bound(S, 144, t, None, None, o, 1, False)
    assert (np.abs(t32 - t) > Et).any()


@pytest.mark.parametrize("bf16", [False, True])
def test_add_site_bound_holds(bf16):
    za, zb = rng.standard_normal((3, 50)), rng.standard_normal((3, 50))
    if bf16:
        za, zb = round_bf16(za), round_bf16(zb)
    t = za + zb
    t32 = (perturb(za, 2, bf16).astype(np.float32) + perturb(zb, 2, bf16).astype(np.float32))
    # perturbed by 2 units, plus the float32 copy's rounding
    assert (np.abs(t32 - t) <= OB.add_site_bound(za, zb, t, 3, bf16)).all()


def test_argmax_certification():
    node = (2, 0, -1, 0, 2, 2, 2, 2, 0, 0, 0, 0)
    z = np.array([[[[1.0], [1.0 + 1e-6]], [[0.0], [0.5]]]])  # one 2x2 window
    oracle_idx = np.array([[[[1]]]], np.uint8)
    assert OB.argmax_flips(node, z, oracle_idx, np.array([[[[0]]]], np.uint8), 1, False) == (1, 1)
    assert OB.argmax_flips(node, z, oracle_idx, np.array([[[[0]]]], np.uint8), 1, True) == (1, 0)
    assert OB.argmax_flips(node, z, oracle_idx, np.array([[[[3]]]], np.uint8), 4, True) == (1, 1)
    assert OB.argmax_flips(node, z, oracle_idx, oracle_idx, 1, True) == (0, 0)


@pytest.mark.parametrize("bf16", [False, True])
def test_pool_flips_of_perturbed_values_are_certified(bf16):
    node = (2, 0, -1, 0, 3, 3, 2, 2, 1, 1, 0, 0)
    z = rng.standard_normal((2, 15, 13, 8))
    z = np.where(rng.random(z.shape) < 0.3, 0.0, z)  # ReLU-like zeros tie
    if bf16:
        z = round_bf16(z)
    _, oi = C.maxpool_fwd(z, 3, 3, 2, 2, 1, 1)
    _, gi = C.maxpool_fwd(perturb(z, 2, bf16), 3, 3, 2, 2, 1, 1)
    n, bad = OB.argmax_flips(node, z, oi, gi, 2, bf16)
    assert bad == 0
