"""Pins of ``oracle/bounds.py``, the certification of a ReLU / argmax
decision from an implementation's own stored inputs.

* ``conv_at`` and ``conv_abs_at`` equal the oracle convolution of x with w
  and of |x| with |w| at every site.
* Float32 implementations written here independently of the oracle --
  torch's CPU float32 convolution (its own summation order) and a float32
  tap loop in reverse tap order -- stay within the accumulation bound E of
  the exact pre-activation from the same inputs at every site, in float32
  and bfloat16 storage; every decision they reach is certified. A planted
  mistake (one weight off by 2%) breaks the bound.
* A bfloat16-stored convolution value added to another stored value stays
  within the fused-value bound.
* The max-pool check accepts exactly the first maximum of the window.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import bounds as OB, column as C
from oracle.bf16 import round_bf16

rng = np.random.default_rng(42)


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


def test_site_sums_match_convolutions():
    x, w = rng.standard_normal((2, 9, 7, 5)), rng.standard_normal((4, 3, 3, 5))
    ref = C.conv_fwd(x, w, 2, 2, 1, 1)
    sites = all_sites(ref.shape)
    np.testing.assert_allclose(OB.conv_at(x, w, 2, 2, 1, 1, sites).reshape(ref.shape), ref,
                               rtol=1e-12, atol=1e-12)
    ref = C.conv_fwd(np.abs(x), np.abs(w), 2, 2, 1, 1)
    np.testing.assert_allclose(OB.conv_abs_at(x, w, 2, 2, 1, 1, sites).reshape(ref.shape),
                               ref, rtol=1e-13, atol=0)


@pytest.mark.parametrize("bf16", [False, True])
@pytest.mark.parametrize("kind", ["torch", "taps_reversed"])
@pytest.mark.parametrize("aff", [0, 1])
def test_float32_layers_stay_within_the_accumulation_bound(bf16, kind, aff):
    x = rng.standard_normal((2, 11, 9, 24)).astype(np.float32).astype(np.float64)
    w = (rng.standard_normal((16, 3, 3, 24)) * np.sqrt(2 / 216)).astype(np.float32)
    w = w.astype(np.float64)
    if bf16:
        x, w = round_bf16(x), round_bf16(w)
    scale = rng.uniform(0.5, 1, 16).astype(np.float32) if aff else None
    shift = rng.uniform(-0.1, 0.1, 16).astype(np.float32) if aff else None
    node = (1, 0, -1, 16, 3, 3, 1, 1, 1, 1, aff, 1)
    out = conv32(x, w, 1, 1, kind)
    if aff:
        out = (out * scale + shift).astype(np.float32)
    sites = all_sites(out.shape)
    t, E = OB.conv_site(x, w, scale, shift, node, sites)
    t, E = t.reshape(out.shape), E.reshape(out.shape)
    assert (np.abs(out.astype(np.float64) - t) <= E).all()
    assert OB.relu_certified(t, E, out > 0).all()
    assert np.median(E) < 1e-3 * np.std(t)  # the bound is tight enough to matter


def test_planted_mistake_breaks_the_bound():
    x = rng.standard_normal((1, 8, 8, 16)).astype(np.float32).astype(np.float64)
    w = (rng.standard_normal((8, 3, 3, 16)) * np.sqrt(2 / 144)).astype(np.float32)
    w = w.astype(np.float64)
    wbad = w.copy()
    wbad[0, 1, 1, 0] *= 1.02
    out = conv32(x, wbad, 1, 1, "torch")
    node = (1, 0, -1, 8, 3, 3, 1, 1, 1, 1, 0, 1)
    t, E = OB.conv_site(x, w, None, None, node, all_sites(out.shape))
    assert (np.abs(out.ravel().astype(np.float64) - t) > E).any()


def test_fused_conv_value_plus_stored_input():
    x = round_bf16(rng.standard_normal((2, 6, 5, 32)))
    w = round_bf16(rng.standard_normal((16, 1, 1, 32)) * 0.25)
    zb = round_bf16(rng.standard_normal((2, 6, 5, 16)))
    scale = rng.uniform(0.5, 1, 16).astype(np.float32)
    shift = rng.uniform(-0.1, 0.1, 16).astype(np.float32)
    node = (1, 0, -1, 16, 1, 1, 1, 1, 0, 0, 1, 0)
    c32 = (conv32(x, w, 1, 0, "torch") * scale + shift).astype(np.float32)
    stored = round_bf16(c32.astype(np.float64))
    t_impl = (stored.astype(np.float32) + zb.astype(np.float32)).astype(np.float64)
    sites = all_sites(c32.shape)
    t, E = OB.conv_site(x, w, scale, shift, node, sites)
    e = OB.fused_conv_value_bound(t, E, True).reshape(c32.shape)
    t = t.reshape(c32.shape)
    tot = t + zb
    assert (np.abs(t_impl - tot) <= e + OB.U32 * (np.abs(tot) + e)).all()


def test_pool_first_maximum():
    node = (2, 0, -1, 0, 3, 3, 2, 2, 1, 1, 0, 0)
    z = rng.standard_normal((2, 15, 13, 8))
    z = np.where(rng.random(z.shape) < 0.4, 0.0, z)  # ties between zeros
    _, idx = C.maxpool_fwd(z, 3, 3, 2, 2, 1, 1)
    assert OB.pool_first_max_violations(node, z, idx) == 0
    bad = idx.copy()
    bad[1, 2, 3, 4] = (bad[1, 2, 3, 4] + 1) % 9
    assert OB.pool_first_max_violations(node, z, bad) == 1
