"""Pins for the column oracle: brute force, library routines, closed forms,
adjoint identities and finite differences. CPU only."""
import itertools

import numpy as np
import pytest
import scipy.signal
import torch

from oracle import brute, column as C
from oracle.bf16 import round_bf16
from workloads import NetBuilder, tiny_net, Inputs, F32

rng = np.random.default_rng(1234)


def rand(*shape):
    return rng.standard_normal(shape)


CONV_CASES = [
    # (B, H, W, C, Co, k, s, p)
    (1, 5, 6, 2, 3, 3, 1, 1),
    (2, 7, 5, 3, 2, 3, 2, 1),
    (1, 6, 6, 2, 2, 2, 1, 0),
    (1, 9, 8, 1, 2, 5, 2, 2),
    (2, 4, 4, 2, 1, 1, 2, 0),
    (1, 8, 7, 2, 2, 7, 2, 3),
    (1, 5, 5, 3, 2, 4, 3, 2),
]


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv_matches_bruteforce(case):
    B, H, W, Ci, Co, k, s, p = case
    x, w = rand(B, H, W, Ci), rand(Co, k, k, Ci)
    ref = np.array(brute.conv(x, w, s, s, p, p))
    out = C.conv_fwd(x, w, s, s, p, p)
    assert out.shape == ref.shape
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)


def test_conv_matches_scipy_correlate2d():
    # stride 1: sum over channels of scipy's 2-D cross-correlation ('valid'
    # on the zero-padded image)
    x, w, p = rand(2, 9, 11, 3), rand(4, 3, 5, 3), (1, 2)
    out = C.conv_fwd(x, w, 1, 1, p[0], p[1])
    for b in range(2):
        for o in range(4):
            acc = 0
            for c in range(3):
                img = np.pad(x[b, :, :, c], ((p[0], p[0]), (p[1], p[1])))
                acc = acc + scipy.signal.correlate2d(img, w[o, :, :, c], "valid")
            np.testing.assert_allclose(out[b, :, :, o], acc, atol=1e-12)


def test_1x1_conv_is_matmul():
    x, w = rand(2, 5, 4, 6), rand(3, 1, 1, 6)
    np.testing.assert_allclose(C.conv_fwd(x, w, 1, 1, 0, 0),
                               x @ w[:, 0, 0, :].T, atol=1e-13)


def test_delta_kernel_is_shift():
    # a kernel with a single identity tap at (2, 0) shifts rows up by 1 when
    # p = 1 (output row y reads input row y - 1 + 2)
    x = rand(1, 6, 5, 2)
    w = np.zeros((2, 3, 3, 2))
    w[0, 2, 0, 0] = w[1, 2, 0, 1] = 1.0
    out = C.conv_fwd(x, w, 1, 1, 1, 1)
    exp = np.zeros_like(x)
    exp[:, :5, 1:, :] = x[:, 1:, :4, :]
    np.testing.assert_array_equal(out, exp)


def test_constant_input_closed_form():
    a = 1.75
    x = np.full((1, 6, 6, 3), a)
    w = rand(4, 3, 3, 3)
    out = C.conv_fwd(x, w, 1, 1, 0, 0)
    exp = a * w.sum(axis=(1, 2, 3))
    np.testing.assert_allclose(out, np.broadcast_to(exp, out.shape), atol=1e-12)


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv_adjoint_identities(case):
    B, H, W, Ci, Co, k, s, p = case
    x, w = rand(B, H, W, Ci), rand(Co, k, k, Ci)
    y = C.conv_fwd(x, w, s, s, p, p)
    g = rand(*y.shape)
    lhs = np.vdot(y, g)
    dx = C.conv_dgrad(g, w, (H, W), s, s, p, p)
    dw = C.conv_wgrad(g, x, k, k, s, s, p, p)
    assert dx.shape == x.shape and dw.shape == w.shape
    assert abs(lhs - np.vdot(x, dx)) <= 1e-12 * max(1, abs(lhs)) * 10
    assert abs(lhs - np.vdot(w, dw)) <= 1e-12 * max(1, abs(lhs)) * 10


@pytest.mark.parametrize("k,s,p", [(2, 2, 0), (3, 2, 1), (3, 1, 1), (2, 1, 0)])
def test_maxpool_matches_bruteforce(k, s, p):
    x = rand(2, 7, 6, 3)
    val, idx = C.maxpool_fwd(x, k, k, s, s, p, p)
    bv, bi = brute.maxpool(x, k, k, s, s, p, p)
    np.testing.assert_array_equal(val, np.array(bv))
    np.testing.assert_array_equal(idx, np.array(bi))


@pytest.mark.parametrize("k,s,p", [(2, 2, 0), (3, 2, 1)])
def test_maxpool_matches_torch_indices(k, s, p):
    # library routine: torch CPU max_pool2d with flat input indices (no ties
    # in continuous random data)
    x = rand(1, 9, 8, 2)
    val, idx = C.maxpool_fwd(x, k, k, s, s, p, p)
    t = torch.from_numpy(x.transpose(0, 3, 1, 2).copy())
    tv, ti = torch.nn.functional.max_pool2d(t, k, s, p, return_indices=True)
    np.testing.assert_array_equal(val, tv.numpy().transpose(0, 2, 3, 1))
    ti = ti.numpy().transpose(0, 2, 3, 1)
    ho, wo = val.shape[1:3]
    yy, xx = np.meshgrid(np.arange(ho), np.arange(wo), indexing="ij")
    r = yy[None, :, :, None] * s - p + idx // k
    q = xx[None, :, :, None] * s - p + idx % k
    np.testing.assert_array_equal(r * x.shape[2] + q, ti)


def test_maxpool_ties_first_max():
    # all-equal window -> index 0; equal maxima -> the first in row-major order
    x = np.zeros((1, 4, 4, 1))
    x[0, 2, 3, 0] = 5.0
    x[0, 3, 2, 0] = 5.0
    val, idx = C.maxpool_fwd(x, 2, 2, 2, 2, 0, 0)
    assert idx[0, 0, 0, 0] == 0 and val[0, 0, 0, 0] == 0.0
    assert idx[0, 1, 1, 0] == 1  # (2,3) precedes (3,2) in row-major order
    # with -inf padding a border window never picks a padded position
    x = -np.ones((1, 3, 3, 1))
    val, idx = C.maxpool_fwd(x, 3, 3, 2, 2, 1, 1)
    # first in-image position of each window (row-major over the 3x3 window)
    np.testing.assert_array_equal(idx[0, :, :, 0], [[4, 3], [1, 0]])
    assert (val == -1).all()
    _, bi = brute.maxpool(x, 3, 3, 2, 2, 1, 1)
    np.testing.assert_array_equal(idx, np.array(bi))


@pytest.mark.parametrize("k,s,p", [(2, 2, 0), (3, 2, 1)])
def test_maxpool_backward_adjoint(k, s, p):
    x = rand(2, 8, 7, 2)
    val, idx = C.maxpool_fwd(x, k, k, s, s, p, p)
    g = rand(*val.shape)
    dx = C.maxpool_bwd(g, idx, (8, 7), k, k, s, s, p, p)
    assert abs(np.vdot(val, g) - np.vdot(x, dx)) < 1e-12 * 100


def _small_dag():
    nb = NetBuilder()
    a = nb.conv(0, 4, 3, 1, 1, affine=1, relu=1)
    b = nb.pool(a, 3, 2, 1)
    c = nb.conv(b, 4, 3, 1, 1, affine=1, relu=1)
    d = nb.conv(c, 6, 1, 1, 0, affine=1, relu=0)
    e = nb.conv(b, 6, 1, 1, 0, affine=1, relu=0)
    f = nb.sum(d, e, relu=1)
    g = nb.conv(f, 5, 3, 2, 1, affine=0, relu=1)
    nb.pool(g, 2, 2, 0)
    return nb.nodes


def _loss(nodes, x, ws, scs, shs, g):
    acts, am = C.forward(nodes, x, ws, scs, shs)
    return float(np.vdot(acts[-1], g)), acts, am


@pytest.mark.parametrize("netname", ["tiny", "dag"])
def test_full_net_gradients_finite_difference(netname):
    nodes = tiny_net() if netname == "tiny" else _small_dag()
    inp = Inputs(nodes, 2, 12, 10, 3, F32, seed=7)
    x = inp.x.astype(np.float64)
    ws = [None if w is None else w.astype(np.float64) for w in inp.weights]
    acts, am = C.forward(nodes, x, ws, inp.scales, inp.shifts)
    g = rand(*acts[-1].shape)
    dws, dx = C.backward(nodes, acts, am, ws, inp.scales, g)
    masks0 = (C.relu_masks(nodes, acts), [a for a in am if a is not None])
    h = 1e-6
    checked = 0
    for trial in range(6):
        vx = rand(*x.shape)
        vw = [None if w is None else rand(*w.shape) for w in ws]
        wp = [None if w is None else w + h * d for w, d in zip(ws, vw)]
        wm = [None if w is None else w - h * d for w, d in zip(ws, vw)]
        lp, ap, amp = _loss(nodes, x + h * vx, wp, inp.scales, inp.shifts, g)
        lm, am_, amm = _loss(nodes, x - h * vx, wm, inp.scales, inp.shifts, g)
        # reject directions that flip a ReLU or an argmax (non-smooth point)
        same = all(np.array_equal(m, C.relu_masks(nodes, a)[v])
                   for a in (ap, am_) for v, m in masks0[0].items())
        same &= all(np.array_equal(i0, i1) for am2 in (amp, amm)
                    for i0, i1 in zip(masks0[1], [q for q in am2 if q is not None]))
        if not same:
            continue
        fd = (lp - lm) / (2 * h)
        an = np.vdot(dx, vx) + sum(np.vdot(dws[v], vw[v - 1])
                                   for v in range(1, len(nodes)) if dws[v] is not None)
        assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (fd, an)
        checked += 1
    assert checked >= 3


def test_forward_convention_relu_and_affine():
    # single conv with affine and ReLU: out = max(a*conv + b, 0)
    nb = NetBuilder()
    nb.conv(0, 3, 3, 1, 1, affine=1, relu=1)
    inp = Inputs(nb.nodes, 1, 5, 5, 2, F32, seed=3)
    acts, _ = C.forward(nb.nodes, inp.x, inp.weights, inp.scales, inp.shifts)
    raw = np.array(brute.conv(inp.x, inp.weights[0], 1, 1, 1, 1))
    exp = np.maximum(raw * inp.scales[0] + inp.shifts[0], 0)
    np.testing.assert_allclose(acts[1], exp, atol=1e-6)


# ------------------------------------------------------------------ bf16
def test_round_bf16_matches_library_conversion():
    v = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-30, 30, 20000),
                        [0.0, -0.0, 1.0, -2.5, 3.0e38, 1e-40, -1e-39]]).astype(np.float32)
    lib = torch.from_numpy(v).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(round_bf16(v.astype(np.float64)), lib.astype(np.float64))


def test_round_bf16_ties_to_even():
    assert round_bf16(1.0 + 2.0 ** -8) == 1.0              # tie -> even (down)
    assert round_bf16(1.0 + 3 * 2.0 ** -8) == 1.0 + 2.0 ** -6  # tie -> even (up)
    assert round_bf16(1.0 + 2.0 ** -8 + 2.0 ** -20) == 1.0 + 2.0 ** -7
    assert round_bf16(-(1.0 + 2.0 ** -8)) == -1.0


def test_bf16_mode_stores_representable_values():
    nodes = _small_dag()
    inp = Inputs(nodes, 1, 10, 9, 3, 1, seed=5)
    acts, _ = C.forward(nodes, inp.x, inp.weights, inp.scales, inp.shifts, bf16=True)
    for a in acts:
        np.testing.assert_array_equal(round_bf16(a), a)


def test_tau_counts_multiply_adds():
    # tau (Section IV-B) = 2 * (number of multiply-adds of the forward convs);
    # count the products a direct evaluation performs, padding taps included
    nodes = _small_dag()
    shp = C.shapes(nodes, 10, 9, 3)
    macs = 0
    for v, nd in enumerate(nodes):
        if nd[0] == C.OP_CONV:
            ho, wo, co = shp[v]
            for _ in itertools.product(range(ho), range(wo), range(co),
                                       range(nd[4]), range(nd[5]),
                                       range(shp[nd[1]][2])):
                macs += 1
    assert C.flops_forward(nodes, 1, 10, 9, 3) == 2 * macs
