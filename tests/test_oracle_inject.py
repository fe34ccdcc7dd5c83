"""Pins of the oracle's decision-injection path: ``column.backward(masks=...)``
is what every GPU gradient comparison runs through (the GPU's ReLU and
argmax decisions are injected), so it must

* reproduce the plain backward bit for bit when given the oracle's own
  decisions;
* treat an injected all-ones ReLU mask exactly like a site without ReLU;
* route a max-pool's error to the injected window position (brute force);
* drop exactly one site's term when one ReLU decision is switched off
  (the weight gradient changes by that site's outer product, computed by
  brute force).
"""
import numpy as np
import pytest

from oracle import column as C
from workloads import NetBuilder, Inputs, F32, BF16


def small_dag():
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


def run(nodes, inp, bf16, masks=None, nodes_bwd=None):
    acts, am = C.forward(nodes, inp.x, inp.weights, inp.scales, inp.shifts, bf16=bf16)
    g = inp.grad(acts[-1].shape)
    dws, dx = C.backward(nodes_bwd or nodes, acts, am, inp.weights, inp.scales, g, bf16=bf16,
                         masks=masks)
    return acts, am, g, dws, dx


def own_decisions(nodes, acts, am):
    m = dict(C.relu_masks(nodes, acts))
    for v, nd in enumerate(nodes):
        if v and nd[0] == C.OP_MAXPOOL:
            m[v] = am[v]
    return m


@pytest.mark.parametrize("dtype", [F32, BF16])
def test_own_decisions_reproduce_plain_backward_bitwise(dtype):
    nodes = small_dag()
    inp = Inputs(nodes, 2, 13, 11, 3, dtype, seed=7)
    bf = dtype == BF16
    acts, am, g, dws, dx = run(nodes, inp, bf)
    m = own_decisions(nodes, acts, am)
    assert len(m) == sum(1 for v, nd in enumerate(nodes)
                         if v and (nd[0] == C.OP_MAXPOOL or nd[11]))
    _, _, _, dws2, dx2 = run(nodes, inp, bf, masks=m)
    assert np.array_equal(dx, dx2)
    for a, b in zip(dws, dws2):
        assert (a is None and b is None) or np.array_equal(a, b)


@pytest.mark.parametrize("site", ["conv", "add"])
def test_all_ones_mask_equals_site_without_relu(site):
    nodes = small_dag()
    inp = Inputs(nodes, 2, 13, 11, 3, F32, seed=3)
    acts, am = C.forward(nodes, inp.x, inp.weights, inp.scales, inp.shifts)
    v = 3 if site == "conv" else 6
    assert nodes[v][0] == (C.OP_CONV if site == "conv" else C.OP_ADD) and nodes[v][11]
    g = inp.grad(acts[-1].shape)
    ones = {v: np.ones(acts[v].shape, bool)}
    linear = [tuple(nd) for nd in nodes]
    nd = list(linear[v])
    nd[11] = 0
    linear[v] = tuple(nd)
    a = C.backward(nodes, acts, am, inp.weights, inp.scales, g, masks=ones)
    b = C.backward(linear, acts, am, inp.weights, inp.scales, g)
    assert np.array_equal(a[1], b[1])
    for x, y in zip(a[0], b[0]):
        assert (x is None and y is None) or np.array_equal(x, y)
    # and it differs from the plain backward (the mask was really used)
    c = C.backward(nodes, acts, am, inp.weights, inp.scales, g)
    assert not np.array_equal(a[1], c[1])


def test_injected_argmax_routes_to_that_position():
    nb = NetBuilder()
    nb.pool(0, 3, 2, 0)
    nodes = nb.nodes
    rng = np.random.default_rng(5)
    x = rng.standard_normal((2, 9, 7, 3))
    acts, am = C.forward(nodes, x, [None], [None], [None])
    dy = rng.standard_normal(acts[1].shape)
    idx = rng.integers(0, 9, acts[1].shape).astype(np.uint8)
    _, dx = C.backward(nodes, acts, am, [None], [None], dy, masks={1: idx})
    want = np.zeros_like(x)
    B, Ho, Wo, Cc = dy.shape
    for b in range(B):
        for y in range(Ho):
            for xx in range(Wo):
                for c in range(Cc):
                    t = int(idx[b, y, xx, c])
                    want[b, 2 * y + t // 3, 2 * xx + t % 3, c] += dy[b, y, xx, c]
    assert np.array_equal(dx, want)


def test_switching_one_relu_decision_drops_that_sites_term():
    nb = NetBuilder()
    nb.conv(0, 3, 3, 2, 1, affine=1, relu=1)
    nodes = nb.nodes
    inp = Inputs(nodes, 1, 7, 6, 2, F32, seed=11)
    acts, am = C.forward(nodes, inp.x, inp.weights, inp.scales, inp.shifts)
    g = inp.grad(acts[1].shape)
    mask = acts[1] > 0
    on = np.argwhere(mask)
    b, y, x, o = on[len(on) // 2]
    m2 = mask.copy()
    m2[b, y, x, o] = False
    dw0, _ = C.backward(nodes, acts, am, inp.weights, inp.scales, g, masks={1: mask})
    dw1, _ = C.backward(nodes, acts, am, inp.weights, inp.scales, g, masks={1: m2})
    # brute force: the site's error operand times the input window it reads
    dc = float(g[b, y, x, o]) * float(inp.scales[0][o])
    term = np.zeros_like(dw0[1])
    H, W = inp.x.shape[1:3]
    for i in range(3):
        for j in range(3):
            sy, sx = 2 * y - 1 + i, 2 * x - 1 + j
            if 0 <= sy < H and 0 <= sx < W:
                term[o, i, j, :] = dc * inp.x[b, sy, sx, :].astype(np.float64)
    assert np.allclose(dw0[1] - dw1[1], term, rtol=0, atol=1e-12)
    assert np.abs(term).max() > 0
