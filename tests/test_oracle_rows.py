"""Pins for the row-partitioned oracle: partition invariance against the
column oracle, interval arithmetic against brute-force dependency sets, the
paper's worked examples, and negative tests for missing dependency handling.
CPU only."""
import json
import os

import numpy as np
import pytest

from oracle import brute, column as C, rows as R
from workloads import NetBuilder, Inputs, tiny_net, F32, BF16

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                   "paper_shape_examples.json")))


def chain_net(spec, cin=2):
    """spec: list of ('c', cout, k, s, p) or ('p', k, s, p)."""
    nb = NetBuilder()
    v = 0
    for t in spec:
        if t[0] == "c":
            v = nb.conv(v, t[1], t[2], t[3], t[4], affine=1, relu=1)
        else:
            v = nb.pool(v, t[1], t[2], t[3])
    return nb.nodes


def dag_net():
    nb = NetBuilder()
    a = nb.conv(0, 4, 7, 2, 3, affine=1, relu=1)
    b = nb.pool(a, 3, 2, 1)
    c1 = nb.conv(b, 3, 1, 1, 0, affine=1, relu=1)
    c2 = nb.conv(c1, 3, 3, 2, 1, affine=1, relu=1)
    c3 = nb.conv(c2, 6, 1, 1, 0, affine=1, relu=0)
    sc = nb.conv(b, 6, 1, 2, 0, affine=1, relu=0)
    s1 = nb.sum(c3, sc, relu=1)
    d1 = nb.conv(s1, 3, 1, 1, 0, affine=1, relu=1)
    d2 = nb.conv(d1, 3, 3, 1, 1, affine=1, relu=1)
    d3 = nb.conv(d2, 6, 1, 1, 0, affine=1, relu=0)
    nb.sum(d3, s1, relu=1)
    return nb.nodes


NETS = {
    "tiny": tiny_net(),
    "vgg_like": chain_net([("c", 4, 3, 1, 1), ("c", 4, 3, 1, 1), ("p", 2, 2, 0),
                           ("c", 5, 3, 1, 1), ("p", 2, 2, 0), ("c", 3, 3, 1, 1)]),
    "odd": chain_net([("c", 3, 5, 2, 2), ("c", 3, 2, 1, 0), ("p", 3, 2, 1),
                      ("c", 2, 4, 3, 1), ("c", 2, 1, 1, 0)]),
    "resnet_like": dag_net(),
}


def random_bounds(rng, h, nb):
    cuts = np.sort(rng.integers(0, h + 1, nb - 1))
    return [0] + [int(c) for c in cuts] + [h]


def column_ref(nodes, inp, g_seed=0, bf16=False):
    acts, am = C.forward(nodes, inp.x, inp.weights, inp.scales, inp.shifts, bf16)
    g = inp.grad(acts[-1].shape)
    dws, dx = C.backward(nodes, acts, am, inp.weights, inp.scales, g, bf16)
    return acts[-1], dws, dx, g


def rel(a, b):
    return np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)


@pytest.mark.parametrize("name", list(NETS))
@pytest.mark.parametrize("trial", range(3))
def test_carry_partition_invariance(name, trial):
    nodes = NETS[name]
    rng = np.random.default_rng(100 + trial)
    h = 37 + trial * 5
    inp = Inputs(nodes, 2, h, 11, 3, F32, seed=trial)
    y, dws, dx, g = column_ref(nodes, inp)
    nb = [1, 3, 5][trial]
    bounds = random_bounds(rng, h, nb) if trial else R.even_bounds(h, nb)
    yr, strips = R.carry_forward(nodes, inp.x, inp.weights, inp.scales,
                                 inp.shifts, bounds)
    np.testing.assert_array_equal(yr, y)  # forward is exact
    dwr, dxr = R.carry_backward(nodes, inp.x, inp.weights, inp.scales,
                                inp.shifts, g, bounds, strips)
    assert rel(dxr, dx) < 1e-12
    for a, b in zip(dwr, dws):
        if b is not None:
            assert rel(a, b) < 1e-12


@pytest.mark.parametrize("name", list(NETS))
def test_carry_with_empty_bands(name):
    nodes = NETS[name]
    h = 30
    inp = Inputs(nodes, 1, h, 9, 3, F32, seed=11)
    y, dws, dx, g = column_ref(nodes, inp)
    bounds = [0, 0, 4, 4, 5, 17, 17, 30, 30]
    yr, strips = R.carry_forward(nodes, inp.x, inp.weights, inp.scales,
                                 inp.shifts, bounds)
    np.testing.assert_array_equal(yr, y)
    dwr, dxr = R.carry_backward(nodes, inp.x, inp.weights, inp.scales,
                                inp.shifts, g, bounds, strips)
    assert rel(dxr, dx) < 1e-12
    for a, b in zip(dwr, dws):
        if b is not None:
            assert rel(a, b) < 1e-12


@pytest.mark.parametrize("name", list(NETS))
@pytest.mark.parametrize("nb", [1, 2, 4, 7])
def test_recompute_partition_invariance(name, nb):
    nodes = NETS[name]
    h = 41
    inp = Inputs(nodes, 2, h, 10, 3, F32, seed=nb)
    y, dws, dx, g = column_ref(nodes, inp)
    hout = y.shape[1]
    ob = R.even_bounds(hout, min(nb, hout))
    yr = R.recompute_forward(nodes, inp.x, inp.weights, inp.scales,
                             inp.shifts, ob)
    np.testing.assert_array_equal(yr, y)
    dwr, dxr = R.recompute_backward(nodes, inp.x, inp.weights, inp.scales,
                                    inp.shifts, g, ob)
    assert rel(dxr, dx) < 1e-12
    for a, b in zip(dwr, dws):
        if b is not None:
            assert rel(a, b) < 1e-12


def test_config1_tiny_four_bands_of_eight_rows():
    nodes = tiny_net()
    inp = Inputs(nodes, 1, 32, 32, 3, F32, seed=1)
    y, dws, dx, g = column_ref(nodes, inp)
    bounds = [0, 8, 16, 24, 32]
    yr, strips = R.carry_forward(nodes, inp.x, inp.weights, inp.scales,
                                 inp.shifts, bounds)
    np.testing.assert_array_equal(yr, y)
    # each 3x3 stride-1 pad-1 layer shares k - s = 2 rows at every boundary
    # (the (k^l - s^l) term of Eq. (12)); the last layer keeps nothing
    for r in (1, 2, 3):
        for v in (0, 1, 2):
            assert strips[(r, v)].shape[1] == 2
        assert strips[(r, 3)].shape[1] == 0
    dwr, dxr = R.carry_backward(nodes, inp.x, inp.weights, inp.scales,
                                inp.shifts, g, bounds, strips)
    assert rel(dxr, dx) < 1e-12


def test_bf16_emulation_is_partition_invariant():
    nodes = NETS["resnet_like"]
    inp = Inputs(nodes, 1, 33, 9, 3, BF16, seed=4)
    y, dws, dx, g = column_ref(nodes, inp, bf16=True)
    bounds = [0, 9, 20, 33]
    yr, strips = R.carry_forward(nodes, inp.x, inp.weights, inp.scales,
                                 inp.shifts, bounds, bf16=True)
    np.testing.assert_array_equal(yr, y)
    dwr, dxr = R.carry_backward(nodes, inp.x, inp.weights, inp.scales,
                                inp.shifts, g, bounds, strips, bf16=True)
    # bf16 rounding of the error operand may land on either side of a tie
    # when the fp64 sums are ordered differently; gradients stay close
    assert rel(dxr, dx) < 1e-2
    for a, b in zip(dwr, dws):
        if b is not None:
            assert rel(a, b) < 1e-2


# ------------------------------------------------------ intervals vs brute
CHAINS = [
    [(3, 1, 1)] * 4,
    [(3, 1, 1), (2, 2, 0), (3, 1, 1), (2, 2, 0)],
    [(7, 2, 3), (3, 2, 1), (1, 1, 0), (3, 2, 1), (1, 2, 0)],
    [(5, 3, 1), (2, 1, 0), (4, 2, 2)],
]


def chain_nodes(ksp):
    nb = NetBuilder()
    v = 0
    for k, s, p in ksp:
        v = nb.conv(v, 1, k, s, p)
    return nb.nodes


@pytest.mark.parametrize("ksp", CHAINS)
def test_cones_equal_bruteforce_dependency_sets(ksp):
    nodes = chain_nodes(ksp)
    h = 53
    shp = C.shapes(nodes, h, 5, 1)
    hout = shp[-1][0]
    for nb in (1, 2, 3, 5):
        ob = R.even_bounds(hout, min(nb, hout))
        for r, (lo, hi) in enumerate(R.cone_intervals(nodes, shp, ob), 1):
            need = brute.dependency_rows(ksp, h, range(ob[r - 1], ob[r]))
            assert need == set(range(lo[0], hi[0])) or (not need and lo[0] == hi[0])


@pytest.mark.parametrize("ksp", CHAINS)
def test_carry_frontier_and_shared_rows_bruteforce(ksp):
    nodes = chain_nodes(ksp)
    h = 61
    shp = C.shapes(nodes, h, 5, 1)
    hout = shp[-1][0]
    rng = np.random.default_rng(0)
    for _ in range(5):
        bounds = random_bounds(rng, h, 4)
        F, T = R.carry_intervals(nodes, shp, bounds)
        for r in range(1, 5):
            # F: exactly the output rows whose full dependency set lies in
            # the input rows seen so far
            ok = [y for y in range(hout)
                  if brute.dependency_rows(ksp, h, [y]) <= set(range(bounds[r]))]
            assert F[r][-1] == len(ok) and ok == list(range(len(ok)))
            # T: every row of layer l that a later band reads was either
            # computed by that band or is held in [T, F)
            for li in range(len(ksp)):
                Fl = F[r][li]
                later = set()
                k, s, p = ksp[li]
                for y in range(F[r][li + 1], shp[li + 1][0]):
                    later |= {y * s - p + i for i in range(k)
                              if 0 <= y * s - p + i < shp[li][0]}
                needed_old = {q for q in later if q < Fl}
                assert needed_old <= set(range(T[r][li], Fl))
                if needed_old:
                    assert T[r][li] == min(needed_old)


def test_greedy_first_row_recursion_eqs_11_13_14():
    # Eq. (11): H_1^l = (H_1^{l+1} - 1) s + k - p gives the input rows band 1
    # needs for H_1^L rows of the last layer; Eq. (13) H_r^l = H_r^{l+1} s for
    # middle rows; Eq. (14) subtracts p for the last row. Feeding the inverted
    # heights back through the frontier gives the requested output rows.
    # (The recursions assume every layer divides exactly: (H + 2p - k) % s
    # == 0, which holds for this chain on an even height.)
    ksp = [(3, 1, 1)] * 3 + [(2, 2, 0), (3, 1, 1)]
    nodes = chain_nodes(ksp)
    h = 64
    shp = C.shapes(nodes, h, 4, 1)
    want = [5, 10, 7, shp[-1][0] - 22]

    def up(rows, first, last):
        for k, s, p in reversed(ksp):
            if first:
                rows = (rows - 1) * s + k - p
            elif last:
                rows = (rows - 1) * s + s - p
            else:
                rows = (rows - 1) * s + s
        return rows

    heights = [up(want[0], True, False), up(want[1], False, False),
               up(want[2], False, False)]
    bounds = [0, heights[0], heights[0] + heights[1],
              heights[0] + heights[1] + heights[2], h]
    assert up(want[3], False, True) == h - bounds[3]
    F, _ = R.carry_intervals(nodes, shp, bounds)
    got = [F[r][-1] - F[r - 1][-1] for r in range(1, 5)]
    assert got == want


def test_k3s1p1_row_recursions_special_case():
    # For 3x3 stride-1 pad-1 layers Eqs. (11), (13), (14) give
    # H_1^l = H_1^{l+1} + 1, H_r^l = H_r^{l+1}, H_N^l = H_N^{l+1} - 1.
    nodes = chain_nodes([(3, 1, 1)] * 6)
    h = 60
    shp = C.shapes(nodes, h, 3, 1)
    bounds = [0, 20, 40, 60]
    F, _ = R.carry_intervals(nodes, shp, bounds)
    for layer in range(1, 7):
        rows = [F[r][layer] - F[r - 1][layer] for r in (1, 2, 3)]
        assert rows == [20 - layer, 20, 20 + layer]


# ------------------------------------------------------ paper's examples
def test_feature_loss_example():
    ex = GOLD["feature_loss"]
    nb = NetBuilder()
    nb.conv(0, 1, ex["k"], ex["s"], ex["p"], relu=0)
    nodes = nb.nodes
    inp = Inputs(nodes, 1, *ex["input_hw"], 1, F32, seed=2)
    bounds = np.cumsum([0] + ex["band_rows"]).tolist()
    naive = R.independent_bands_forward(nodes, inp.x, inp.weights, inp.scales,
                                        inp.shifts, bounds)
    assert list(naive.shape[1:3]) == ex["naive_concat_output_hw"]
    y, _ = R.carry_forward(nodes, inp.x, inp.weights, inp.scales, inp.shifts,
                           bounds)
    col = C.forward(nodes, inp.x, inp.weights, inp.scales, inp.shifts)[0][-1]
    assert list(y.shape[1:3]) == ex["column_output_hw"]
    np.testing.assert_array_equal(y, col)
    # a second k=2 convolution cannot even run on one band's 1-row output
    assert ex["per_band_output_hw"][0] < ex["k"]


def test_padding_redundancy_changes_values():
    # Section III-B: zero padding at internal band edges keeps the height
    # for 3x3/p1 but changes values next to the edge (Fig. 2b)
    nodes = tiny_net()
    inp = Inputs(nodes, 1, 16, 8, 3, F32, seed=3)
    bounds = [0, 8, 16]
    naive = R.independent_bands_forward(nodes, inp.x, inp.weights, inp.scales,
                                        inp.shifts, bounds)
    col = C.forward(nodes, inp.x, inp.weights, inp.scales, inp.shifts)[0][-1]
    assert naive.shape == col.shape
    diff = np.abs(naive - col).max(axis=(0, 2, 3))
    assert diff[5:11].max() > 1e-3          # rows near the band edge differ
    assert diff[:4].max() == 0 and diff[12:].max() == 0  # far rows agree


def test_no_sharing_gives_wrong_gradients():
    # the "w/o sharing" branch of Section V-D: bands trained independently
    nodes = tiny_net()
    inp = Inputs(nodes, 1, 16, 8, 3, F32, seed=3)
    y, dws, dx, g = column_ref(nodes, inp)
    bounds = [0, 8, 16]
    tot = [None] * len(nodes)
    for r in (1, 2):
        xb = inp.x[:, bounds[r - 1]:bounds[r]]
        acts, am = C.forward(nodes, xb, inp.weights, inp.scales, inp.shifts)
        d, _ = C.backward(nodes, acts, am, inp.weights, inp.scales,
                          g[:, bounds[r - 1]:bounds[r]])
        tot = [a if t is None else (t if a is None else t + a)
               for t, a in zip(tot, d)]
    assert max(rel(a, b) for a, b in zip(tot, dws) if b is not None) > 1e-3


def test_two_phase_skew_example():
    ex = GOLD["two_phase_skew"]
    nb = NetBuilder()
    v = 0
    for _ in range(ex["layers"]):
        v = nb.conv(v, 1, ex["k"], ex["s"], ex["p"], relu=0)
    nodes = nb.nodes
    shp = C.shapes(nodes, *ex["input_hw"], 1)
    bounds = np.cumsum([0] + ex["band_rows"]).tolist()
    F, T = R.carry_intervals(nodes, shp, bounds)
    assert [F[r][1] - F[r - 1][1] for r in (1, 2)] == ex["layer1_band_rows"]
    assert [F[r][2] - F[r - 1][2] for r in (1, 2)] == ex["layer2_band_rows"]
    # R2 shares k - s = 1 row of the input and of z^1 with R1
    assert F[1][0] - T[1][0] == 1 and F[1][1] - T[1][1] == 1
    inp = Inputs(nodes, 1, *ex["input_hw"], 1, F32, seed=9)
    y, _ = R.carry_forward(nodes, inp.x, inp.weights, inp.scales, inp.shifts,
                           bounds)
    col = C.forward(nodes, inp.x, inp.weights, inp.scales, inp.shifts)[0][-1]
    np.testing.assert_array_equal(y, col)


def test_overlap_example():
    ex = GOLD["overlap"]
    nb = NetBuilder()
    nb.conv(0, 1, ex["k"], ex["s"], ex["p"], relu=0)
    nodes = nb.nodes
    shp = C.shapes(nodes, *ex["input_hw"], 1)
    assert shp[-1][0] == ex["output_rows"]
    ob = R.even_bounds(shp[-1][0], ex["bands"])
    (lo1, hi1), (lo2, hi2) = R.cone_intervals(nodes, shp, ob)
    shared = len(set(range(lo1[0], hi1[0])) & set(range(lo2[0], hi2[0])))
    assert shared >= ex["min_shared_input_rows"]
