"""Band placement policies of the planner on the CPU (host-only calls).

* PAPER_2PS, the greedy partition of two-phase sharing (Section IV-A): on a
  chain of layers that divide exactly, the band heights the planner gives
  are the ones Eq. (11) (first band), Eq. (13) (middle bands) and Eq. (14)
  (last band) give, recomputed here by inverting the layers; on DAGs every
  band end is the smallest input row count whose last-node frontier (from
  the oracle's own interval code) reaches the band's target.
* BALANCED never lays out a larger workspace than the even split.
* The layer-wise baseline's workspace is the same whatever the row
  partition (policy, band count, backward refinement, mode).
* The budget search with PAPER_2PS (Eq. (12): fewest backward bands, then
  the largest first band) agrees with a brute-force scan.
"""
import pytest

from oracle import column as OC, rows as OR
from paper_2401_11471_amd import lrcnn as L
from workloads import CONFIGS, NetBuilder, net_nodes, resnet50_net, vgg16_net


def chain(ksp):
    nb = NetBuilder()
    v = 0
    for k, s, p in ksp:
        v = nb.conv(v, 2, k, s, p)
    return nb.nodes


def paper_heights(ksp, rows, kind):
    """Input rows of a band with `rows` rows at the last layer, inverting
    the layers from the last one: Eq. (11) for the first band, Eq. (13) for
    a middle band, Eq. (14) for the last."""
    for k, s, p in reversed(ksp):
        if kind == "first":
            rows = (rows - 1) * s + k - p
        elif kind == "last":
            rows = (rows - 1) * s + s - p
        else:
            rows = (rows - 1) * s + s
    return rows


@pytest.mark.parametrize("first", [0, 3, 6])
def test_paper_2ps_chain_follows_eqs_11_13_14(first):
    ksp = [(3, 1, 1)] * 3 + [(2, 2, 0), (3, 1, 1), (3, 1, 1)]
    nodes = chain(ksp)
    H = 96
    shp = OC.shapes(nodes, H, 5, 1)
    HL = shp[-1][0]
    nb = 4
    p = L.lrcnn_plan(nodes, 1, 1, H, 5, L.F32, L.CARRY, nb, L.PAPER_2PS, first_rows=first)
    h1 = first if first else -(-HL // nb)
    t = [h1 + (r - 1) * (HL - h1) // (nb - 1) for r in range(1, nb)]
    want = [0, paper_heights(ksp, t[0], "first")]
    for r in range(1, nb - 1):
        want.append(want[-1] + paper_heights(ksp, t[r] - t[r - 1], "middle"))
    want.append(H)
    # the last band: Eq. (14) inverts its own output rows to what is left
    assert paper_heights(ksp, HL - t[-1], "last") == H - want[-2]
    got = [p.band_rows(r, 0, phase=1)[0] for r in range(nb)] + [H]
    assert got == want
    F, _ = OR.carry_intervals(nodes, shp, got)
    assert [F[r][-1] for r in range(1, nb)] == t


@pytest.mark.parametrize("net,h,nb,first", [("resnet50", 224, 8, 0), ("resnet50", 320, 5, 4),
                                            ("vgg16", 224, 4, 0), ("vgg16", 250, 3, 2)])
def test_paper_2ps_bounds_are_smallest_inputs_reaching_targets(net, h, nb, first):
    nodes = net_nodes(net)
    shp = OC.shapes(nodes, h, 32, 3)
    HL = shp[-1][0]
    p = L.lrcnn_plan(nodes, 1, 3, h, 32, L.F32, L.CARRY, nb, L.PAPER_2PS, first_rows=first)
    bounds = [p.band_rows(r, 0, phase=1)[0] for r in range(nb)] + [h]
    h1 = min(first, HL) if first else -(-HL // nb)
    for r in range(1, nb):
        t = h1 + (r - 1) * (HL - h1) // (nb - 1)
        F, _ = OR.carry_intervals(nodes, shp, [0, bounds[r], h])
        assert F[1][-1] >= t
        if bounds[r] > bounds[r - 1]:
            F, _ = OR.carry_intervals(nodes, shp, [0, bounds[r] - 1, h])
            assert F[1][-1] < t


def test_paper_2ps_forward_bands_are_every_refine_th_backward_band():
    nodes = vgg16_net()
    p = L.lrcnn_plan(nodes, 1, 3, 224, 32, L.F32, L.CARRY, 2, L.PAPER_2PS, bp_refine=3)
    bp = [p.band_rows(r, 0, phase=1)[0] for r in range(6)] + [224]
    fp = [p.band_rows(r, 0, phase=0)[0] for r in range(2)] + [224]
    assert fp == bp[::3]


def test_paper_2ps_needs_carry_mode():
    with pytest.raises(L.LrcnnError):
        L.lrcnn_plan(vgg16_net(), 1, 3, 224, 32, L.F32, L.RECOMPUTE, 2, L.PAPER_2PS)


@pytest.mark.parametrize("cid", [2, 3])
def test_balanced_never_larger_than_even(cid):
    c = CONFIGS[cid]
    nodes = net_nodes(c["net"])
    for nb in (2, c["bands"]):
        for rf in (1, 2):
            ev = L.lrcnn_plan(nodes, c["batch"], 3, c["h"], c["w"], c["dtype"], L.CARRY, nb,
                              L.EVEN, bp_refine=rf).info()
            ba = L.lrcnn_plan(nodes, c["batch"], 3, c["h"], c["w"], c["dtype"], L.CARRY, nb,
                              L.BALANCED, bp_refine=rf)
            assert ba.info()["workspace_bytes"] <= ev["workspace_bytes"]
            rows = [ba.band_rows(r, 0, phase=0) for r in range(nb)]
            assert rows[0][0] == 0 and rows[-1][1] == c["h"]
            assert all(rows[i][1] == rows[i + 1][0] for i in range(nb - 1))


@pytest.mark.parametrize("cid", [2, 3, 5])
def test_layerwise_workspace_independent_of_partition(cid):
    c = CONFIGS[cid]
    nodes = net_nodes(c["net"])
    sizes = set()
    cases = [(L.CARRY, L.EVEN, c["bands"], 1, None), (L.CARRY, L.EVEN, 2, 3, None),
             (L.CARRY, L.PAPER_2PS, c["bands"], 1, None), (L.RECOMPUTE, L.EVEN, 3, 1, None),
             (L.CARRY, L.EXPLICIT, 3, 1, [0, c["h"] // 5, c["h"] // 2, c["h"]])]
    if cid != 5:
        cases.append((L.CARRY, L.BALANCED, c["bands"], 2, None))
    for mode, pol, nb, rf, bounds in cases:
        p = L.lrcnn_plan(nodes, c["batch"], 3, c["h"], c["w"], c["dtype"], mode, nb, pol,
                         bounds, rf)
        sizes.add(p.info()["layerwise_workspace_bytes"])
    assert len(sizes) == 1, sizes


def test_budget_search_paper_2ps_matches_brute_force():
    nodes = vgg16_net()
    B, H, W = 2, 160, 48
    HL = OC.shapes(nodes, H, W, 3)[-1][0]
    sizes = {}
    for nbp in range(1, 6):
        # the search's range of H_1^L: all rows down to an even share
        for h1 in range(HL, -(-HL // nbp) - 1, -1):
            p = L.lrcnn_plan(nodes, B, 3, H, W, L.F32, L.CARRY, nbp, L.PAPER_2PS,
                             first_rows=h1)
            sizes[nbp, h1] = p.step_bytes()
    lo, hi = min(sizes.values()), max(sizes.values())
    for M in (hi, (lo + hi) // 2, lo + (hi - lo) // 5, lo):
        want = None
        for nbp in range(1, 6):
            h_lo = 1 if nbp == 1 else -(-HL // nbp)
            cands = [HL] if nbp == 1 else range(HL, h_lo - 1, -1)
            for h1 in cands:
                s = sizes[nbp, h1 if nbp > 1 else HL]
                if s <= M:
                    want = (nbp, s)
                    break
            if want:
                break
        p = L.lrcnn_plan_for_budget(nodes, B, 3, H, W, M, policy=L.PAPER_2PS, max_bands=5)
        assert (p.info()["bp_bands"], p.step_bytes()) == want
