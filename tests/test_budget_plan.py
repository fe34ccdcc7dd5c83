"""Budget-driven planning on the CPU (host-only planner calls).

* lrcnn_plan_step_bytes = workspace + xi, with xi (Eqs. (9)-(10): every
  other buffer of the step) recomputed here from the node shapes.
* lrcnn_plan_for_budget returns the first (N_BP, N_FP) in increasing order
  whose step fits, checked against a brute-force scan of lrcnn_plan.
* lrcnn_max_batch returns B with step(B) <= M < step(B + 1).
"""
import pytest

from paper_2401_11471_amd import lrcnn as L
from workloads import net_nodes, tiny_net, vgg16_net


def a256(x):
    return (x + 255) // 256 * 256


def xi_bytes(nodes, plan, batch, h, w, c, es, want_dx):
    oh, ow, oc = plan.node_shape(len(nodes) - 1)
    xb = batch * h * w * c * es
    yb = batch * oh * ow * oc * es
    t = a256(xb) + 2 * a256(yb) + (a256(xb) if want_dx else 0)
    for v, nd in enumerate(nodes):
        if v == 0 or nd[0] != L.OP_CONV:
            continue
        ci = plan.node_shape(nd[1])[2]
        n = nd[3] * nd[4] * nd[5] * ci
        t += a256(n * es) + a256(n * 4)
        if nd[10]:
            t += 2 * a256(nd[3] * 4)
    return t


@pytest.mark.parametrize("dtype", [L.F32, L.BF16])
@pytest.mark.parametrize("want_dx", [False, True])
def test_step_bytes_is_workspace_plus_xi(dtype, want_dx):
    for name, (B, H, W) in {"vgg16": (2, 64, 48), "resnet50": (3, 96, 64),
                            "tiny": (1, 32, 32)}.items():
        nodes = net_nodes(name)
        es = 2 if dtype == L.BF16 else 4
        p = L.lrcnn_plan(nodes, B, 3, H, W, dtype, L.CARRY, 4)
        inf = p.info()
        xi = xi_bytes(nodes, p, B, H, W, 3, es, want_dx)
        assert p.step_bytes(False, want_dx) == inf["workspace_bytes"] + xi
        assert p.step_bytes(True, want_dx) == inf["layerwise_workspace_bytes"] + xi


def brute_first_fit(nodes, B, H, W, M, dtype, mode, max_bands, max_refine):
    for nbp in range(1, max_bands + 1):
        for nfp in range(1, nbp + 1):
            if nbp % nfp or nbp // nfp > max_refine:
                continue
            p = L.lrcnn_plan(nodes, B, 3, H, W, dtype, mode, nfp, bp_refine=nbp // nfp)
            if p.step_bytes() <= M:
                return nbp, nfp, p.step_bytes()
    return None


@pytest.mark.parametrize("mode", [L.CARRY, L.RECOMPUTE])
@pytest.mark.parametrize("max_refine", [1, 3])
def test_plan_for_budget_is_the_first_fit(mode, max_refine):
    nodes = vgg16_net()
    B, H, W = 2, 96, 64
    one = L.lrcnn_plan(nodes, B, 3, H, W, L.F32, mode, 1).step_bytes()
    for frac in (1.0, 0.8, 0.6, 0.5, 0.45):
        M = int(one * frac)
        ref = brute_first_fit(nodes, B, H, W, M, L.F32, mode, 12, max_refine)
        if ref is None:
            with pytest.raises(L.LrcnnError) as e:
                L.lrcnn_plan_for_budget(nodes, B, 3, H, W, M, L.F32, mode, max_bands=12,
                                        max_refine=max_refine)
            assert e.value.code == -8
            continue
        p = L.lrcnn_plan_for_budget(nodes, B, 3, H, W, M, L.F32, mode, max_bands=12,
                                    max_refine=max_refine)
        inf = p.info()
        assert (inf["bp_bands"], inf["n_bands"]) == ref[:2], (frac, ref)
        assert p.step_bytes() == ref[2] <= M


def test_plan_for_budget_prefers_one_band_and_reports_infeasible():
    nodes = tiny_net()
    p = L.lrcnn_plan_for_budget(nodes, 1, 3, 32, 32, 1 << 40)
    assert p.info()["n_bands"] == 1 and p.info()["bp_bands"] == 1
    with pytest.raises(L.LrcnnError) as e:
        L.lrcnn_plan_for_budget(nodes, 1, 3, 32, 32, 1000)
    assert e.value.code == -8
    with pytest.raises(L.LrcnnError) as e:
        L.lrcnn_plan_for_budget(nodes, 1, 3, 32, 32, 1 << 30, policy=L.EXPLICIT)
    assert e.value.code == -1


@pytest.mark.parametrize("layerwise", [False, True])
def test_max_batch_is_the_largest_fitting_batch(layerwise):
    nodes = vgg16_net()
    H, W, nb = 128, 96, 4
    for M in (300e6, 1.5e9, 7e9):
        B = L.lrcnn_max_batch(nodes, 3, H, W, M, L.F32, L.CARRY, nb, layerwise=layerwise)
        fits = L.lrcnn_plan(nodes, B, 3, H, W, L.F32, L.CARRY, nb).step_bytes(layerwise)
        over = L.lrcnn_plan(nodes, B + 1, 3, H, W, L.F32, L.CARRY, nb).step_bytes(layerwise)
        assert fits <= M < over, (M, B)


def test_max_batch_row_centric_exceeds_layerwise_and_infeasible_budget():
    nodes = net_nodes("resnet50")
    M = 20e9
    lw = L.lrcnn_max_batch(nodes, 3, 600, 900, M, L.BF16, L.CARRY, 8, layerwise=True)
    rc = L.lrcnn_max_batch(nodes, 3, 600, 900, M, L.BF16, L.CARRY, 8)
    assert rc > 2 * lw >= 2
    with pytest.raises(L.LrcnnError) as e:
        L.lrcnn_max_batch(nodes, 3, 600, 900, 1e6, L.BF16, L.CARRY, 8)
    assert e.value.code == -8
