"""The C-ABI library on the CPU: it loads, exports every function the header
declares, and its host-only planner agrees with the oracle's independent
interval arithmetic, shape rules, Eq. (3) memory and tau. No GPU calls."""
import os
import re

import numpy as np
import pytest

from oracle import column as OC, rows as OR
from paper_2401_11471_amd import lrcnn as L
from workloads import (NetBuilder, net_nodes, tiny_net, vgg16_net, resnet50_net,
                       CONFIGS)

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    names = set()
    inc = os.path.join(ROOT, "include")
    for f in sorted(os.listdir(inc)):
        if f.endswith(".h"):
            txt = open(os.path.join(inc, f)).read()
            txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
            names |= set(re.findall(r"\b(lrcnn_\w+)\s*\(", txt))
    return sorted(names)


def test_library_exports_every_declared_function():
    names = header_functions()
    assert set(names) == set(L.EXPORTS), names
    for nm in names:
        assert hasattr(L.LIB, nm), nm


def small_dag():
    nb = NetBuilder()
    a = nb.conv(0, 8, 7, 2, 3, affine=1)
    b = nb.pool(a, 3, 2, 1)
    c1 = nb.conv(b, 4, 1, 1, 0, affine=1)
    c2 = nb.conv(c1, 4, 3, 2, 1, affine=1)
    c3 = nb.conv(c2, 16, 1, 1, 0, affine=1, relu=0)
    sc = nb.conv(b, 16, 1, 2, 0, affine=1, relu=0)
    s = nb.sum(c3, sc)
    d1 = nb.conv(s, 4, 1, 1, 0, affine=1)
    d2 = nb.conv(d1, 4, 3, 1, 1, affine=1)
    d3 = nb.conv(d2, 16, 1, 1, 0, affine=1, relu=0)
    nb.sum(d3, s)
    return nb.nodes


def odd_chain():
    nb = NetBuilder()
    v = nb.conv(0, 5, 5, 2, 2)
    v = nb.conv(v, 6, 2, 1, 0)
    v = nb.pool(v, 3, 2, 1)
    v = nb.conv(v, 3, 4, 3, 1)
    nb.conv(v, 7, 1, 1, 0)
    return nb.nodes


NETS = {"tiny": tiny_net(), "vgg16": vgg16_net(), "resnet50": resnet50_net(),
        "dag": small_dag(), "odd": odd_chain()}


@pytest.mark.parametrize("name", list(NETS))
def test_shapes_match_oracle(name):
    nodes = NETS[name]
    h, w = (224, 200) if name in ("vgg16", "resnet50") else (61, 37)
    p = L.lrcnn_plan(nodes, 2, 3, h, w)
    shp = OC.shapes(nodes, h, w, 3)
    for v in range(len(nodes)):
        assert p.node_shape(v) == shp[v]


@pytest.mark.parametrize("name", list(NETS))
@pytest.mark.parametrize("seed", range(3))
def test_carry_intervals_match_oracle(name, seed):
    nodes = NETS[name]
    h, w = (224, 64) if name in ("vgg16", "resnet50") else (61, 9)
    rng = np.random.default_rng(seed)
    nb = [1, 4, 7][seed]
    cuts = sorted(rng.integers(0, h + 1, nb - 1).tolist())
    bounds = [0] + cuts + [h]
    p = L.lrcnn_plan(nodes, 1, 3, h, w, L.F32, L.CARRY, nb, L.EXPLICIT, bounds)
    F, T = OR.carry_intervals(nodes, OC.shapes(nodes, h, w, 3), bounds)
    for r in range(nb):
        for v in range(len(nodes)):
            assert p.band_rows(r, v) == (F[r][v], F[r + 1][v], T[r][v], F[r + 1][v])


@pytest.mark.parametrize("name", list(NETS))
@pytest.mark.parametrize("nb", [1, 3, 8])
def test_cone_intervals_match_oracle(name, nb):
    nodes = NETS[name]
    h, w = (224, 64) if name in ("vgg16", "resnet50") else (61, 9)
    shp = OC.shapes(nodes, h, w, 3)
    p = L.lrcnn_plan(nodes, 1, 3, h, w, L.F32, L.RECOMPUTE, nb)
    ob = OR.even_bounds(shp[-1][0], nb)
    for r, (lo, hi) in enumerate(OR.cone_intervals(nodes, shp, ob)):
        for v in range(len(nodes)):
            assert p.band_rows(r, v) == (lo[v], hi[v], lo[v], hi[v])


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_tau_and_omega(cid):
    c = CONFIGS[cid]
    nodes = net_nodes(c["net"])
    p = L.lrcnn_plan(nodes, c["batch"], 3, c["h"], c["w"], c["dtype"], L.CARRY, c["bands"])
    info = p.info()
    tau = OC.flops_forward(nodes, c["batch"], c["h"], c["w"], 3)
    assert info["flops_tau"] == tau
    # 2PS costs 4 tau (Section IV-B); the last band's BP recompute is
    # skipped because FP leaves its maps in place
    shp = OC.shapes(nodes, c["h"], c["w"], 3)
    F, _ = OR.carry_intervals(nodes, shp, OR.even_bounds(c["h"], c["bands"]))
    last = sum(2 * nd[4] * nd[5] * c["batch"] * shp[nd[1]][2] * nd[3] * shp[v][1] *
               (F[-1][v] - F[-2][v]) for v, nd in enumerate(nodes) if nd[0] == 1)
    assert info["flops_rows"] == 4 * tau - last
    assert info["flops_layerwise"] == 3 * tau
    es = 2 if c["dtype"] == L.BF16 else 4
    shp = OC.shapes(nodes, c["h"], c["w"], 3)
    omega = sum(c["batch"] * h * w * ch * es for (h, w, ch) in shp[1:])  # Eq. (3)
    assert info["omega_bytes"] == omega


def test_tau_per_image_published_scale():
    # tau for VGG-16 at 224x224 is the well-known ~15.5 GMAC per image
    p = L.lrcnn_plan(vgg16_net(), 1, 3, 224, 224)
    assert abs(p.info()["flops_tau"] / 2 / 1e9 - 15.35) < 0.2


def test_recompute_flops_include_overlap():
    nodes = vgg16_net()
    p1 = L.lrcnn_plan(nodes, 1, 3, 224, 224, L.F32, L.RECOMPUTE, 1)
    p4 = L.lrcnn_plan(nodes, 1, 3, 224, 224, L.F32, L.RECOMPUTE, 4)
    i1, i4 = p1.info(), p4.info()
    # one band: FP + input and weight gradients, its maps kept for BP
    assert i1["flops_rows"] == 3 * i1["flops_tau"] and i1["halo_rows"] == 0
    # four bands: 4(tau + iota) less the kept last band's recompute
    assert i4["flops_rows"] > 3.5 * i4["flops_tau"] and i4["halo_rows"] > 0


def test_shared_rows_eq12_term():
    # 3x3 stride-1 pad-1 layers: every boundary keeps k - s = 2 rows of every
    # layer feeding a conv (Eq. (12)); the last layer keeps none
    nodes = tiny_net()
    p = L.lrcnn_plan(nodes, 1, 3, 32, 32, L.F32, L.CARRY, 4)
    for r in range(3):
        for v in range(4):
            a, b, lo, hi = p.band_rows(r + 1, v)
            assert a - lo == (2 if v < 3 else 0)
    assert p.info()["shared_rows"] == 3 * 3 * 2


def test_balanced_policy_cuts_the_workspace():
    nodes = resnet50_net()
    ev = L.lrcnn_plan(nodes, 16, 3, 224, 224, L.BF16, L.CARRY, 4, L.EVEN).info()
    ba = L.lrcnn_plan(nodes, 16, 3, 224, 224, L.BF16, L.CARRY, 4, L.BALANCED)
    assert ba.info()["workspace_bytes"] < ev["workspace_bytes"]
    rows = [ba.band_rows(r, 0) for r in range(4)]
    assert rows[0][0] == 0 and rows[-1][1] == 224
    assert all(rows[i][1] == rows[i + 1][0] for i in range(3))


def test_plan_errors():
    good = tiny_net()
    with pytest.raises(L.LrcnnError) as e:
        L.lrcnn_plan(good, 1, 3, 32, 32, L.F32, L.CARRY, 0)
    assert e.value.code == -3
    with pytest.raises(L.LrcnnError) as e:
        L.lrcnn_plan(good, 1, 3, 32, 32, L.F32, L.CARRY, 2, L.EXPLICIT, [0, 20, 10])
    assert e.value.code == -3
    with pytest.raises(L.LrcnnError) as e:
        L.lrcnn_plan(good, 1, 3, 32, 32, L.F32, L.CARRY, 2, L.EXPLICIT, [0, 10, 31])
    assert e.value.code == -3
    with pytest.raises(L.LrcnnError) as e:
        L.lrcnn_plan(good, 1, 3, 32, 32, 7, L.CARRY, 2)
    assert e.value.code == -6
    with pytest.raises(L.LrcnnError) as e:
        L.lrcnn_plan(good, 1, 3, 32, 32, L.F32, L.RECOMPUTE, 2, L.BALANCED)
    assert e.value.code == -1
    bad = list(good)
    bad[2] = (1, 5, -1, 8, 3, 3, 1, 1, 1, 1, 0, 1)  # in0 names a later node
    with pytest.raises(L.LrcnnError) as e:
        L.lrcnn_plan(bad, 1, 3, 32, 32)
    assert e.value.code == -2
    with pytest.raises(L.LrcnnError) as e:       # 7x7 window on a 4x4 image
        L.lrcnn_plan([(0,) + (-1,) * 11, (1, 0, -1, 4, 7, 7, 1, 1, 0, 0, 0, 1)],
                     1, 3, 4, 4)
    assert e.value.code == -2
    nb = NetBuilder()
    a = nb.conv(0, 4, 3, 1, 1)
    b = nb.conv(0, 5, 3, 1, 1)
    nb.sum(a, b)                                  # channel mismatch
    with pytest.raises(L.LrcnnError) as e:
        L.lrcnn_plan(nb.nodes, 1, 3, 8, 8)
    assert e.value.code == -2
    nb = NetBuilder()
    nb.conv(0, 4, 3, 1, 1)
    nb.conv(0, 4, 3, 1, 1)                        # node 1 feeds nothing
    with pytest.raises(L.LrcnnError) as e:
        L.lrcnn_plan(nb.nodes, 1, 3, 8, 8)
    assert e.value.code == -2


def test_entry_points_reject_bad_arguments_before_any_launch():
    # every check below happens on the host before the library touches HIP
    import ctypes as C
    nodes = tiny_net()
    p = L.lrcnn_plan(nodes, 1, 3, 32, 32, L.F32, L.CARRY, 4)
    need = p.info()["workspace_bytes"]
    fake = 1 << 20  # an aligned non-null address that is never dereferenced
    ptrs = (C.c_void_p * 4)(None, fake, fake, fake)
    nulls = (C.c_void_p * 4)()
    st = L.LIB.lrcnn_forward_rows(p.handle, None, ptrs, nulls, nulls, fake, fake,
                                  need, None, None)
    assert st == -1                                # x is null
    st = L.LIB.lrcnn_forward_rows(p.handle, fake + 4, ptrs, nulls, nulls, fake, fake,
                                  need, None, None)
    assert st == -1                                # misaligned
    st = L.LIB.lrcnn_forward_rows(p.handle, fake, ptrs, nulls, nulls, fake, fake,
                                  need - 1, None, None)
    assert st == -4                                # workspace too small
    dws = (C.c_void_p * 4)(None, fake, fake, fake)
    st = L.LIB.lrcnn_backward_rows(p.handle, fake, ptrs, nulls, nulls, fake, dws,
                                   None, fake, need, None)
    assert st == -5                                # CARRY BP before FP
    assert b"forward" in L.LIB.lrcnn_last_error()
    nb = NetBuilder()
    nb.conv(0, 4, 3, 1, 1, affine=1)
    pa = L.lrcnn_plan(nb.nodes, 1, 3, 8, 8)
    pw = (C.c_void_p * 2)(None, fake)
    st = L.LIB.lrcnn_forward_rows(pa.handle, fake, pw, (C.c_void_p * 2)(),
                                  (C.c_void_p * 2)(), fake, fake, 1 << 30, None, None)
    assert st == -1                                # affine without scale/shift


class _Fake:
    """Stands in for a device tensor in dry runs: an aligned address that the
    library never dereferences."""

    def __init__(self, addr, n=1 << 40):
        self.addr, self.n = addr, n

    def data_ptr(self):
        return self.addr

    def numel(self):
        return self.n


def dry_run(nodes, batch, h, w, dtype, mode, nb, policy=L.EVEN, bounds=None,
            dx=True, bp_refine=1, hybrid_from=0):
    p = L.lrcnn_plan(nodes, batch, 3, h, w, dtype, mode, nb, policy, bounds, bp_refine,
                     hybrid_from)
    f = _Fake(1 << 30)
    per = [None] + [f if nd[0] == L.OP_CONV else None for nd in nodes[1:]]
    aff = [None] + [f if (nd[0] == L.OP_CONV and nd[10]) else None for nd in nodes[1:]]
    masks = [None] + [f] * (len(nodes) - 1)
    L.lrcnn_debug_dry_run(True)
    try:
        L.lrcnn_forward_rows(p, f, per, aff, aff, f, f, masks, stream=0)
        L.lrcnn_backward_rows(p, f, per, aff, aff, f, per, f if dx else None, f, stream=0)
        L.lrcnn_layerwise_reference_gpu(p, f, per, aff, aff, f, f, per,
                                        f if dx else None, f, masks, stream=0)
    finally:
        L.lrcnn_debug_dry_run(False)
    return p


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
@pytest.mark.parametrize("mode", ["carry", "balanced", "recompute"])
@pytest.mark.parametrize("refine", [1, 2, 3])
def test_executor_dry_run_configs(cid, mode, refine):
    c = CONFIGS[cid]
    m = L.RECOMPUTE if mode == "recompute" else L.CARRY
    pol = L.BALANCED if mode == "balanced" else L.EVEN
    dry_run(net_nodes(c["net"]), c["batch"], c["h"], c["w"], c["dtype"], m,
            c["bands"], pol, bp_refine=refine)


@pytest.mark.parametrize("name", list(NETS))
@pytest.mark.parametrize("seed", range(4))
def test_executor_dry_run_random_partitions(name, seed):
    nodes = NETS[name]
    h, w = (224, 64) if name in ("vgg16", "resnet50") else (61, 9)
    rng = np.random.default_rng(50 + seed)
    nb = int(rng.integers(1, 9))
    cuts = sorted(rng.integers(0, h + 1, nb - 1).tolist())
    dry_run(nodes, 2, h, w, L.F32, L.CARRY, nb, L.EXPLICIT, [0] + cuts + [h],
            dx=bool(seed % 2), bp_refine=1 + seed % 3)
    dry_run(nodes, 2, h, w, L.BF16, L.RECOMPUTE, nb, dx=bool(seed % 2),
            bp_refine=1 + (seed + 1) % 3)


@pytest.mark.parametrize("refine", [2, 3])
def test_backward_partition_refines_forward(refine):
    # Section III-C: BP may use a finer partition than FP. Each forward band
    # is split evenly; frontiers of both partitions agree at shared
    # boundaries, and the plan's rows match the oracle's intervals for each.
    nodes = NETS["dag"]
    h, w = 61, 9
    bounds = [0, 7, 30, 61]
    p = L.lrcnn_plan(nodes, 1, 3, h, w, L.F32, L.CARRY, 3, L.EXPLICIT, bounds, refine)
    inf = p.info()
    assert inf["n_bands"] == 3 and inf["bp_bands"] == 3 * refine
    shp = OC.shapes(nodes, h, w, 3)
    bb = []
    for r in range(3):
        for j in range(refine):
            bb.append(bounds[r] + (bounds[r + 1] - bounds[r]) * j // refine)
    bb.append(h)
    Ff, Tf = OR.carry_intervals(nodes, shp, bounds)
    Fb, Tb = OR.carry_intervals(nodes, shp, bb)
    for v in range(len(nodes)):
        for r in range(3):
            assert p.band_rows(r, v, phase=0) == (Ff[r][v], Ff[r + 1][v], Tf[r][v], Ff[r + 1][v])
        for q in range(3 * refine):
            assert p.band_rows(q, v, phase=1) == (Fb[q][v], Fb[q + 1][v], Tb[q][v], Fb[q + 1][v])
        for r in range(1, 3):
            assert Fb[r * refine][v] == Ff[r][v] and Tb[r * refine][v] == Tf[r][v]


def test_finer_backward_bands_cut_memory_on_vgg():
    c = CONFIGS[2]
    nodes = net_nodes("vgg16")
    one = L.lrcnn_plan(nodes, 8, 3, 224, 224, L.F32, L.CARRY, 4).info()
    two = L.lrcnn_plan(nodes, 8, 3, 224, 224, L.F32, L.CARRY, 4, bp_refine=2).info()
    assert two["workspace_bytes"] < one["workspace_bytes"]
    assert two["band_cache_bytes"] < one["band_cache_bytes"]
    assert two["layerwise_workspace_bytes"] > 3 * two["workspace_bytes"]


def _cuts(nodes):
    n = len(nodes)
    return [k for k in range(2, n)
            if all(nodes[v][1] >= k - 1 and (nodes[v][0] != L.OP_ADD or nodes[v][2] >= k - 1)
                   for v in range(k, n))]


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
@pytest.mark.parametrize("mode", ["carry", "recompute"])
def test_hybrid_depth_dry_run(cid, mode):
    # every valid checkpoint of every workload plans and runs through the
    # executor's host checks; the workspace is at most the row part's plus
    # the layer-wise part's and the checkpoint's
    c = CONFIGS[cid]
    nodes = net_nodes(c["net"])
    m = L.RECOMPUTE if mode == "recompute" else L.CARRY
    cuts = _cuts(nodes)
    assert cuts
    for k in cuts[:: max(1, len(cuts) // 4)]:
        p = dry_run(nodes, c["batch"], c["h"], c["w"], c["dtype"], m, c["bands"], hybrid_from=k)
        info = p.info()
        rp = L.lrcnn_plan(nodes[:k], c["batch"], 3, c["h"], c["w"], c["dtype"], m, c["bands"])
        assert info["workspace_bytes"] >= rp.info()["workspace_bytes"]
        # layer-wise nodes are whole in band 0 and empty after it
        a, b, lo, hi = p.band_rows(0, len(nodes) - 1)
        assert (a, b) == (0, p.node_shape(len(nodes) - 1)[0])
        if info["n_bands"] > 1:
            assert p.band_rows(1, len(nodes) - 1)[:2] == (0, 0)
        # the row part's nodes keep the row part's bands
        assert p.band_rows(0, k - 1) == rp.band_rows(0, k - 1)


def test_hybrid_depth_errors():
    nodes = resnet50_net()
    good = set(_cuts(nodes))
    bad = next(k for k in range(2, len(nodes)) if k not in good)
    for k in (1, -2, len(nodes), bad):
        with pytest.raises(L.LrcnnError) as e:
            L.lrcnn_plan(nodes, 2, 3, 64, 64, L.F32, L.CARRY, 2, hybrid_from=k)
        assert "EINVAL" in str(e.value)


def test_hybrid_cuts_vgg_flops_and_memory():
    # a checkpoint after pool3 runs conv4/conv5 layer-wise: less recompute
    # than the all-row-centric plan, and a smaller workspace at 4 bands
    c = CONFIGS[2]
    nodes = vgg16_net()
    full = L.lrcnn_plan(nodes, c["batch"], 3, c["h"], c["w"], c["dtype"], L.CARRY, 4).info()
    hy = L.lrcnn_plan(nodes, c["batch"], 3, c["h"], c["w"], c["dtype"], L.CARRY, 4,
                      hybrid_from=11).info()
    assert hy["flops_rows"] < full["flops_rows"]
    assert hy["workspace_bytes"] < full["workspace_bytes"]
    assert hy["flops_layerwise"] == full["flops_layerwise"]


@pytest.mark.parametrize("cid", [2, 3, 5])
def test_hybrid_auto_picks_the_smallest_workspace(cid):
    # budget-driven placement: the planner's checkpoint is a valid cut whose
    # workspace is the minimum over every cut and the all-row-centric plan
    c = CONFIGS[cid]
    nodes = net_nodes(c["net"])
    args = (nodes, c["batch"], 3, c["h"], c["w"], c["dtype"], L.CARRY, c["bands"])
    auto = L.lrcnn_plan(*args, hybrid_from=L.HYBRID_AUTO).info()
    sizes = {0: L.lrcnn_plan(*args).info()["workspace_bytes"]}
    for k in _cuts(nodes):
        sizes[k] = L.lrcnn_plan(*args, hybrid_from=k).info()["workspace_bytes"]
    assert auto["hybrid_from"] in sizes
    assert auto["workspace_bytes"] == min(sizes.values())
    assert auto["workspace_bytes"] == sizes[auto["hybrid_from"]]


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_executor_dry_run_pipelined_forward(cid):
    # the opt-in pipelined forward walks the same host checks (windows,
    # strips, carried rows) with its per-node waits and records
    c = CONFIGS[cid]
    L.lrcnn_debug_fp_pipeline(True)
    try:
        dry_run(net_nodes(c["net"]), c["batch"], c["h"], c["w"], c["dtype"], L.CARRY,
                c["bands"])
    finally:
        L.lrcnn_debug_fp_pipeline(False)
