"""Forward pass pipelined over bands (opt-in; consecutive bands on two streams, each
step waiting until the previous band no longer reads the windows it writes;
the second stream's split-K partial sums in the idle backward arena) against
the bands one after another: the same launches, so the output, the masks
and the following backward are bitwise equal; the sequential forward is
pinned against the oracle by the parity tests."""
import numpy as np
import pytest

from gpu_harness import gpu_run
from paper_2401_11471_amd import lrcnn as L
from workloads import BF16, F32, Inputs, resnet50_net, tiny_net, vgg16_net

pytestmark = pytest.mark.gpu


def _run(nodes, inp, on, **kw):
    L.lrcnn_debug_fp_pipeline(on)
    try:
        return gpu_run(nodes, inp, **kw)
    finally:
        L.lrcnn_debug_fp_pipeline(False)


CASES = [
    ("tiny_f32_carry4", tiny_net, F32, 2, 32, 32, dict(mode=L.CARRY, nb=4)),
    ("vgg16_f32_carry4", vgg16_net, F32, 2, 96, 64, dict(mode=L.CARRY, nb=4)),
    ("vgg16_f32_carry7", vgg16_net, F32, 1, 224, 32, dict(mode=L.CARRY, nb=7)),
    ("resnet50_bf16_carry5", resnet50_net, BF16, 2, 160, 64, dict(mode=L.CARRY, nb=5)),
    ("resnet50_f32_carry3", resnet50_net, F32, 1, 96, 96, dict(mode=L.CARRY, nb=3)),
]


@pytest.mark.parametrize("name,net,dt,b,h,w,kw", CASES, ids=[c[0] for c in CASES])
def test_pipelined_forward_bitwise(name, net, dt, b, h, w, kw):
    print(f"forward pipeline {name}", flush=True)
    nodes = net()
    inp = Inputs(nodes, b, h, w, 3, dt, seed=41)
    pp = _run(nodes, inp, True, want_dx=True, repeat_bwd=2, **kw)
    sq = _run(nodes, inp, False, want_dx=True, **kw)
    for k in ("y", "dx"):
        assert np.array_equal(pp[k], sq[k]), k
    for v, (p, q) in enumerate(zip(pp["dw"], sq["dw"])):
        if p is not None:
            assert np.array_equal(p, q), v
    for v, m in sq["masks"].items():
        assert np.array_equal(pp["masks"][v], m), v
