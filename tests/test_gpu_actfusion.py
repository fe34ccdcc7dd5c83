"""Error operands formed by the input gradient of a convolution's only
consumer (the error window of the convolution is never written) against
the separate activation-backward pass: the same arithmetic in the same
order, so outputs, weight gradients and input gradients are bitwise equal.
The fused path itself is pinned against the oracle by every CARRY parity
test."""
import numpy as np
import pytest

from gpu_harness import gpu_run
from paper_2401_11471_amd import lrcnn as L
from workloads import BF16, F32, Inputs, resnet50_net, tiny_net, vgg16_net

pytestmark = pytest.mark.gpu


def _run(nodes, inp, on, **kw):
    L.lrcnn_debug_act_fusion(on)
    try:
        return gpu_run(nodes, inp, **kw)
    finally:
        L.lrcnn_debug_act_fusion(True)


CASES = [
    ("tiny_f32_carry4", tiny_net, F32, 2, 32, 32, dict(mode=L.CARRY, nb=4)),
    ("vgg16_f32_carry3", vgg16_net, F32, 2, 64, 64, dict(mode=L.CARRY, nb=3)),
    ("vgg16_f32_refine", vgg16_net, F32, 1, 96, 64, dict(mode=L.CARRY, nb=2, bp_refine=2)),
    ("vgg16_f32_layerwise", vgg16_net, F32, 1, 64, 64, dict(layerwise=True)),
    ("resnet50_bf16_carry4", resnet50_net, BF16, 2, 128, 64, dict(mode=L.CARRY, nb=4)),
    ("resnet50_f32_carry2", resnet50_net, F32, 1, 96, 96, dict(mode=L.CARRY, nb=2)),
]


@pytest.mark.parametrize("name,net,dt,b,h,w,kw", CASES, ids=[c[0] for c in CASES])
def test_fused_error_operand_bitwise(name, net, dt, b, h, w, kw):
    print(f"error-operand fusion {name}", flush=True)
    nodes = net()
    inp = Inputs(nodes, b, h, w, 3, dt, seed=31)
    fu = _run(nodes, inp, True, want_dx=True, **kw)
    se = _run(nodes, inp, False, want_dx=True, **kw)
    for k in ("y", "dx"):
        assert np.array_equal(fu[k], se[k]), k
    for v, (p, q) in enumerate(zip(fu["dw"], se["dw"])):
        if p is not None:
            assert np.array_equal(p, q), v
