"""Large kernels at the edges of the tap-mask loaders, against the float64
oracle. The 16-byte loaders test taps against one 64-bit mask per tile row.
An 8x8 kernel (64 taps) uses its last bit, and the mask row for kernel row 7
starts at bit 56. A 9x9 kernel (81 taps) is sent to the element-wise loader
although its channel count fills 16-byte vectors. Each net has odd map sizes
(ragged tiles), padding on both sides (rows and columns outside the window
under many taps), stride 1 and stride 2 (input-gradient stride phases), and
band boundaries (CARRY) or a layer-wise run."""
import pytest

from gpu_harness import assert_parity, gpu_run
from paper_2401_11471_amd import lrcnn as L
from workloads import BF16, F32, Inputs, NetBuilder

pytestmark = pytest.mark.gpu


def net_8x8():
    nb = NetBuilder()
    v = nb.conv(0, 16, 3, 1, 1)
    v = nb.conv(v, 32, 8, 1, 4)       # 64 taps, stride 1 (output one wider)
    v = nb.conv(v, 32, 8, 2, 3)       # 64 taps, stride 2 (phases of 16 taps)
    return nb.nodes


def net_9x9():
    nb = NetBuilder()
    v = nb.conv(0, 16, 3, 1, 1)
    v = nb.conv(v, 32, 9, 1, 4)       # 81 taps: element-wise loader
    v = nb.conv(v, 16, 9, 2, 4)
    return nb.nodes


CASES = [
    ("k8_f32_carry3", net_8x8, F32, 2, 45, 39, dict(mode=L.CARRY, nb=3)),
    ("k8_bf16_carry2", net_8x8, BF16, 2, 45, 39, dict(mode=L.CARRY, nb=2)),
    ("k8_f32_layerwise", net_8x8, F32, 1, 37, 41, dict(layerwise=True)),
    ("k9_f32_carry3", net_9x9, F32, 2, 47, 35, dict(mode=L.CARRY, nb=3)),
    ("k9_bf16_layerwise", net_9x9, BF16, 1, 41, 43, dict(layerwise=True)),
]


@pytest.mark.parametrize("name,net,dt,b,h,w,kw", CASES, ids=[c[0] for c in CASES])
def test_large_kernel_parity(name, net, dt, b, h, w, kw):
    print(f"large kernel {name}", flush=True)
    nodes = net()
    inp = Inputs(nodes, b, h, w, 3, dt, seed=31)
    out = gpu_run(nodes, inp, want_dx=True, **kw)
    assert_parity(nodes, inp, out)
