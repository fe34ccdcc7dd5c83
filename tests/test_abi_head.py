"""Host-side checks of the head / update entry points (no GPU work)."""
import ctypes as C

import pytest

from paper_2401_11471_amd import lrcnn as L
from workloads import tiny_net, vgg16_net


def test_head_workspace_bytes():
    p = L.lrcnn_plan(vgg16_net(), 8, 3, 224, 224)
    k = 7 * 7 * 512
    chunks = -(-k // 8192)
    a = lambda x: -(-x // 256) * 256
    want = a(a(a(8 * chunks * 10 * 4) + 8 * 10 * 4) + 8 * 4)
    assert L.lrcnn_head_workspace_bytes(p, 10) == want
    for bad in (0, 65):
        with pytest.raises(L.LrcnnError) as e:
            L.lrcnn_head_workspace_bytes(p, bad)
        assert e.value.code == -1


def test_head_and_update_reject_bad_arguments():
    p = L.lrcnn_plan(tiny_net(), 1, 3, 32, 32, L.F32, L.CARRY, 4)
    fake = 1 << 20
    need = L.lrcnn_head_workspace_bytes(p, 10)
    args = [fake] * 4
    st = L.LIB.lrcnn_head_loss(p.handle, None, *args[:3], 10, *([fake] * 6), need, None)
    assert st == -1                                  # y is null
    st = L.LIB.lrcnn_head_loss(p.handle, fake + 4, *args[:3], 10, *([fake] * 6), need, None)
    assert st == -1                                  # misaligned
    st = L.LIB.lrcnn_head_loss(p.handle, fake, *args[:3], 10, *([fake] * 6), need - 1, None)
    assert st == -4                                  # head workspace too small
    st = L.LIB.lrcnn_head_loss(p.handle, fake, *args[:3], 99, *([fake] * 6), need, None)
    assert st == -1                                  # too many classes
    nulls = (C.c_void_p * 4)()
    st = L.LIB.lrcnn_sgd_update(p.handle, C.c_float(0.1), nulls, nulls, None, None, None, None,
                                0, None)
    assert st == -1                                  # conv weights missing
