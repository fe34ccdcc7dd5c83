"""Seeded synthetic workloads shared by the CPU oracle and the HIP path.

This module only describes networks as node lists and draws random numbers.
It contains none of the row-centric method's arithmetic (no shape inference,
no convolution, no partitioning), so both sides can take their inputs from it
without sharing code.

Node tuple layout (mirrors ``lrcnn_node`` in ``include/lrcnn.h``):
    (op, in0, in1, c_out, kh, kw, sh, sw, ph, pw, affine, relu)
op: 0 = input, 1 = conv (cross-correlation, bias-free), 2 = max-pool, 3 = add.

Networks follow the paper's benchmarks (VGG-16 and ResNet-50, Section V-A);
ImageNet is not available, so every tensor is drawn from N(0, 1) with the
paper's shapes.
"""
from __future__ import annotations

import numpy as np

OP_INPUT, OP_CONV, OP_MAXPOOL, OP_ADD = 0, 1, 2, 3
F32, BF16 = 0, 1
CARRY, RECOMPUTE = 0, 1


def _n(op, in0=-1, in1=-1, c_out=0, k=1, s=1, p=0, affine=0, relu=0):
    return (op, in0, in1, c_out, k, k, s, s, p, p, affine, relu)


class NetBuilder:
    def __init__(self):
        self.nodes = [_n(OP_INPUT)]

    def add(self, node):
        self.nodes.append(node)
        return len(self.nodes) - 1

    def conv(self, src, c_out, k, s=1, p=0, affine=0, relu=1):
        return self.add(_n(OP_CONV, src, -1, c_out, k, s, p, affine, relu))

    def pool(self, src, k, s, p=0):
        return self.add(_n(OP_MAXPOOL, src, -1, 0, k, s, p))

    def sum(self, a, b, relu=1):
        return self.add(_n(OP_ADD, a, b, 0, 1, 1, 0, 0, relu))


def tiny_net(channels=(8, 8, 8)):
    """Three 3x3 stride-1 pad-1 convs with ReLU (the 3->8->8->8 stack)."""
    nb = NetBuilder()
    v = 0
    for c in channels:
        v = nb.conv(v, c, 3, 1, 1)
    return nb.nodes


def vgg16_net(with_pool5=True):
    """VGG-16 conv trunk: 13 3x3 pad-1 convs with ReLU, 2x2/2 max-pool after
    each of the five blocks (channels 64/128/256/512/512)."""
    nb = NetBuilder()
    v = 0
    blocks = [(64, 2), (128, 2), (256, 3), (512, 3), (512, 3)]
    for bi, (c, n) in enumerate(blocks):
        for _ in range(n):
            v = nb.conv(v, c, 3, 1, 1)
        if with_pool5 or bi < 4:
            v = nb.pool(v, 2, 2, 0)
    return nb.nodes


def resnet50_net(layers=(3, 4, 6, 3)):
    """ResNet-50 conv trunk (v1.5: stride on the 3x3), BatchNorm replaced by a
    fixed per-channel affine. Output is the last block's ReLU output."""
    nb = NetBuilder()
    v = nb.conv(0, 64, 7, 2, 3, affine=1, relu=1)
    v = nb.pool(v, 3, 2, 1)
    c_in = 64
    for li, nblocks in enumerate(layers):
        width = 64 * (2 ** li)
        for bi in range(nblocks):
            stride = 2 if (li > 0 and bi == 0) else 1
            c1 = nb.conv(v, width, 1, 1, 0, affine=1, relu=1)
            c2 = nb.conv(c1, width, 3, stride, 1, affine=1, relu=1)
            c3 = nb.conv(c2, 4 * width, 1, 1, 0, affine=1, relu=0)
            if bi == 0:
                sc = nb.conv(v, 4 * width, 1, stride, 0, affine=1, relu=0)
            else:
                sc = v
            v = nb.sum(c3, sc, relu=1)
            c_in = 4 * width
    del c_in
    return nb.nodes


# The five benchmark workloads: (name, net, dtype, batch, H, W, bands).
CONFIGS = {
    1: dict(name="tiny3x3_f32_b1_32x32", net="tiny", dtype=F32, batch=1,
            h=32, w=32, bands=4),
    # step: the row-centric step's plan options at this workload (policy 0
    # even / 1 balanced; bp_refine backward bands per forward band;
    # hybrid_from -1 = the planner's checkpoint): at 224 px the plain
    # two-phase-sharing step keeps about 2.5x less activation memory than
    # the layer-wise step, these about 3.2-3.5x, at the same or better speed
    2: dict(name="vgg16_f32_b8_224x224", net="vgg16", dtype=F32, batch=8,
            h=224, w=224, bands=4, step=dict(policy=0, bp_refine=2, hybrid_from=-1)),
    3: dict(name="resnet50_bf16_b16_224x224", net="resnet50", dtype=BF16,
            batch=16, h=224, w=224, bands=8, step=dict(policy=1, bp_refine=1, hybrid_from=-1)),
    4: dict(name="vgg16_f32_b4_1200x1800", net="vgg16", dtype=F32, batch=4,
            h=1200, w=1800, bands=16),
    5: dict(name="resnet50_bf16_b8_2400x3600", net="resnet50", dtype=BF16,
            batch=8, h=2400, w=3600, bands=32),
}


def net_nodes(name):
    return {"tiny": tiny_net, "vgg16": vgg16_net,
            "resnet50": resnet50_net}[name]()


def to_bf16_values(a):
    """Round float32 values to the nearest bfloat16 (library conversion),
    returned as float32 so both sides receive bf16-representable inputs."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


class Inputs:
    """Seeded inputs for one workload: x (B,H,W,C) NHWC, conv weights in
    [C_out][kh][kw][C_in] (drawn OIHW, He-normal fan-in, then permuted),
    per-conv affine (scale, shift) or None, and a deferred upstream gradient
    G drawn once its shape is known."""

    def __init__(self, nodes, batch, h, w, c=3, dtype=F32, seed=0,
                 x_scale=1.0):
        self.nodes = nodes
        self.dtype = dtype
        ss = np.random.SeedSequence(seed).spawn(4)
        self._rx, self._rw, self._ra = (np.random.default_rng(s)
                                        for s in ss[:3])
        self._gseed = ss[3]
        x = self._rx.standard_normal((batch, h, w, c), dtype=np.float32)
        if x_scale != 1.0:
            x *= np.float32(x_scale)
        self.x = self._cast(x)
        self.weights = []
        self.scales = []
        self.shifts = []
        # channel count per node, needed only to size the weight draws
        chans = [c]
        for (op, in0, in1, c_out, kh, kw, *_rest) in nodes[1:]:
            aff = _rest[-2]
            if op == OP_CONV:
                ci = chans[in0]
                std = np.sqrt(2.0 / (ci * kh * kw))
                wt = self._rw.standard_normal((c_out, ci, kh, kw))
                wt = (wt * std).astype(np.float32).transpose(0, 2, 3, 1)
                self.weights.append(self._cast(np.ascontiguousarray(wt)))
                if aff:
                    self.scales.append(self._ra.uniform(0.5, 1.0, c_out)
                                       .astype(np.float32))
                    self.shifts.append(self._ra.uniform(-0.1, 0.1, c_out)
                                       .astype(np.float32))
                else:
                    self.scales.append(None)
                    self.shifts.append(None)
                chans.append(c_out)
            else:
                self.weights.append(None)
                self.scales.append(None)
                self.shifts.append(None)
                chans.append(chans[in0])
        self._g = None

    def _cast(self, a):
        return to_bf16_values(a) if self.dtype == BF16 else a

    def grad(self, shape):
        """Upstream gradient G (dL/dy for L = sum(y * G)) of the given shape."""
        if self._g is None or self._g.shape != tuple(shape):
            rng = np.random.default_rng(self._gseed)
            g = rng.standard_normal(tuple(shape), dtype=np.float32)
            self._g = self._cast(g)
        return self._g


def config_inputs(cfg_id, batch=None, h=None, w=None):
    c = CONFIGS[cfg_id]
    nodes = net_nodes(c["net"])
    return nodes, Inputs(nodes, batch or c["batch"], h or c["h"], w or c["w"],
                         3, c["dtype"], seed=cfg_id)
