"""Device tensors for one workload, arranged as the C ABI's per-node arrays
(index = node id; entries of nodes without weights are None). Marshalling
only: host arrays are copied to torch device tensors of the plan's dtype."""
from __future__ import annotations

import numpy as np
import torch

from .lrcnn import BF16, OP_CONV


def torch_dtype(dtype):
    return torch.bfloat16 if dtype == BF16 else torch.float32


class DeviceModel:
    def __init__(self, nodes, x, weights, scales, shifts, dtype, device="cuda"):
        tdt = torch_dtype(dtype)
        self.nodes = list(nodes)
        self.dtype = dtype
        self.device = device
        self.x = torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(device=device, dtype=tdt)
        self.w = [None]
        self.sc = [None]
        self.sf = [None]
        self.dw = [None]
        for v, nd in enumerate(self.nodes[1:], start=1):
            wv, sv, fv = weights[v - 1], scales[v - 1], shifts[v - 1]
            if nd[0] == OP_CONV:
                self.w.append(torch.from_numpy(np.ascontiguousarray(wv, np.float32))
                              .to(device=device, dtype=tdt))
                self.dw.append(torch.empty(wv.shape, device=device, dtype=torch.float32))
            else:
                self.w.append(None)
                self.dw.append(None)
            self.sc.append(None if sv is None else torch.from_numpy(
                np.ascontiguousarray(sv, np.float32)).to(device))
            self.sf.append(None if fv is None else torch.from_numpy(
                np.ascontiguousarray(fv, np.float32)).to(device))

    @classmethod
    def from_inputs(cls, nodes, inp, device="cuda"):
        return cls(nodes, inp.x, inp.weights, inp.scales, inp.shifts, inp.dtype, device)

    def empty(self, shape, dtype=None):
        return torch.empty(shape, device=self.device,
                           dtype=dtype or torch_dtype(self.dtype))

    def workspace(self, nbytes):
        return torch.empty(max(int(nbytes), 256), device=self.device, dtype=torch.uint8)

    def to_device(self, a):
        return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(
            device=self.device, dtype=torch_dtype(self.dtype))
