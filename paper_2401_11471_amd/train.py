"""A full training step on the C ABI (Algorithm 1): row-centric FP over the
bands, classifier head and loss, row-centric BP over the bands in reverse,
then the SGD update. Argument marshalling only; every step runs in the HIP
library. The layer-wise baseline runs the same step with
``lrcnn_layerwise_reference_gpu`` (its FP and BP are one call, so the
baseline computes the forward twice: once for y, once with dL/dy)."""
from __future__ import annotations

import torch

from . import lrcnn as L
from .device import DeviceModel, torch_dtype


class Trainer:
    """Owns the device buffers of one training configuration: trunk
    parameters (a DeviceModel), head parameters, workspaces, y and dL/dy."""

    def __init__(self, plan, dm: DeviceModel, fc_w, fc_b, labels, layerwise=False):
        info = plan.info()
        self.plan, self.dm, self.layerwise = plan, dm, layerwise
        B = dm.x.shape[0]
        oshape = (B,) + plan.node_shape(plan.n - 1)
        dev = dm.device
        self.fc_w = torch.as_tensor(fc_w, dtype=torch.float32).to(dev).contiguous()
        self.fc_b = torch.as_tensor(fc_b, dtype=torch.float32).to(dev).contiguous()
        self.labels = torch.as_tensor(labels, dtype=torch.int32).to(dev).contiguous()
        nc = self.fc_w.shape[0]
        self.d_fc_w = torch.empty_like(self.fc_w)
        self.d_fc_b = torch.empty_like(self.fc_b)
        self.logits = torch.empty((B, nc), device=dev, dtype=torch.float32)
        self.loss = torch.empty(4, device=dev, dtype=torch.float32)
        self.y = torch.empty(oshape, device=dev, dtype=torch_dtype(dm.dtype))
        self.dy = torch.zeros_like(self.y)
        self.ws = dm.workspace(info["layerwise_workspace_bytes" if layerwise
                                   else "workspace_bytes"])
        self.head_ws = dm.workspace(L.lrcnn_head_workspace_bytes(plan, nc))

    def step(self, lr):
        """One SGD step; returns the loss (a device scalar view) before the
        update."""
        p, dm = self.plan, self.dm
        if self.layerwise:
            L.lrcnn_layerwise_reference_gpu(p, dm.x, dm.w, dm.sc, dm.sf, self.dy, self.y, dm.dw,
                                            None, self.ws)
        else:
            L.lrcnn_forward_rows(p, dm.x, dm.w, dm.sc, dm.sf, self.y, self.ws)
        L.lrcnn_head_loss(p, self.y, self.fc_w, self.fc_b, self.labels, self.logits,
                          self.loss, self.dy, self.d_fc_w, self.d_fc_b, self.head_ws)
        if self.layerwise:
            L.lrcnn_layerwise_reference_gpu(p, dm.x, dm.w, dm.sc, dm.sf, self.dy, self.y, dm.dw,
                                            None, self.ws)
        else:
            L.lrcnn_backward_rows(p, dm.x, dm.w, dm.sc, dm.sf, self.dy, dm.dw, None, self.ws)
        L.lrcnn_sgd_update(p, lr, dm.w, dm.dw, self.fc_w, self.d_fc_w, self.fc_b, self.d_fc_b)
        return self.loss[0]
