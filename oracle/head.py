"""Classifier head, loss and parameter update of a training step in float64
(Algorithm 1: fully connected FP, Loss, fully connected BP, then the update
of every kernel and of the fully connected weights).

TEST INFRASTRUCTURE. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package. It shares no
code with the HIP library and never calls it.

Readings (the paper names the steps, not their form): one fully connected
layer over the flattened trunk output (NHWC order) with a bias; softmax
cross-entropy averaged over the batch; plain SGD, theta <- theta - lr * g,
on the conv kernels and the fully connected weights and bias (the fixed
per-channel affine parameters are not trained). In bfloat16 mode the conv
weights are stored in bfloat16, so each update is rounded to bfloat16, and
dL/dy enters the trunk's backward rounded to bfloat16 (the storage dtype of
y); the head itself stays float64.
"""
from __future__ import annotations

import numpy as np

from . import column as OC
from .bf16 import round_bf16


def head_forward(y, fc_w, fc_b):
    """logits[b, c] = sum_k flat(y)[b, k] * fc_w[c, k] + fc_b[c]."""
    yb = np.asarray(y, np.float64).reshape(y.shape[0], -1)
    return yb @ np.asarray(fc_w, np.float64).T + np.asarray(fc_b, np.float64)


def softmax_xent(logits, labels):
    """Mean softmax cross-entropy over the batch and its gradient with
    respect to the logits: (softmax - onehot) / B."""
    z = np.asarray(logits, np.float64)
    z = z - z.max(axis=1, keepdims=True)
    p = np.exp(z)
    p /= p.sum(axis=1, keepdims=True)
    b = z.shape[0]
    rows = np.arange(b)
    loss = -np.mean(np.log(p[rows, labels]))
    d = p.copy()
    d[rows, labels] -= 1.0
    return loss, d / b


def head_backward(y, fc_w, dlogits):
    """Chain rule through the fully connected layer: dy (shape of y),
    d fc_w = dlogits^T flat(y), d fc_b = column sums of dlogits."""
    yb = np.asarray(y, np.float64).reshape(y.shape[0], -1)
    dy = (dlogits @ np.asarray(fc_w, np.float64)).reshape(y.shape)
    return dy, dlogits.T @ yb, dlogits.sum(axis=0)


def sgd(param, grad, lr, bf16=False):
    out = np.asarray(param, np.float64) - lr * np.asarray(grad, np.float64)
    return round_bf16(out) if bf16 else out


def train(nodes, x, weights, scales, shifts, fc_w, fc_b, labels, lr, steps, bf16=False):
    """``steps`` SGD steps of column training with the head on one batch.
    Returns the loss before each update and the final parameters."""
    weights = [None if w is None else np.asarray(w, np.float64) for w in weights]
    fc_w = np.asarray(fc_w, np.float64)
    fc_b = np.asarray(fc_b, np.float64)
    losses = []
    for _ in range(steps):
        acts, am = OC.forward(nodes, x, weights, scales, shifts, bf16=bf16)
        y = acts[-1]
        loss, dlog = softmax_xent(head_forward(y, fc_w, fc_b), labels)
        dy, dfw, dfb = head_backward(y, fc_w, dlog)
        if bf16:
            dy = round_bf16(dy)
        dws, _ = OC.backward(nodes, acts, am, weights, scales, dy, bf16=bf16, want_dx=False)
        losses.append(loss)
        weights = [None if w is None else sgd(w, dws[v + 1], lr, bf16)
                   for v, w in enumerate(weights)]
        fc_w = sgd(fc_w, dfw, lr)
        fc_b = sgd(fc_b, dfb, lr)
    return losses, weights, fc_w, fc_b
