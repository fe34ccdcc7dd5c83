"""Pins of the oracle's classifier head, loss and SGD update (CPU only).

* softmax cross-entropy and its gradient equal torch's float64
  ``cross_entropy`` and autograd (a library routine);
* closed forms: uniform logits give log(C) and gradient (1/C - onehot)/B;
  the gradient of every row sums to zero;
* the chain rule through the fully connected layer matches central finite
  differences of the loss in y, fc_w and fc_b;
* a training step with a small learning rate lowers the loss (first-order
  descent) and lr = 0 leaves it unchanged.
"""
import numpy as np
import pytest
import torch

from oracle import head as OH
from workloads import Inputs, tiny_net

rng = np.random.default_rng(5)


def test_softmax_xent_matches_torch():
    for b, c in ((1, 2), (4, 10), (7, 33)):
        z = rng.standard_normal((b, c)) * 3
        lab = rng.integers(0, c, b)
        loss, d = OH.softmax_xent(z, lab)
        t = torch.tensor(z, dtype=torch.float64, requires_grad=True)
        ref = torch.nn.functional.cross_entropy(t, torch.tensor(lab))
        ref.backward()
        assert abs(loss - ref.item()) < 1e-12
        np.testing.assert_allclose(d, t.grad.numpy(), rtol=0, atol=1e-14)


def test_softmax_xent_closed_forms():
    b, c = 5, 10
    lab = np.arange(b) % c
    loss, d = OH.softmax_xent(np.full((b, c), 0.7), lab)
    assert abs(loss - np.log(c)) < 1e-14
    exp = np.full((b, c), 1.0 / c)
    exp[np.arange(b), lab] -= 1.0
    np.testing.assert_allclose(d, exp / b, atol=1e-16)
    _, d2 = OH.softmax_xent(rng.standard_normal((b, c)), lab)
    np.testing.assert_allclose(d2.sum(axis=1), 0.0, atol=1e-16)


def test_head_gradients_match_finite_differences():
    b, h, w, ch, c = 3, 2, 3, 4, 5
    y = rng.standard_normal((b, h, w, ch))
    fw = rng.standard_normal((c, h * w * ch)) * 0.3
    fb = rng.standard_normal(c) * 0.1
    lab = rng.integers(0, c, b)

    def loss(y_, fw_, fb_):
        return OH.softmax_xent(OH.head_forward(y_, fw_, fb_), lab)[0]

    _, dlog = OH.softmax_xent(OH.head_forward(y, fw, fb), lab)
    dy, dfw, dfb = OH.head_backward(y, fw, dlog)
    eps = 1e-6
    for _ in range(4):
        vy, vw, vb = (rng.standard_normal(t.shape) for t in (y, fw, fb))
        fd = (loss(y + eps * vy, fw + eps * vw, fb + eps * vb) -
              loss(y - eps * vy, fw - eps * vw, fb - eps * vb)) / (2 * eps)
        an = (dy * vy).sum() + (dfw * vw).sum() + (dfb * vb).sum()
        assert abs(fd - an) <= 1e-7 * max(1.0, abs(an))


@pytest.mark.parametrize("bf16", [False, True])
def test_training_step_descends(bf16):
    nodes = tiny_net()
    inp = Inputs(nodes, 2, 16, 16, 3, dtype=1 if bf16 else 0, seed=3)
    k = 16 * 16 * 8
    fw = np.random.default_rng(1).standard_normal((10, k)) * 0.01
    fb = np.zeros(10)
    lab = np.array([3, 7])
    l0, w0, fw0, _ = OH.train(nodes, inp.x, inp.weights, inp.scales, inp.shifts, fw, fb, lab,
                              0.0, 2, bf16=bf16)
    assert l0[0] == l0[1]
    np.testing.assert_array_equal(fw0, fw)
    ls, _, _, _ = OH.train(nodes, inp.x, inp.weights, inp.scales, inp.shifts, fw, fb, lab,
                           1e-4, 3, bf16=bf16)
    assert ls[1] < ls[0] and ls[2] < ls[1]


def test_sgd_rounds_to_bf16():
    p = np.array([1.0, -2.5, 3.0])
    g = np.array([1e-3, 2e-3, -1e-4])
    out = OH.sgd(p, g, 0.5, bf16=True)
    t = torch.tensor(p - 0.5 * g, dtype=torch.float64).to(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(out, t)
