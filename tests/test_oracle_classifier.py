"""Pins for the oracle's FDCNN classifier head and Adam step (section 2.5.1, Fig. 3;
section 3.1's loss and optimiser).

Closed forms (uniform logits, the first Adam step), an independent library
implementation (torch's cross-entropy and Adam on the CPU, float64), central finite
differences of the loss through the head and through the whole classifier, and
special cases (ReLU cut, weight decay alone).
"""

import numpy as np
import pytest
import torch

from oracle import classifier, fdc

RNG = np.random.default_rng(97531)


def _head_inputs(B=3, F=7, classes=2):
    y = RNG.standard_normal((B, F))
    W = RNG.standard_normal((classes, F))
    bias = RNG.standard_normal(classes)
    labels = RNG.integers(0, classes, B)
    return y, W, bias, labels


def test_uniform_logits_give_log_classes():
    # W = 0, bias = 0: every logit is 0, the softmax is uniform and the loss is ln(classes)
    for classes in (2, 5):
        y = RNG.standard_normal((4, 6))
        logits, loss = classifier.head_forward(y, np.zeros((classes, 6)), np.zeros(classes), np.zeros(4, int))
        assert np.all(logits == 0)
        assert loss == pytest.approx(np.log(classes), rel=1e-15)


def test_head_matches_torch_cross_entropy():
    y, W, bias, labels = _head_inputs(B=5, F=11, classes=3)
    logits, loss = classifier.head_forward(y, W, bias, labels)
    t_logits = torch.relu(torch.from_numpy(y)) @ torch.from_numpy(W).T + torch.from_numpy(bias)
    t_loss = torch.nn.functional.cross_entropy(t_logits, torch.from_numpy(labels))
    np.testing.assert_allclose(logits, t_logits.numpy(), rtol=1e-13, atol=1e-13)
    assert loss == pytest.approx(t_loss.item(), rel=1e-13)


def test_head_backward_finite_differences():
    y, W, bias, labels = _head_inputs(B=3, F=7, classes=3)
    y[np.abs(y) < 0.05] = 0.3  # keep the ReLU kinks away from the difference steps
    logits, _ = classifier.head_forward(y, W, bias, labels)
    gy, gW, gbias = classifier.head_backward(y, W, logits, labels)
    h = 1e-6

    def loss_at(yy, WW, bb):
        return classifier.head_forward(yy, WW, bb, labels)[1]

    for arr, grad, which in ((y, gy, 0), (W, gW, 1), (bias, gbias, 2)):
        num = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            args_p = [y.copy(), W.copy(), bias.copy()]
            args_m = [y.copy(), W.copy(), bias.copy()]
            args_p[which][idx] += h
            args_m[which][idx] -= h
            num[idx] = (loss_at(*args_p) - loss_at(*args_m)) / (2 * h)
        np.testing.assert_allclose(grad, num, rtol=1e-6, atol=1e-9)


def test_relu_cut_blocks_gradient():
    y, W, bias, labels = _head_inputs(B=2, F=5, classes=2)
    y[:, :2] = -1.0
    logits, _ = classifier.head_forward(y, W, bias, labels)
    gy, gW, _ = classifier.head_backward(y, W, logits, labels)
    assert np.all(gy[:, :2] == 0)
    assert np.all(gW[:, :2] == 0)


def test_adam_first_step_closed_form():
    # m = v = 0, step 1, no decay: m_hat = g, v_hat = g^2, so p1 = p0 - lr g / (|g| + eps)
    p = RNG.standard_normal(9)
    g = RNG.standard_normal(9)
    lr, eps = 1e-3, 1e-8
    p1, m1, v1 = classifier.adam_step(p, g, np.zeros(9), np.zeros(9), 1, lr, 0.9, 0.999, eps)
    np.testing.assert_allclose(p1, p - lr * g / (np.abs(g) + eps), rtol=0, atol=1e-15)
    np.testing.assert_allclose(m1, 0.1 * g, rtol=1e-15)
    np.testing.assert_allclose(v1, 0.001 * g * g, rtol=1e-12)


def test_adam_weight_decay_alone():
    # g = 0: the step follows the decay term wd p alone
    p = RNG.standard_normal(6)
    lr, wd = 1e-2, 0.5
    p1, _, _ = classifier.adam_step(p, np.zeros(6), np.zeros(6), np.zeros(6), 1, lr, 0.9, 0.999, 0.0, wd)
    np.testing.assert_allclose(p1, p - lr * np.sign(p), rtol=1e-14)


def test_adam_matches_torch_over_steps():
    n = 13
    p0 = RNG.standard_normal(n)
    grads = [RNG.standard_normal(n) for _ in range(4)]
    lr, b1, b2, eps, wd = 1e-3, 0.8, 0.95, 1e-6, 1e-2
    tp = torch.nn.Parameter(torch.from_numpy(p0.copy()))
    opt = torch.optim.Adam([tp], lr=lr, betas=(b1, b2), eps=eps, weight_decay=wd, foreach=False)
    p, m, v = p0.copy(), np.zeros(n), np.zeros(n)
    for t, g in enumerate(grads, start=1):
        tp.grad = torch.from_numpy(g.copy())
        opt.step()
        p, m, v = classifier.adam_step(p, g, m, v, t, lr, b1, b2, eps, wd)
        np.testing.assert_allclose(p, tp.detach().numpy(), rtol=1e-13, atol=1e-15)


def test_classifier_gradients_finite_differences():
    # whole classifier (chain + head): dL/dK of a layer against central differences of the loss
    sizes, channels, B = (8, 4), (1, 2), 2
    x = RNG.random((B, channels[0], sizes[0], sizes[0]))
    kernels = [RNG.standard_normal((channels[1], sizes[0], sizes[0] // 2 + 1))
               + 1j * RNG.standard_normal((channels[1], sizes[0], sizes[0] // 2 + 1))]
    F = channels[-1] * sizes[-1] ** 2
    W = RNG.standard_normal((2, F)) * 0.3
    bias = np.zeros(2)
    labels = np.array([0, 1])
    loss, _, gks, gW, _ = classifier.classifier_gradients(x, kernels, W, bias, labels, sizes)
    h = 1e-6
    for idx in [(0, 0, 0), (1, 3, 2), (0, 5, 1), (1, 7, 4), (0, 2, 3)]:
        for unit in (1.0, 1j):
            kp = [kernels[0].copy()]
            km = [kernels[0].copy()]
            kp[0][idx] += h * unit
            km[0][idx] -= h * unit
            lp = classifier.classifier_gradients(x, kp, W, bias, labels, sizes)[0]
            lm = classifier.classifier_gradients(x, km, W, bias, labels, sizes)[0]
            num = (lp - lm) / (2 * h)
            # real-pair convention: dL/dRe + i dL/dIm
            got = gks[0][idx].real if unit == 1.0 else gks[0][idx].imag
            assert got == pytest.approx(num, rel=1e-5, abs=1e-9), (idx, unit)
    # the head's weight gradient equals relu(y) weighted by dlogits
    y, _ = fdc.cic_chain_forward(x, kernels, sizes)
    assert gW.shape == (2, F) and np.all(gW[:, (y.reshape(B, -1) <= 0).all(axis=0)] == 0)
