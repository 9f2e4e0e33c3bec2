"""Pins for the oracle's Full FDC layer (Algorithm 2 with the per-bin sum of Eq. 2).

Checked against brute-force spatial convolution over volume, a library
convolution, the CIC special case, adjoint identities and finite differences.
"""

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import conv, fdc

RNG = np.random.default_rng(777)


@pytest.mark.parametrize("p,n", [(8, 3), (10, 3), (8, 1), (12, 5)])
def test_full_fdc_crop_is_valid_convolution_over_volume(p, n):
    b, c, s = 2, 3, 4
    x = RNG.standard_normal((b, c, p, p))
    w = RNG.standard_normal((s, c, n, n))
    y, _ = fdc.full_fdc_forward(x, w, fdc.ARTIFACT_CROP)
    assert y.shape == (b, s, p - n + 1, p - n + 1)
    ref = F.conv2d(torch.from_numpy(x), torch.from_numpy(w[..., ::-1, ::-1].copy())).numpy()
    np.testing.assert_allclose(y, ref, atol=1e-11)
    # Eq. 2 with Eq. 1 by loops, for one image
    np.testing.assert_allclose(y[1], conv.cov_valid(x[1], w), atol=1e-11)


def test_full_fdc_roll_is_circular_same_convolution():
    b, c, s, p, n = 1, 2, 3, 8, 3
    x = RNG.standard_normal((b, c, p, p))
    w = RNG.standard_normal((s, c, n, n))
    y, _ = fdc.full_fdc_forward(x, w, fdc.ARTIFACT_ROLL)
    xp = F.pad(torch.from_numpy(x), (1, 1, 1, 1), mode="circular")
    ref = F.conv2d(xp, torch.from_numpy(w[..., ::-1, ::-1].copy())).numpy()
    np.testing.assert_allclose(y, ref, atol=1e-11)


def test_full_fdc_contains_cic():
    # A COV kernel set that is zero unless c = s // J reduces to CIC (Eq. 5 vs Eq. 2).
    b, c, j, p = 2, 2, 3, 8
    s = c * j
    x = RNG.standard_normal((b, c, p, p))
    k = RNG.standard_normal((s, 3, 3))
    w = np.zeros((s, c, 3, 3))
    for o in range(s):
        w[o, o // j] = k[o]
    y_full, _ = fdc.full_fdc_forward(x, w, fdc.ARTIFACT_NONE)
    y_cic, _ = fdc.cic_fdp_layer_forward(x, fdc.kernel_spectrum(k, p, p), p)
    np.testing.assert_allclose(y_full, y_cic, atol=1e-11)


def test_full_fdc_adjoint_in_x():
    b, c, s, p, n = 2, 2, 3, 8, 3
    x = RNG.standard_normal((b, c, p, p))
    w = RNG.standard_normal((s, c, n, n))
    y, xs = fdc.full_fdc_forward(x, w)
    gy = RNG.standard_normal(y.shape)
    gx, _ = fdc.full_fdc_backward(gy, xs, w)
    assert abs(np.sum(y * gy) - np.sum(x * gx)) < 1e-9


@pytest.mark.parametrize("mode", [fdc.ARTIFACT_CROP, fdc.ARTIFACT_ROLL])
def test_full_fdc_gradients_finite_difference(mode):
    b, c, s, p, n = 2, 2, 3, 8, 3
    x = RNG.standard_normal((b, c, p, p))
    w = RNG.standard_normal((s, c, n, n))
    y, xs = fdc.full_fdc_forward(x, w, mode)
    gy = RNG.standard_normal(y.shape)
    gx, gw = fdc.full_fdc_backward(gy, xs, w, mode)
    loss = lambda xx, ww: float(np.sum(fdc.full_fdc_forward(xx, ww, mode)[0] * gy))
    eps = 1e-6
    for idx in [(0, 0, 0, 0), (2, 1, 2, 1), (1, 0, 1, 2)]:
        wp, wm = w.copy(), w.copy()
        wp[idx] += eps
        wm[idx] -= eps
        assert abs((loss(x, wp) - loss(x, wm)) / (2 * eps) - gw[idx]) < 1e-7
    for idx in [(0, 1, 0, 0), (1, 0, 7, 3)]:
        xp, xm = x.copy(), x.copy()
        xp[idx] += eps
        xm[idx] -= eps
        assert abs((loss(xp, w) - loss(xm, w)) / (2 * eps) - gx[idx]) < 1e-7


def test_weight_gradient_matches_library_autograd():
    # torch autograd of the library convolution gives dL/dw independently.
    b, c, s, p, n = 2, 3, 2, 9 + 1, 3
    x = RNG.standard_normal((b, c, p, p))
    w = RNG.standard_normal((s, c, n, n))
    y, xs = fdc.full_fdc_forward(x, w)
    gy = RNG.standard_normal(y.shape)
    gx, gw = fdc.full_fdc_backward(gy, xs, w)
    xt = torch.from_numpy(x).requires_grad_(True)
    wt = torch.from_numpy(w).requires_grad_(True)
    out = F.conv2d(xt, wt.flip(-1, -2))
    (out * torch.from_numpy(gy)).sum().backward()
    np.testing.assert_allclose(gw, wt.grad.numpy(), atol=1e-10)
    np.testing.assert_allclose(gx, xt.grad.numpy(), atol=1e-10)
