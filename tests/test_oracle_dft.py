"""Pins for the oracle's real 2-D DFT and its inverse/adjoints (section 2.4.1.1, Eq. 4).

Each test checks the oracle against something other than itself: a hand-worked
example, a closed form, an identity of the DFT, or an independent FFT library.
"""

import numpy as np
import pytest

from oracle import dft

RNG = np.random.default_rng(1234)
SHAPES = [(4, 4), (8, 8), (6, 10), (16, 8), (14, 14)]


def test_worked_4x4_rfft2(golden):
    g = golden("worked_4x4.txt")
    got = dft.rfft2(np.array(g["x"], dtype=float))
    np.testing.assert_allclose(got, np.array(g["rfft2_x"]), atol=1e-12)
    got_k = dft.rfft2(np.pad(np.array(g["kernel"], dtype=float), ((0, 2), (0, 2))))
    np.testing.assert_allclose(got_k, np.array(g["rfft2_kernel"]), atol=1e-12)


def test_closed_form_single_pixel():
    # An impulse at (a, b) has spectrum exp(-2 pi i (a k / H + b l / W)).
    h, w, a, b = 8, 6, 3, 5
    x = np.zeros((h, w))
    x[a, b] = 1.0
    k = np.arange(h)[:, None]
    l = np.arange(w // 2 + 1)[None, :]
    expect = np.exp(-2j * np.pi * (a * k / h + b * l / w))
    np.testing.assert_allclose(dft.rfft2(x), expect, atol=1e-12)


def test_closed_form_cosine():
    # x = cos(2 pi (k0 h / H + l0 w / W)) has X = HW/2 at (k0, l0) and nothing else in 0 < l < W/2.
    h, w, k0, l0 = 8, 8, 3, 2
    hh, ww = np.meshgrid(np.arange(h), np.arange(w), indexing="ij")
    x = np.cos(2 * np.pi * (k0 * hh / h + l0 * ww / w))
    X = dft.rfft2(x)
    expect = np.zeros_like(X)
    expect[k0, l0] = h * w / 2
    np.testing.assert_allclose(X, expect, atol=1e-10)


@pytest.mark.parametrize("shape", SHAPES)
def test_against_numpy_fft(shape):
    x = RNG.standard_normal((3,) + shape)
    np.testing.assert_allclose(dft.rfft2(x), np.fft.rfft2(x), atol=1e-10)
    y = RNG.standard_normal((3, shape[0], shape[1] // 2 + 1)) + 1j * RNG.standard_normal(
        (3, shape[0], shape[1] // 2 + 1))
    np.testing.assert_allclose(dft.irfft2(y, *shape), np.fft.irfft2(y, s=shape), atol=1e-12)


@pytest.mark.parametrize("shape", SHAPES)
def test_parseval(shape):
    x = RNG.standard_normal(shape)
    X = dft.rfft2(x)
    c = dft.half_weights(shape[1])
    lhs = np.sum(x * x)
    rhs = np.sum(c * np.abs(X) ** 2) / (shape[0] * shape[1])
    assert abs(lhs - rhs) < 1e-10 * lhs


@pytest.mark.parametrize("shape", SHAPES)
def test_inverse_and_projection(shape):
    h, w = shape
    x = RNG.standard_normal((2, h, w))
    np.testing.assert_allclose(dft.irfft2(dft.rfft2(x), h, w), x, atol=1e-12)
    # A non-Hermitian half spectrum comes back Hermitian-projected; the projection
    # fixes spectra of real images and is idempotent.
    y = RNG.standard_normal((2, h, w // 2 + 1)) + 1j * RNG.standard_normal((2, h, w // 2 + 1))
    py = dft.hermitian_projection(y)
    np.testing.assert_allclose(dft.rfft2(dft.irfft2(y, h, w)), py, atol=1e-12)
    np.testing.assert_allclose(dft.hermitian_projection(py), py, atol=1e-14)
    X = dft.rfft2(x)
    np.testing.assert_allclose(dft.hermitian_projection(X), X, atol=1e-12)
    # columns 0 < l < W/2 are never touched
    np.testing.assert_array_equal(py[..., 1:-1], y[..., 1:-1])


def _rdot(a, b):
    return float(np.sum(np.real(a * np.conj(b))))


@pytest.mark.parametrize("shape", SHAPES)
def test_adjoints(shape):
    h, w = shape
    x = RNG.standard_normal((2, h, w))
    g = RNG.standard_normal((2, h, w // 2 + 1)) + 1j * RNG.standard_normal((2, h, w // 2 + 1))
    # <rfft2 x, g> = <x, rfft2* g>
    assert abs(_rdot(dft.rfft2(x), g) - _rdot(x, dft.rfft2_adjoint(g, h, w))) < 1e-9
    # <irfft2 g, x> = <g, irfft2* x>
    assert abs(_rdot(dft.irfft2(g, h, w), x) - _rdot(g, dft.irfft2_adjoint(x))) < 1e-9


def test_adjoint_finite_difference():
    # dL/dRe Y and dL/dIm Y of L = <irfft2(Y), g>, by central differences.
    h, w = 4, 6
    g = RNG.standard_normal((h, w))
    y = RNG.standard_normal((h, w // 2 + 1)) + 1j * RNG.standard_normal((h, w // 2 + 1))
    grad = dft.irfft2_adjoint(g)
    eps = 1e-6
    for k in range(h):
        for l in range(w // 2 + 1):
            for unit, part in ((1.0, np.real), (1j, np.imag)):
                yp = y.copy()
                ym = y.copy()
                yp[k, l] += eps * unit
                ym[k, l] -= eps * unit
                fd = (np.sum(dft.irfft2(yp, h, w) * g) - np.sum(dft.irfft2(ym, h, w) * g)) / (2 * eps)
                assert abs(fd - part(grad[k, l])) < 1e-8
