"""Pins for the oracle's CIC + FDP layer (Eq. 4, Eq. 5, Algorithm 1, sections 2.4.1.3 and 2.4.2).

Brute-force spatial convolution, a library convolution, closed forms for the
pooling crop, hand-worked values, adjoint identities and finite differences.
"""

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import conv, dft, fdc

RNG = np.random.default_rng(4321)


def _spectral_from_spatial(k, n):
    """K = rfft2 of the kernel padded at the top-left (used to build test kernels)."""
    return fdc.kernel_spectrum(k, n, n)


def _rand_complex(shape):
    return RNG.standard_normal(shape) + 1j * RNG.standard_normal(shape)


# ---------------------------------------------------------------------------- P1
@pytest.mark.parametrize("n_img", [4, 8, 16])
@pytest.mark.parametrize("n_k", [1, 2, 3, 5])
def test_cic_is_circular_convolution(n_img, n_k):
    if n_k > n_img:
        pytest.skip("kernel larger than image")
    b, c, j = 2, 2, 2
    x = RNG.standard_normal((b, c, n_img, n_img))
    k = RNG.standard_normal((c * j, n_k, n_k))
    y, _ = fdc.cic_fdp_layer_forward(x, _spectral_from_spatial(k, n_img), n_img)
    for bi in range(b):
        for o in range(c * j):
            ref = conv.circular_convolve(x[bi, o // j], k[o])
            np.testing.assert_allclose(y[bi, o], ref, atol=1e-11)


def test_full_size_kernel_is_circular_convolution():
    # A kernel as large as the image (spectral kernels have no smaller support).
    n = 8
    x = RNG.standard_normal((1, 1, n, n))
    k = RNG.standard_normal((3, n, n))
    y, _ = fdc.cic_fdp_layer_forward(x, _spectral_from_spatial(k, n), n)
    for o in range(3):
        np.testing.assert_allclose(y[0, o], conv.circular_convolve(x[0, 0], k[o]), atol=1e-10)


def test_worked_4x4_cic(golden):
    g = golden("worked_4x4.txt")
    x = np.array(g["x"], dtype=float)[None, None]
    K = np.array(g["rfft2_kernel"])[None]
    y, _ = fdc.cic_fdp_layer_forward(x, K, 4)
    np.testing.assert_allclose(y[0, 0], np.array(g["cic_circular"], dtype=float), atol=1e-12)
    yc, _ = fdc.cic_fdp_layer_forward(x, K, 4, fdc.ARTIFACT_CROP, 2)
    np.testing.assert_allclose(yc[0, 0], np.array(g["cic_crop"], dtype=float), atol=1e-12)


# ---------------------------------------------------------------------------- P2
@pytest.mark.parametrize("n_k", [1, 2, 3, 5])
def test_crop_equals_library_valid_conv(n_k):
    # Artifact cropping of n-1 rows/cols leaves the valid convolution (section 2.4.1.3);
    # PyTorch's conv2d is a cross-correlation, so the kernel is flipped.  groups=C
    # with S outputs puts output o on input o // J: the CIC channel order.
    b, c, j, n = 2, 3, 2, 12
    x = RNG.standard_normal((b, c, n, n))
    k = RNG.standard_normal((c * j, n_k, n_k))
    y, _ = fdc.cic_fdp_layer_forward(x, _spectral_from_spatial(k, n), n, fdc.ARTIFACT_CROP, n_k)
    ref = F.conv2d(torch.from_numpy(x), torch.from_numpy(k[:, None, ::-1, ::-1].copy()), groups=c)
    np.testing.assert_allclose(y, ref.numpy(), atol=1e-11)


@pytest.mark.parametrize("n_k", [1, 3, 5])
def test_roll_equals_library_circular_same_conv(n_k):
    b, c, j, n = 2, 2, 3, 10
    x = RNG.standard_normal((b, c, n, n))
    k = RNG.standard_normal((c * j, n_k, n_k))
    y, _ = fdc.cic_fdp_layer_forward(x, _spectral_from_spatial(k, n), n, fdc.ARTIFACT_ROLL, n_k)
    p = (n_k - 1) // 2
    xp = F.pad(torch.from_numpy(x), (p, p, p, p), mode="circular")
    ref = F.conv2d(xp, torch.from_numpy(k[:, None, ::-1, ::-1].copy()), groups=c)
    np.testing.assert_allclose(y, ref.numpy(), atol=1e-11)


def test_roll_even_kernel_against_brute_force():
    n, n_k = 8, 4
    x = RNG.standard_normal((1, 1, n, n))
    k = RNG.standard_normal((1, n_k, n_k))
    y, _ = fdc.cic_fdp_layer_forward(x, _spectral_from_spatial(k, n), n, fdc.ARTIFACT_ROLL, n_k)
    circ = conv.circular_convolve(x[0, 0], k[0])
    s = (n_k - 1) // 2
    for i in range(n):
        for jj in range(n):
            assert abs(y[0, 0, i, jj] - circ[(i + s) % n, (jj + s) % n]) < 1e-11


def test_valid_conv_matches_eq1_brute_force():
    # Eq. 1 written out by loops, against the library routine used above.
    x = RNG.standard_normal((7, 9))
    k = RNG.standard_normal((3, 2))
    ref = F.conv2d(torch.from_numpy(x)[None, None], torch.from_numpy(k)[None, None])[0, 0].numpy()
    np.testing.assert_allclose(conv.correlate_valid(x, k), ref, atol=1e-12)


# ---------------------------------------------------------------------------- P6 (FDP)
def _bandlimited(n, m, count=6):
    hh, ww = np.meshgrid(np.arange(n), np.arange(n), indexing="ij")
    x = np.full((n, n), 0.3)
    for _ in range(count):
        fk = RNG.integers(-(m // 2) + 1, m // 2)
        fl = RNG.integers(0, m // 2)
        ph = RNG.random() * 2 * np.pi
        x += RNG.standard_normal() * np.cos(2 * np.pi * (fk * hh + fl * ww) / n + ph)
    return x


@pytest.mark.parametrize("n,m", [(8, 4), (16, 8), (16, 4), (32, 16), (12, 6)])
def test_fdp_of_bandlimited_image_is_scaled_decimation(n, m):
    x = _bandlimited(n, m)
    y = dft.irfft2(fdc.fdp(dft.rfft2(x), m, m), m, m)
    np.testing.assert_allclose(y, (n / m) ** 2 * x[:: n // m, :: n // m], atol=1e-10)


def test_fdp_constant():
    n, m = 16, 8
    y = dft.irfft2(fdc.fdp(dft.rfft2(np.full((n, n), 0.7)), m, m), m, m)
    np.testing.assert_allclose(y, np.full((m, m), 0.7 * 4), atol=1e-12)


def test_fdp_rows_and_columns_kept():
    # Frequency rows f in [-M/2, M/2) and columns 0..M/2 survive, in rfft2 order.
    n, m = 12, 8
    spec = np.arange(n * (n // 2 + 1)).reshape(n, n // 2 + 1).astype(complex)
    out = fdc.fdp(spec, m, m)
    rows = list(range(m // 2)) + list(range(n - m // 2, n))
    np.testing.assert_array_equal(out, spec[rows][:, : m // 2 + 1])


def test_fdp_nonsquare():
    spec = _rand_complex((10, 7))   # H=10, W=12
    out = fdc.fdp(spec, 6, 8)
    rows = [0, 1, 2, 7, 8, 9]
    np.testing.assert_array_equal(out, spec[rows][:, :5])


def test_worked_4x4_fdp(golden):
    g = golden("worked_4x4.txt")
    X = np.array(g["rfft2_x"])
    Z = fdc.fdp(X, 2, 2)
    np.testing.assert_allclose(Z, np.array(g["fdp_2x2_spectrum"]), atol=1e-12)
    np.testing.assert_allclose(dft.irfft2(Z, 2, 2), np.array(g["fdp_2x2_image"]), atol=1e-12)
    x = np.array(g["x"], dtype=float)[None, None]
    K = np.array(g["rfft2_kernel"])[None]
    y, xs = fdc.cic_fdp_layer_forward(x, K, 2)
    np.testing.assert_allclose(y[0, 0], np.array(g["cic_fdp_2x2_image"]), atol=1e-12)
    gy = np.zeros((1, 1, 2, 2))
    gy[0, 0, 0, 0] = 1.0
    gx, gk = fdc.cic_fdp_layer_backward(gy, xs, K, 2)
    expect_gk = np.zeros((4, 3), dtype=complex)
    for (k, l), v in g["cic_fdp_grad_kernel_kept"].items():
        expect_gk[k, l] = v
    np.testing.assert_allclose(gk[0], expect_gk, atol=1e-12)
    np.testing.assert_allclose(gx[0, 0], np.array(g["cic_fdp_grad_x"], dtype=float), atol=1e-12)


# ---------------------------------------------------------------------------- P7
def test_impulse_response():
    n, m = 16, 8
    x = np.zeros((1, 1, n, n))
    x[0, 0, 0, 0] = 1.0
    K = _rand_complex((3, n, n // 2 + 1))
    y, _ = fdc.cic_fdp_layer_forward(x, K, m)
    for o in range(3):
        rows = list(range(m // 2)) + list(range(n - m // 2, n))
        np.testing.assert_allclose(y[0, o], dft.irfft2(K[o][rows][:, : m // 2 + 1], m, m), atol=1e-12)


# ---------------------------------------------------------------------------- P13
def test_shift_equivariance_under_halving():
    n, m, a, b = 16, 8, 3, 1
    x = RNG.standard_normal((1, 2, n, n))
    K = _rand_complex((4, n, n // 2 + 1))
    y, _ = fdc.cic_fdp_layer_forward(x, K, m)
    ys, _ = fdc.cic_fdp_layer_forward(np.roll(x, (2 * a, 2 * b), axis=(-2, -1)), K, m)
    np.testing.assert_allclose(ys, np.roll(y, (a, b), axis=(-2, -1)), atol=1e-11)


def test_linearity():
    n, m = 8, 4
    x1, x2 = RNG.standard_normal((2, 1, 2, n, n))
    K1, K2 = _rand_complex((2, 4, n, n // 2 + 1))
    f = lambda x, K: fdc.cic_fdp_layer_forward(x, K, m)[0]
    np.testing.assert_allclose(f(2 * x1 - 3 * x2, K1), 2 * f(x1, K1) - 3 * f(x2, K1), atol=1e-11)
    np.testing.assert_allclose(f(x1, 1.5 * K1 + 0.5j * K2), 1.5 * f(x1, K1) + f(x1, 0.5j * K2), atol=1e-11)


def test_cic_channel_constraint():
    with pytest.raises(ValueError):
        fdc.cic(_rand_complex((1, 3, 4, 3)), _rand_complex((4, 4, 3)))


# ---------------------------------------------------------------------------- P8
def _rdot(a, b):
    return float(np.sum(np.real(a * np.conj(b))))


def test_step_adjoints():
    n, m = 8, 4
    # FDP
    s = _rand_complex((2, n, n // 2 + 1))
    g = _rand_complex((2, m, m // 2 + 1))
    assert abs(_rdot(fdc.fdp(s, m, m), g) - _rdot(s, fdc.fdp_backward(g, n, n))) < 1e-10
    # CIC, both arguments
    X = _rand_complex((2, 2, n, 5))
    K = _rand_complex((6, n, 5))
    G = _rand_complex((2, 6, n, 5))
    gX, gK = fdc.cic_backward(G, X, K)
    dX = _rand_complex(X.shape)
    dK = _rand_complex(K.shape)
    # the map is bilinear: d/dt <cic(X + t dX, K + t dK), G> at t=0
    lin = _rdot(fdc.cic(dX, K), G) + _rdot(fdc.cic(X, dK), G)
    assert abs(lin - (_rdot(dX, gX) + _rdot(dK, gK))) < 1e-9
    # artifact handling
    for mode, nk in ((fdc.ARTIFACT_CROP, 3), (fdc.ARTIFACT_ROLL, 4), (fdc.ARTIFACT_NONE, 1)):
        y = RNG.standard_normal((2, n, n))
        gy = RNG.standard_normal(fdc.artifact_apply(y, mode, nk).shape)
        assert abs(np.sum(fdc.artifact_apply(y, mode, nk) * gy)
                   - np.sum(y * fdc.artifact_backward(gy, mode, nk, n, n))) < 1e-10


@pytest.mark.parametrize("mode,nk", [(fdc.ARTIFACT_NONE, 1), (fdc.ARTIFACT_CROP, 3), (fdc.ARTIFACT_ROLL, 3)])
def test_layer_adjoint_in_x(mode, nk):
    n, m = 8, 4
    K = _rand_complex((4, n, n // 2 + 1))
    x = RNG.standard_normal((2, 2, n, n))
    y, xs = fdc.cic_fdp_layer_forward(x, K, m, mode, nk)
    gy = RNG.standard_normal(y.shape)
    gx, _ = fdc.cic_fdp_layer_backward(gy, xs, K, m, mode, nk)
    assert abs(np.sum(y * gy) - np.sum(x * gx)) < 1e-9


# ---------------------------------------------------------------------------- P9
@pytest.mark.parametrize("n,m", [(4, 2), (8, 4), (8, 8)])
def test_layer_gradients_finite_difference(n, m):
    c, j, b = 2, 2, 2
    x = RNG.standard_normal((b, c, n, n))
    K = _rand_complex((c * j, n, n // 2 + 1))
    gy = RNG.standard_normal((b, c * j, m, m))
    _, xs = fdc.cic_fdp_layer_forward(x, K, m)
    gx, gk = fdc.cic_fdp_layer_backward(gy, xs, K, m)
    loss = lambda xx, KK: float(np.sum(fdc.cic_fdp_layer_forward(xx, KK, m)[0] * gy))
    eps = 1e-6
    for idx in [(0, 0, 0), (1, 1, n // 2), (2, n - 1, n // 2), (3, n // 2, 1), (0, m // 2, m // 2),
                (1, n - m // 2, m // 2), (2, m // 2 - 1, 0)]:
        for unit, part in ((1.0, np.real), (1j, np.imag)):
            Kp, Km = K.copy(), K.copy()
            Kp[idx] += eps * unit
            Km[idx] -= eps * unit
            fd = (loss(x, Kp) - loss(x, Km)) / (2 * eps)
            assert abs(fd - part(gk[idx])) < 1e-7, (idx, fd, gk[idx])
    for idx in [(0, 0, 0, 0), (1, 1, n - 1, 2), (0, 1, 2, n - 1)]:
        xp, xm = x.copy(), x.copy()
        xp[idx] += eps
        xm[idx] -= eps
        fd = (loss(xp, K) - loss(xm, K)) / (2 * eps)
        assert abs(fd - gx[idx]) < 1e-7


def test_layer_gradients_finite_difference_crop_mode():
    n, m, nk = 8, 8, 3
    x = RNG.standard_normal((1, 1, n, n))
    K = _rand_complex((2, n, n // 2 + 1))
    y, xs = fdc.cic_fdp_layer_forward(x, K, m, fdc.ARTIFACT_CROP, nk)
    gy = RNG.standard_normal(y.shape)
    gx, gk = fdc.cic_fdp_layer_backward(gy, xs, K, m, fdc.ARTIFACT_CROP, nk)
    loss = lambda KK: float(np.sum(fdc.cic_fdp_layer_forward(x, KK, m, fdc.ARTIFACT_CROP, nk)[0] * gy))
    eps = 1e-6
    for idx in [(0, 1, 2), (1, 5, 4), (0, 0, 0)]:
        Kp, Km = K.copy(), K.copy()
        Kp[idx] += eps
        Km[idx] -= eps
        assert abs((loss(Kp) - loss(Km)) / (2 * eps) - gk[idx].real) < 1e-7


def test_dropped_bins_get_zero_kernel_gradient():
    n, m = 8, 4
    x = RNG.standard_normal((2, 1, n, n))
    K = _rand_complex((2, n, n // 2 + 1))
    y, xs = fdc.cic_fdp_layer_forward(x, K, m)
    _, gk = fdc.cic_fdp_layer_backward(RNG.standard_normal(y.shape), xs, K, m)
    kept = np.zeros((n, n // 2 + 1), bool)
    kept[list(range(m // 2)) + list(range(n - m // 2, n)), : m // 2 + 1] = True
    assert np.all(gk[:, ~kept] == 0)
    assert np.all(np.abs(gk[:, kept]) > 0)


# ---------------------------------------------------------------------------- P10
def test_round_trip_stack_equals_projected_spectral_chain():
    sizes = (32, 16, 8, 4)
    chans = (1, 2, 4, 8)
    x = RNG.standard_normal((2, 1, 32, 32))
    Ks = [0.1 * _rand_complex((chans[i + 1], sizes[i], sizes[i] // 2 + 1)) for i in range(3)]
    y, _ = fdc.cic_stack_forward(x, Ks, sizes)
    yc = fdc.cic_spectral_chain(x, Ks, sizes)
    np.testing.assert_allclose(y, yc, atol=1e-12 * np.abs(y).max() + 1e-15)


def test_stack_gradients_finite_difference():
    sizes = (8, 4, 2)
    chans = (1, 2, 4)
    x = RNG.standard_normal((2, 1, 8, 8))
    Ks = [_rand_complex((chans[i + 1], sizes[i], sizes[i] // 2 + 1)) for i in range(2)]
    y, saved = fdc.cic_stack_forward(x, Ks, sizes)
    gy = RNG.standard_normal(y.shape)
    gks, gx = fdc.cic_stack_backward(gy, saved, Ks, sizes, want_input_grad=True)
    eps = 1e-6

    def loss(KK, xx=x):
        return float(np.sum(fdc.cic_stack_forward(xx, KK, sizes)[0] * gy))

    for li, idx in [(0, (1, 7, 1)), (0, (0, 0, 0)), (1, (3, 1, 1)), (1, (2, 0, 1))]:
        for unit, part in ((1.0, np.real), (1j, np.imag)):
            Kp = [k.copy() for k in Ks]
            Km = [k.copy() for k in Ks]
            Kp[li][idx] += eps * unit
            Km[li][idx] -= eps * unit
            assert abs((loss(Kp) - loss(Km)) / (2 * eps) - part(gks[li][idx])) < 1e-7
    xp, xm = x.copy(), x.copy()
    xp[1, 0, 3, 5] += eps
    xm[1, 0, 3, 5] -= eps
    assert abs((loss(Ks, xp) - loss(Ks, xm)) / (2 * eps) - gx[1, 0, 3, 5]) < 1e-7


# ---------------------------------------------------------------------------- FDCNN chain
def test_chain_single_layer_is_the_layer():
    x = RNG.standard_normal((2, 1, 16, 16))
    K = [0.1 * _rand_complex((3, 16, 9))]
    y, _ = fdc.cic_chain_forward(x, K, (16, 8))
    ref, _ = fdc.cic_fdp_layer_forward(x, K[0], 8)
    np.testing.assert_allclose(y, ref, atol=1e-13)


def test_chain_of_a_cosine_is_a_cosine():
    """A single frequency (p, q) inside every pooled band passes every layer as one
    bin: the output of channel o is (2 / M^2) |V| cos(2 pi (p h + q w) / M + arg V) with
    V = (N0^2 / 2) times the product of each layer's kernel at that frequency, read at
    (p mod N_i, q) for the channel o's ancestor in layer i (CIC: channel o of a layer
    reads input channel o // J)."""
    sizes, chans = (32, 16, 8), (1, 2, 4)
    n0, m = sizes[0], sizes[-1]
    p, q = 3, 2
    hh, ww = np.meshgrid(np.arange(n0), np.arange(n0), indexing="ij")
    x = np.cos(2 * np.pi * (p * hh + q * ww) / n0)[None, None]
    Ks = [_rand_complex((chans[i + 1], sizes[i], sizes[i] // 2 + 1)) for i in range(2)]
    y, _ = fdc.cic_chain_forward(x, Ks, sizes)
    hm, wm = np.meshgrid(np.arange(m), np.arange(m), indexing="ij")
    for o in range(chans[-1]):
        v = n0 * n0 / 2.0
        ch = o
        for i in reversed(range(2)):
            v = v * Ks[i][ch, p % sizes[i], q]
            ch = ch // (chans[i + 1] // chans[i])
        expect = (2.0 / (m * m)) * np.abs(v) * np.cos(2 * np.pi * (p * hm + q * wm) / m + np.angle(v))
        np.testing.assert_allclose(y[0, o], expect, atol=1e-9 * np.abs(v) / (m * m))


def test_chain_backward_is_the_adjoint():
    sizes, chans = (16, 8, 4), (1, 2, 4)
    x = RNG.standard_normal((2, 1, 16, 16))
    Ks = [_rand_complex((chans[i + 1], sizes[i], sizes[i] // 2 + 1)) for i in range(2)]
    y, saved = fdc.cic_chain_forward(x, Ks, sizes)
    gy = RNG.standard_normal(y.shape)
    gks, gx = fdc.cic_chain_backward(gy, saved, Ks, sizes, want_input_grad=True)
    # linear in x: <y(dx), gy> = <dx, gx>
    dx = RNG.standard_normal(x.shape)
    ydx, _ = fdc.cic_chain_forward(dx, Ks, sizes)
    np.testing.assert_allclose(np.sum(ydx * gy), np.sum(dx * gx), rtol=1e-10)
    # finite differences in Re and Im of kernel entries of both layers
    eps = 1e-6
    for li, (o, k, l) in [(0, (1, 3, 2)), (0, (0, 15, 0)), (1, (3, 1, 1)), (1, (2, 7, 4))]:
        for comp in (1.0, 1j):
            Kp = [k_.copy() for k_ in Ks]
            Km = [k_.copy() for k_ in Ks]
            Kp[li][o, k, l] += eps * comp
            Km[li][o, k, l] -= eps * comp
            yp, _ = fdc.cic_chain_forward(x, Kp, sizes)
            ym, _ = fdc.cic_chain_forward(x, Km, sizes)
            fd = np.sum((yp - ym) * gy) / (2 * eps)
            an = gks[li][o, k, l].real if comp == 1.0 else gks[li][o, k, l].imag
            np.testing.assert_allclose(an, fd, rtol=1e-6, atol=1e-9)


# ---------------------------------------------------------------------------- spatial kernels
@pytest.mark.parametrize("n,artifact", [(3, fdc.ARTIFACT_CROP), (5, fdc.ARTIFACT_CROP), (3, fdc.ARTIFACT_ROLL)])
def test_spatial_cic_is_depthwise_convolution(n, artifact):
    """Without pooling the spatial-kernel CIC layer is a depthwise convolution with
    channel multiplier J and flipped kernels (valid for CROP, circular same-size for
    ROLL); its weight gradient is the library's autograd gradient of that convolution."""
    B, C, J, N = 2, 2, 3, 16
    x = RNG.standard_normal((B, C, N, N))
    w = RNG.standard_normal((C * J, n, n))
    y, xs = fdc.cic_spatial_layer_forward(x, w, N, artifact)
    xt = torch.from_numpy(x)
    if artifact == fdc.ARTIFACT_ROLL:
        p = (n - 1) // 2
        xt = F.pad(xt, (p, n - 1 - p, p, n - 1 - p), mode="circular")
    wt = torch.from_numpy(w[:, None, ::-1, ::-1].copy()).requires_grad_(True)
    ref = F.conv2d(xt, wt, groups=C)
    np.testing.assert_allclose(y, ref.detach().numpy(), atol=1e-10)
    gy = RNG.standard_normal(y.shape)
    ref.backward(torch.from_numpy(gy))
    _, gw = fdc.cic_spatial_layer_backward(gy, xs, w, N, artifact, want_gx=False)
    np.testing.assert_allclose(gw, wt.grad.numpy()[:, 0, ::-1, ::-1], atol=1e-9)
