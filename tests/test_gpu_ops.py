"""GPU parity of the standalone ops against the float64 oracle: the 2-D real FFT
plans and their adjoints (section 2.4.1.1), spectral CIC (Eq. 5) and FDP
(section 2.4.2).  Sizes span single-thread transforms (2..16), one and two
Stockham passes, the radix-7 length 224, non-square images and ragged column
tiles."""

import zlib

import numpy as np
import pytest
import torch

from _parity import assert_parity, to_np
from oracle import dft, fdc
from paper_2106_12736_amd import layers

pytestmark = pytest.mark.gpu

FFT_SIZES = [(2, 2), (4, 4), (8, 16), (16, 8), (32, 32), (64, 64), (128, 128), (256, 256), (512, 512),
             (1024, 1024), (224, 224), (224, 64), (1024, 32), (32, 1024), (64, 224)]


def _rng(*key):
    return np.random.default_rng(zlib.crc32(repr(key).encode()))


def _crand(rng, shape):
    return (rng.standard_normal(shape) + 1j * rng.standard_normal(shape)).astype(np.complex64)


def _gpu(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.mark.parametrize("h,w", FFT_SIZES)
def test_fft_plan_forward_inverse_and_adjoints(h, w):
    print(f"fft plan {h}x{w}", flush=True)
    rng = _rng("fft", h, w)
    count = 3
    plan = layers.FftPlan(count, h, w)
    x = rng.standard_normal((count, h, w)).astype(np.float32)
    Y = _crand(rng, (count, h, w // 2 + 1))  # not Hermitian: exercises the real-part semantics
    x64, Y128 = x.astype(np.float64), Y.astype(np.complex128)

    assert_parity(to_np(plan.rfft2(_gpu(x))), dft.rfft2(x64), "rfft2")
    assert_parity(to_np(plan.irfft2(_gpu(Y))), dft.irfft2(Y128, h, w), "irfft2")
    assert_parity(to_np(plan.rfft2_backward(_gpu(Y))), dft.rfft2_adjoint(Y128, h, w), "rfft2_backward")
    assert_parity(to_np(plan.irfft2_backward(_gpu(x))), dft.irfft2_adjoint(x64), "irfft2_backward")
    torch.cuda.synchronize()


@pytest.mark.parametrize("n,count", [(16, 2051), (32, 1029), (32, 1), (64, 2050), (64, 1027)])
def test_fft_small_planes_many_per_workgroup(n, count):
    # square planes up to 64 x 64 take one launch per transform with 1, 2 or 4 planes per
    # workgroup (by batch size); ragged counts leave a partly filled last workgroup
    print(f"fft small {n} x {count}", flush=True)
    rng = _rng("fft_small", n, count)
    plan = layers.FftPlan(count, n, n)
    x = rng.standard_normal((count, n, n)).astype(np.float32)
    Y = _crand(rng, (count, n, n // 2 + 1))
    x64, Y128 = x.astype(np.float64), Y.astype(np.complex128)
    assert_parity(to_np(plan.rfft2(_gpu(x))), dft.rfft2(x64), "rfft2")
    assert_parity(to_np(plan.irfft2(_gpu(Y))), dft.irfft2(Y128, n, n), "irfft2")
    assert_parity(to_np(plan.rfft2_backward(_gpu(Y))), dft.rfft2_adjoint(Y128, n, n), "rfft2_backward")
    assert_parity(to_np(plan.irfft2_backward(_gpu(x))), dft.irfft2_adjoint(x64), "irfft2_backward")
    torch.cuda.synchronize()


@pytest.mark.parametrize("count,h,w,mh,mw", [
    (3, 1024, 1024, 512, 512),  # the first layer of the 1024 stack
    (5, 512, 512, 256, 256), (2, 256, 256, 128, 128), (4, 128, 128, 64, 64),
    (3, 224, 224, 112, 112),    # radix-7 lengths
    (2, 128, 64, 32, 48),       # non-square, different kept heights and widths
    (2, 256, 256, 2, 2),        # one kept row at each end, two kept columns
    (2, 128, 128, 128, 64),     # every row kept
    (2, 256, 128, 64, 128),     # every column kept
    (3, 512, 512, 512, 512),    # everything kept: fdc_rfft2
    (7, 32, 32, 16, 16),        # one-launch size: every bin formed
    (1, 8, 16, 4, 8),
])
def test_rfft2_pooled(count, h, w, mh, mw):
    print(f"rfft2_pooled {count} x {h}x{w} -> {mh}x{mw}", flush=True)
    rng = _rng("rfft2_pooled", count, h, w, mh, mw)
    plan = layers.FftPlan(count, h, w)
    x = rng.standard_normal((count, h, w)).astype(np.float32)
    nan = float("nan")
    out = torch.full((count, h, w // 2 + 1), complex(nan, nan), dtype=torch.complex64, device="cuda")
    got = to_np(plan.rfft2_pooled(_gpu(x), mh, mw, out=out))
    ref = dft.rfft2(x.astype(np.float64))
    rows = np.r_[0:mh // 2, h - mh // 2:h]
    cols = np.arange(mw // 2 + 1)
    # the kept bins only: the others are undefined (left as they were, or row-pass values)
    assert_parity(got[:, rows][:, :, cols], ref[:, rows][:, :, cols], "kept bins")
    # with a workspace (rows in runs of 8 bins there, tiled column reads): the same bits
    ws = torch.empty(count * h * (mw // 2 + 1) * 8, dtype=torch.uint8, device="cuda")
    out2 = torch.full((count, h, w // 2 + 1), complex(nan, nan), dtype=torch.complex64, device="cuda")
    got2 = to_np(plan.rfft2_pooled(_gpu(x), mh, mw, out=out2, ws=ws))
    assert np.array_equal(got2[:, rows][:, :, cols], got[:, rows][:, :, cols])
    torch.cuda.synchronize()


@pytest.mark.parametrize("count,H,W", [(1, 2, 2), (3, 8, 8), (2, 16, 32), (5, 64, 32), (4, 224, 224), (2, 1024, 1024)])
def test_hermitian_project(count, H, W):
    rng = _rng("pi_h", count, H, W)
    Y = _crand(rng, (count, H, W // 2 + 1))
    got = to_np(layers.hermitian_project(_gpu(Y)))
    ref = dft.hermitian_projection(Y.astype(np.complex128))
    assert_parity(got, ref, "Pi_H")
    # untouched columns are bit-exact copies, and the projected columns are Hermitian exactly
    assert np.array_equal(got[..., 1:-1], Y[..., 1:-1])
    neg = (-np.arange(H)) % H
    for l in (0, W // 2):
        assert np.array_equal(got[..., :, l], np.conj(got[..., neg, l]))
    # Pi_H(irfft2's input) leaves irfft2 unchanged, and rfft2 of a real image is a fixed point
    plan = layers.FftPlan(count, H, W)
    assert_parity(to_np(plan.irfft2(_gpu(got))), dft.irfft2(Y.astype(np.complex128), H, W), "irfft2(Pi_H Y)")
    X = to_np(plan.rfft2(_gpu(rng.standard_normal((count, H, W)).astype(np.float32))))
    assert_parity(to_np(layers.hermitian_project(_gpu(X))), X.astype(np.complex128), "Pi_H(rfft2 x)")
    torch.cuda.synchronize()


def test_fft_structured_inputs():
    # impulse, constant and a single cosine through the 1024 x 1024 plan
    h = w = 1024
    plan = layers.FftPlan(3, h, w)
    x = np.zeros((3, h, w), np.float32)
    x[0, 5, 7] = 1.0
    x[1] = 0.25
    hh, ww = np.meshgrid(np.arange(h), np.arange(w), indexing="ij")
    x[2] = np.cos(2 * np.pi * (3 * hh / h + 17 * ww / w)).astype(np.float32)
    got = to_np(plan.rfft2(_gpu(x)))
    assert_parity(got, dft.rfft2(x.astype(np.float64)), "rfft2 structured")
    back = to_np(plan.irfft2(_gpu(got)))
    assert_parity(back, x.astype(np.float64), "round trip")


@pytest.mark.parametrize("B,C,S,H,W", [(2, 1, 4, 8, 8), (3, 2, 6, 16, 10), (1, 4, 8, 64, 64), (4, 3, 3, 7, 9)])
def test_cic_spectral(B, C, S, H, W):
    rng = _rng("cic", B, C, S, H, W)
    Wf = W // 2 + 1 if W % 2 == 0 else W  # spectral ops take any [H][Wf] grid
    X = _crand(rng, (B, C, H, Wf))
    K = _crand(rng, (S, H, Wf))
    gY = _crand(rng, (B, S, H, Wf))
    Y = layers.cic_forward(_gpu(X), _gpu(K))
    assert_parity(to_np(Y), fdc.cic(X.astype(np.complex128), K.astype(np.complex128)), "cic")
    gX, gK = layers.cic_backward(_gpu(gY), _gpu(X), _gpu(K))
    rgX, rgK = fdc.cic_backward(gY.astype(np.complex128), X.astype(np.complex128), K.astype(np.complex128))
    assert_parity(to_np(gX), rgX, "cic gX")
    assert_parity(to_np(gK), rgK, "cic gK")
    gX2, gK2 = layers.cic_backward(_gpu(gY), _gpu(X), _gpu(K))
    assert torch.equal(gK, gK2) and torch.equal(gX, gX2), "gradients must be bitwise reproducible"


@pytest.mark.parametrize("count,H,W,Mh,Mw", [(3, 8, 8, 4, 4), (2, 16, 16, 16, 16), (5, 12, 10, 6, 8),
                                             (2, 1024, 1024, 512, 512), (7, 64, 64, 2, 2)])
def test_fdp(count, H, W, Mh, Mw):
    rng = _rng("fdp", count, H, W, Mh, Mw)
    X = _crand(rng, (count, H, W // 2 + 1))
    Y = layers.fdp_forward(_gpu(X), Mh, Mw)
    ref = fdc.fdp(X.astype(np.complex128), Mh, Mw)
    np.testing.assert_array_equal(to_np(Y), ref.astype(np.complex64))  # a pure gather: bit-exact
    gY = _crand(rng, (count, Mh, Mw // 2 + 1))
    gX = layers.fdp_backward(_gpu(gY), H, W)
    np.testing.assert_array_equal(to_np(gX), fdc.fdp_backward(gY.astype(np.complex128), H, W).astype(np.complex64))
