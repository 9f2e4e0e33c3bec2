"""FDC, FDP, artifact handling and Full FDC, forward and backward, in float64.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Layouts follow the library's: activations [B][C][H][W] real, spectra
[B][C][H][W/2+1] complex in unshifted rfft2 order, CIC kernels [S][H][W/2+1]
complex, Full FDC weights [S][C][n][n] real.

Readings of the paper taken here (each is listed with its reason in the
design notes of the repository):

* Channel order of CIC (Eq. 5): output channel o = c*J + j reads input
  channel c = o // J and kernel o; J = S / C, S mod C = 0.
* FDP (section 2.4.2): RFFT shift (swap the two row halves), remove the same
  number of rows from top and bottom and of columns from the right, shift back.
  No rescaling: the crop is a pure slice.
* Artifact handling (section 2.4.1.3): "crop" cuts n-1 rows/columns from the
  top and left; "roll" moves the artifact to all edges by shifting the image
  by s = (n-1)//2 so that out[i, j] = y[(i+s) mod H, (j+s) mod W].
* Full FDC: the per-bin product sums over input channels (the convolution over
  volume of Eq. 2, done in the frequency domain by Eq. 4); kernels are n x n
  spatial weights padded at the top-left corner to the image size and
  transformed with the RFFT on every call (section 2.4.1.2, Algorithm 1).
* Gradients of complex quantities use dL/dRe + i dL/dIm.  For a product
  Z = X K this gives dL/dX = G conj(K) and dL/dK = G conj(X).
"""

import numpy as np

from . import dft

ARTIFACT_NONE = "none"
ARTIFACT_CROP = "crop"
ARTIFACT_ROLL = "roll"


# ----------------------------------------------------------------------------
# Channel Independent Convolution (section 2.4.1.4, Eq. 5, Algorithm 1)
# ----------------------------------------------------------------------------

def cic(x_spec, k_spec):
    """CIC_c = concatenation over j of X_c o K_{c,j}  (Eq. 5).

    x_spec [B][C][H][Wf], k_spec [S][H][Wf] with S mod C = 0 -> [B][S][H][Wf].
    """
    b, c = x_spec.shape[:2]
    s = k_spec.shape[0]
    if s % c:
        raise ValueError("CIC needs S mod C == 0")
    j_fac = s // c
    out = np.empty((b, s) + x_spec.shape[2:], dtype=np.complex128)
    for ci in range(c):
        for j in range(j_fac):
            out[:, ci * j_fac + j] = x_spec[:, ci] * k_spec[ci * j_fac + j]
    return out


def cic_backward(g_spec, x_spec, k_spec):
    """Gradients of ``cic``: (dL/dX [B][C][H][Wf], dL/dK [S][H][Wf]).

    dL/dK[o] = sum_b G[b, o] conj(X[b, o // J]);
    dL/dX[b, c] = sum_j G[b, c J + j] conj(K[c J + j]).
    """
    b, c = x_spec.shape[:2]
    s = k_spec.shape[0]
    j_fac = s // c
    gx = np.zeros(x_spec.shape, dtype=np.complex128)
    gk = np.zeros(k_spec.shape, dtype=np.complex128)
    for ci in range(c):
        for j in range(j_fac):
            o = ci * j_fac + j
            gk[o] = np.sum(g_spec[:, o] * np.conj(x_spec[:, ci]), axis=0)
            gx[:, ci] += g_spec[:, o] * np.conj(k_spec[o])
    return gx, gk


# ----------------------------------------------------------------------------
# Frequency Domain Pooling (section 2.4.2)
# ----------------------------------------------------------------------------

def rfft_shift(spec):
    """RFFT shift (section 2.4.2.2): split the rows in two halves and swap them."""
    h = spec.shape[-2]
    if h % 2:
        raise ValueError("even number of rows only")
    return np.concatenate([spec[..., h // 2:, :], spec[..., : h // 2, :]], axis=-2)


def rfft_unshift(spec):
    """Inverse of ``rfft_shift`` (for an even row count the same swap)."""
    h = spec.shape[-2]
    return np.concatenate([spec[..., h - h // 2:, :], spec[..., : h - h // 2, :]], axis=-2)


def fdp(spec, mh, mw):
    """FDP (section 2.4.2.1): hard rectangular crop of the shifted half spectrum.

    spec [..][H][W/2+1] -> [..][mh][mw/2+1].  After the RFFT shift the low
    frequencies sit in the middle of the left edge; (H - mh)/2 rows are removed
    from the top and from the bottom, and (W - mw)/2 columns from the right.
    The result is shifted back so it is again in unshifted rfft2 order.
    """
    h, wf = spec.shape[-2:]
    w = 2 * (wf - 1)
    _check_pool(h, w, mh, mw)
    r = (h - mh) // 2
    shifted = rfft_shift(spec)
    cropped = shifted[..., r: h - r, : mw // 2 + 1]
    return rfft_unshift(cropped)


def fdp_backward(g, h, w):
    """Adjoint of ``fdp``: undo each step in reverse (shift back, zero-pad, unshift)."""
    mh, mwf = g.shape[-2:]
    mw = 2 * (mwf - 1)
    _check_pool(h, w, mh, mw)
    r = (h - mh) // 2
    g_shifted = rfft_shift(g)          # adjoint of rfft_unshift on mh rows
    padded = np.zeros(g.shape[:-2] + (h, w // 2 + 1), dtype=np.complex128)
    padded[..., r: h - r, : mw // 2 + 1] = g_shifted
    return rfft_unshift(padded)        # adjoint of rfft_shift on h rows


def _check_pool(h, w, mh, mw):
    for v in (h, w, mh, mw):
        if v <= 0 or v % 2:
            raise ValueError("FDP sizes must be positive and even")
    if mh > h or mw > w:
        raise ValueError("FDP output larger than its input")


# ----------------------------------------------------------------------------
# Convolution artifact handling (section 2.4.1.3)
# ----------------------------------------------------------------------------

def artifact_apply(y, mode, n):
    """Remove (crop) or redistribute (roll) the wrap-around artifact of an n x n kernel."""
    if mode == ARTIFACT_NONE:
        return y
    if mode == ARTIFACT_CROP:
        return y[..., n - 1:, n - 1:]
    if mode == ARTIFACT_ROLL:
        s = (n - 1) // 2
        return np.roll(y, shift=(-s, -s), axis=(-2, -1))
    raise ValueError(mode)


def artifact_backward(g, mode, n, h, w):
    """Adjoint of ``artifact_apply`` back to an h x w image."""
    if mode == ARTIFACT_NONE:
        return g
    if mode == ARTIFACT_CROP:
        out = np.zeros(g.shape[:-2] + (h, w))
        out[..., n - 1:, n - 1:] = g
        return out
    if mode == ARTIFACT_ROLL:
        s = (n - 1) // 2
        return np.roll(g, shift=(s, s), axis=(-2, -1))
    raise ValueError(mode)


# ----------------------------------------------------------------------------
# One CIC + FDP layer on spatial activations: rfft2 -> CIC -> FDP -> irfft2
# ----------------------------------------------------------------------------

def cic_fdp_layer_forward(x, k_spec, m, artifact=ARTIFACT_NONE, n=1):
    """Spatial x [B][C][N][N] -> y [B][S][M][M] (before artifact handling).

    Steps in the paper's order: RFFT of the image (section 2.4.1.1), FDC with
    CIC against the given spectral kernels (Algorithm 1, Eq. 5), FDP crop
    (section 2.4.2), IRFFT, artifact handling (section 2.4.1.3).
    Returns (y, x_spec) -- x_spec is what the backward pass needs.
    """
    x_spec = dft.rfft2(x)
    z = cic(x_spec, k_spec)
    zp = fdp(z, m, m)
    y = dft.irfft2(zp, m, m)
    return artifact_apply(y, artifact, n), x_spec


def cic_fdp_layer_backward(gy, x_spec, k_spec, m, artifact=ARTIFACT_NONE, n=1, want_gx=True):
    """Reverse of ``cic_fdp_layer_forward``: returns (gx [B][C][N][N] or None, gK [S][N][N/2+1])."""
    nh = x_spec.shape[-2]
    nw = 2 * (x_spec.shape[-1] - 1)
    g = artifact_backward(gy, artifact, n, m, m)
    g_zp = dft.irfft2_adjoint(g)
    g_z = fdp_backward(g_zp, nh, nw)
    g_xs, g_k = cic_backward(g_z, x_spec, k_spec)
    gx = dft.rfft2_adjoint(g_xs, nh, nw) if want_gx else None
    return gx, g_k


def cic_stack_forward(x, kernels, sizes):
    """A stack of CIC+FDP layers; layer i maps size sizes[i] -> sizes[i+1].

    Returns (y, saved) where saved[i] = (x_spec_i, m_i) for the backward pass.
    """
    saved = []
    h = x
    for i, k in enumerate(kernels):
        m = sizes[i + 1]
        h, xs = cic_fdp_layer_forward(h, k, m)
        saved.append(xs)
    return h, saved


def cic_stack_backward(gy, saved, kernels, sizes, want_input_grad=False):
    """Backward of ``cic_stack_forward``; returns (list of gK per layer, gx of the input or None)."""
    gks = [None] * len(kernels)
    g = gy
    for i in reversed(range(len(kernels))):
        need_gx = want_input_grad or i > 0
        g, gks[i] = cic_fdp_layer_backward(g, saved[i], kernels[i], sizes[i + 1], want_gx=need_gx)
    return gks, g


def cic_spectral_chain(x, kernels, sizes):
    """Alternative formulation used as a cross-check: transform once, stay in the
    frequency domain through every layer, apply the Hermitian projection that
    the round trip implies after each layer, and invert once at the end.
    """
    spec = dft.rfft2(x)
    for i, k in enumerate(kernels):
        m = sizes[i + 1]
        spec = dft.hermitian_projection(fdp(cic(spec, k), m, m))
    m = sizes[-1]
    return dft.irfft2(spec, m, m)


# ----------------------------------------------------------------------------
# CIC with spatial kernels (section 2.4.1.2): n x n kernels transformed on every call
# ----------------------------------------------------------------------------

def cic_spatial_layer_forward(x, w, m, artifact=ARTIFACT_NONE):
    """Algorithm 1 with the kernel steps: w [S][n][n] padded to N x N at the top-left
    and transformed, then the CIC + FDP layer.  Returns (y, x_spec)."""
    n_img = x.shape[-1]
    k_spec = kernel_spectrum(w, n_img, n_img)
    return cic_fdp_layer_forward(x, k_spec, m, artifact, w.shape[-1])


def cic_spatial_layer_backward(gy, x_spec, w, m, artifact=ARTIFACT_NONE, want_gx=True):
    """Reverse of ``cic_spatial_layer_forward``: (gx or None, gw [S][n][n])."""
    n_img = x_spec.shape[-2]
    n = w.shape[-1]
    k_spec = kernel_spectrum(w, n_img, n_img)
    gx, g_k = cic_fdp_layer_backward(gy, x_spec, k_spec, m, artifact, n, want_gx)
    return gx, kernel_spectrum_backward(g_k, n)


# ----------------------------------------------------------------------------
# FDCNN data flow (section 2.5.1): one RFFT before all FDC/FDP layers, one IRFFT after
# ----------------------------------------------------------------------------

def cic_chain_forward(x, kernels, sizes):
    """The FDCNN of section 2.5.1: RFFT once, then every FDC (CIC, Eq. 5) and FDP layer
    on spectra (Algorithm 1's spectral in/out form), then IRFFT once.  No projection
    between layers.  Returns (y, saved) with saved[i] = layer i's input spectrum."""
    spec = dft.rfft2(x)
    saved = []
    for i, k in enumerate(kernels):
        saved.append(spec)
        m = sizes[i + 1]
        spec = fdp(cic(spec, k), m, m)
    m = sizes[-1]
    return dft.irfft2(spec, m, m), saved


def cic_chain_backward(gy, saved, kernels, sizes, want_input_grad=False):
    """Reverse of ``cic_chain_forward``: (list of dL/dK per layer, dL/dx or None)."""
    g = dft.irfft2_adjoint(gy)
    gks = [None] * len(kernels)
    for i in reversed(range(len(kernels))):
        n = sizes[i]
        gz = fdp_backward(g, n, n)
        g, gks[i] = cic_backward(gz, saved[i], kernels[i])
    gx = dft.rfft2_adjoint(g, sizes[0], sizes[0]) if want_input_grad else None
    return gks, gx


# ----------------------------------------------------------------------------
# Full FDC (Algorithm 2) with the convolution-over-volume sum of Eq. 2 per bin
# ----------------------------------------------------------------------------

def kernel_spectrum(w, h, wd):
    """Algorithm 1's kernel steps: pad n x n kernels to h x wd (top-left corner), then RFFT."""
    n0, n1 = w.shape[-2:]
    padded = np.zeros(w.shape[:-2] + (h, wd))
    padded[..., :n0, :n1] = w
    return dft.rfft2(padded)


def kernel_spectrum_backward(g_k, n):
    """Adjoint of ``kernel_spectrum``: adjoint RFFT, then keep the n x n support."""
    h = g_k.shape[-2]
    wd = 2 * (g_k.shape[-1] - 1)
    return dft.rfft2_adjoint(g_k, h, wd)[..., :n, :n]


def cov_spectral(x_spec, k_spec):
    """Y[b, s] = sum_c X[b, c] o K[s, c] at every bin (Eq. 2 via Eq. 4)."""
    return np.einsum("bchw,schw->bshw", x_spec, k_spec)


def cov_spectral_backward(g_spec, x_spec, k_spec):
    """(dL/dX [B][C][..], dL/dK [S][C][..]) of ``cov_spectral``."""
    gx = np.einsum("bshw,schw->bchw", g_spec, np.conj(k_spec))
    gk = np.einsum("bshw,bchw->schw", g_spec, np.conj(x_spec))
    return gx, gk


def full_fdc_forward(x, w, artifact=ARTIFACT_CROP):
    """Algorithm 2: RFFT the image, per-bin contraction with the kernel spectra,
    IRFFT, artifact handling.  x [B][C][P][P], w [S][C][n][n] -> y.
    Returns (y, x_spec)."""
    p = x.shape[-1]
    n = w.shape[-1]
    x_spec = dft.rfft2(x)
    k_spec = kernel_spectrum(w, p, p)
    y = dft.irfft2(cov_spectral(x_spec, k_spec), p, p)
    return artifact_apply(y, artifact, n), x_spec


def full_fdc_backward(gy, x_spec, w, artifact=ARTIFACT_CROP, want_gx=True):
    """Reverse of ``full_fdc_forward``: (gx or None, gw [S][C][n][n])."""
    p = x_spec.shape[-2]
    n = w.shape[-1]
    k_spec = kernel_spectrum(w, p, p)
    g = artifact_backward(gy, artifact, n, p, p)
    g_spec = dft.irfft2_adjoint(g)
    g_xs, g_k = cov_spectral_backward(g_spec, x_spec, k_spec)
    gw = kernel_spectrum_backward(g_k, n)
    gx = dft.rfft2_adjoint(g_xs, p, p) if want_gx else None
    return gx, gw
