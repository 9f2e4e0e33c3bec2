"""2-D real DFT, its inverse, and their adjoints, written out from the definition.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Section 2.4.1.1 of the paper transforms real images with the real-to-complex
FFT: the spectrum of an N-row, W-column real image is Hermitian symmetric, so
only the columns l = 0 .. W/2 are kept (N x (W/2+1) complex values).  The paper
computes it with PyTorch's ``rfft2``/``irfft2``; the sign and scaling below are
that convention (forward e^{-2 pi i}, unnormalised; inverse scaled by 1/(H W)).

Everything here is the plain definition evaluated with explicit DFT matrices
(an O(n^2) matrix per 1-D DFT, applied with a library matmul).  Twiddle exponents
are reduced modulo n as exact integers before scaling, so the matrices carry no
accumulated phase error.
"""

import numpy as np


def dft_matrix(n, sign):
    """E[a, b] = exp(sign * 2 pi i * (a b mod n) / n) for a, b in [0, n)."""
    a = np.arange(n)
    return np.exp(sign * 2j * np.pi * (np.outer(a, a) % n) / n)


def half_weights(w):
    """c_l for l = 0 .. W/2 (W even): 1 at l = 0 and l = W/2, 2 elsewhere.

    These count how many of the W full-spectrum columns each kept column
    stands for once Hermitian symmetry is used (section 2.4.1.1).
    """
    if w % 2:
        raise ValueError("even widths only")
    c = np.full(w // 2 + 1, 2.0)
    c[0] = 1.0
    c[w // 2] = 1.0
    return c


def rfft2(x):
    """Real 2-D DFT of the last two axes, keeping columns l = 0 .. W/2.

    X[k, l] = sum_{h<H, w<W} x[h, w] exp(-2 pi i (h k / H + w l / W)).
    """
    x = np.asarray(x, dtype=np.float64)
    h, w = x.shape[-2:]
    fh = dft_matrix(h, -1)
    fw = dft_matrix(w, -1)[: w // 2 + 1]  # rows l = 0 .. W/2
    return fh @ x @ fw.T


def irfft2(y, h, w):
    """Inverse of ``rfft2`` for an h x w real output.

    out[h', w'] = (1/(H W)) sum_{k<H} sum_{l<=W/2} c_l Re(Y[k, l] exp(+2 pi i (h' k/H + w' l/W))).

    This is the inverse real DFT for any complex Y, Hermitian or not: the
    imaginary parts that Hermitian symmetry would force to zero (columns 0
    and W/2 after the column inverse) simply drop out through Re().
    """
    y = np.asarray(y, dtype=np.complex128)
    if y.shape[-2] != h or y.shape[-1] != w // 2 + 1:
        raise ValueError("spectrum shape does not match the output size")
    eh = dft_matrix(h, +1)
    ew = dft_matrix(w, +1)[:, : w // 2 + 1]  # ew[w', l] = exp(+2 pi i w' l / W)
    c = half_weights(w)
    return np.real(eh @ (y * c) @ ew.T) / (h * w)


def rfft2_adjoint(g, h, w):
    """Adjoint of ``rfft2`` under the real inner product <A, B> = sum Re(A conj(B)).

    If X = rfft2(x) and G = dL/dX (as dL/dRe + i dL/dIm), then
    dL/dx[h', w'] = sum_{k, l<=W/2} Re(G[k, l] exp(+2 pi i (h' k/H + w' l/W))).
    """
    g = np.asarray(g, dtype=np.complex128)
    eh = dft_matrix(h, +1)
    ew = dft_matrix(w, +1)[:, : w // 2 + 1]
    return np.real(eh @ g @ ew.T)


def irfft2_adjoint(g):
    """Adjoint of ``irfft2`` under the real inner product.

    If y = irfft2(Y) and g = dL/dy, then
    dL/dY[k, l] = (c_l / (H W)) sum_{h', w'} g[h', w'] exp(-2 pi i (h' k/H + w' l/W)).
    """
    g = np.asarray(g, dtype=np.float64)
    h, w = g.shape[-2:]
    return rfft2(g) * half_weights(w) / (h * w)


def hermitian_projection(y):
    """Pi_H: rfft2(irfft2(Y)) for a half spectrum Y with an even number of rows and columns.

    Columns 0 and W/2 become (Y[k, l] + conj(Y[-k mod H, l])) / 2; other columns
    are unchanged.  Written out directly so that tests can check the identity.
    """
    y = np.array(y, dtype=np.complex128)
    h, wf = y.shape[-2:]
    out = y.copy()
    neg = (-np.arange(h)) % h
    for l in (0, wf - 1):
        col = y[..., :, l]
        out[..., :, l] = 0.5 * (col + np.conj(col[..., neg]))
    return out
