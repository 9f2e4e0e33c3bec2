"""Brute-force spatial convolutions (no transforms), used to pin the frequency-domain oracle.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).
"""

import numpy as np


def correlate_valid(img, k):
    """Eq. 1: O(i, j) = sum_{a<n, b<n} I(i + a, j + b) K(a, b), output (N-n+1) x (N-n+1).

    Written with explicit loops over output pixels and kernel taps.
    """
    img = np.asarray(img, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    h, w = img.shape
    n0, n1 = k.shape
    out = np.zeros((h - n0 + 1, w - n1 + 1))
    for i in range(out.shape[0]):
        for j in range(out.shape[1]):
            acc = 0.0
            for a in range(n0):
                for b in range(n1):
                    acc += img[i + a, j + b] * k[a, b]
            out[i, j] = acc
    return out


def circular_convolve(img, k):
    """Circular (wrap-around) convolution, the operation the convolution theorem (Eq. 4)
    turns into a pointwise product: y[i, j] = sum_{a, b} k[a, b] img[(i-a) mod H, (j-b) mod W].

    The kernel may be any size up to the image size.  Loops over every output
    pixel and every kernel tap.
    """
    img = np.asarray(img, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    h, w = img.shape
    n0, n1 = k.shape
    out = np.zeros((h, w))
    for i in range(h):
        for j in range(w):
            acc = 0.0
            for a in range(n0):
                for b in range(n1):
                    acc += k[a, b] * img[(i - a) % h, (j - b) % w]
            out[i, j] = acc
    return out


def cov_valid(x, w):
    """Eq. 2 with Eq. 1 as the per-channel operation, but with the kernel flipped so the
    per-channel operation is a true convolution: out[s] = sum_c conv_valid(x[c], w[s, c]).

    x [C][H][W], w [S][C][n][n] -> [S][H-n+1][W-n+1].
    """
    s_n, c_n = w.shape[:2]
    outs = []
    for s in range(s_n):
        acc = 0.0
        for c in range(c_n):
            acc = acc + correlate_valid(x[c], w[s, c][::-1, ::-1])
        outs.append(acc)
    return np.stack(outs)
