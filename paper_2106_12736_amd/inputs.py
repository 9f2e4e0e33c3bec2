"""Seeded synthetic inputs for the FDC/FDP hot path.

This module is the only code shared by the HIP path's tests/bench and the CPU
oracle.  It holds random draws and workload shapes only -- no transform, product,
pooling or gradient arithmetic of the method.

The paper trains on grayscale APTOS 2019 fundus photographs, preprocessed to
512 x 512 (section 2.1-2.2).  That dataset is not available here, so the
generators below stand in for it with images of the same shape and character:
a bright disc on a black background with a radial vignette, and (for the
1024 x 1024 workload) small bright and dark Gaussian blobs of 2-6 px radius in
the role of exudates and microaneurysms.

Draw order for each workload: activations, then the kernels of every layer in
layer order, then the upstream gradient.  Every draw uses
numpy.random.default_rng(20210600 + workload index) and is returned as float32
(complex spectra as complex64).
"""

from dataclasses import dataclass, field

import numpy as np

SEED_BASE = 20210600


@dataclass(frozen=True)
class CicStack:
    """A stack of CIC + FDP layers on square images.

    sizes[i] -> sizes[i+1] is layer i's spatial size before and after pooling;
    channels[i] -> channels[i+1] its channel fan-out (S = J * C).
    """
    name: str
    index: int
    batch: int
    sizes: tuple
    channels: tuple
    image: str  # "uniform" | "disc" | "fundus"

    @property
    def layers(self):
        return len(self.sizes) - 1


@dataclass(frozen=True)
class FullFdcLayer:
    """One Full FDC layer: B x C x P x P -> B x C x (P-n+1)^2 with n x n weights (crop mode)."""
    name: str
    index: int
    batch: int
    size: int
    cin: int
    cout: int
    n: int = 3


LAYER64 = CicStack("cic_layer_64", 1, 2, (64, 32), (1, 4), "uniform")
STACK256 = CicStack("cic_stack_256", 2, 16, (256, 128, 64, 32), (1, 8, 16, 32), "uniform")
STACK512 = CicStack("cic_stack_512", 3, 32, (512, 256, 128, 64, 32), (1, 8, 16, 32, 64), "disc")
STACK1024 = CicStack("cic_stack_1024", 4, 8, (1024, 512, 256, 128, 64, 32), (1, 8, 16, 32, 64, 128),
                     "fundus")
CIC_WORKLOADS = (LAYER64, STACK256, STACK512, STACK1024)

FULL_FDC_WORKLOADS = tuple(
    FullFdcLayer(f"full_fdc_{p}_c{c}", 5, 16, p, c, c) for p in (224, 512) for c in (64, 128, 256)
)


@dataclass(frozen=True)
class FullCicLayer:
    """A Full FDC layer with CIC as the paper's VGG16 variants use it (the layers of
    Conv Block 4 at 512 x 512 input, i.e. 64 x 64 activations): B x Cin x P x P ->
    B x Cout x (P-n+1)^2, n x n spatial kernels, crop, Cout = J * Cin."""
    name: str
    index: int
    batch: int
    size: int
    cin: int
    cout: int
    n: int = 3


FULL_CIC_WORKLOADS = (
    FullCicLayer("full_cic_64_c256_512", 6, 16, 64, 256, 512),
    FullCicLayer("full_cic_64_c512_512", 6, 16, 64, 512, 512),
)


def rng_for(index, salt=0):
    return np.random.default_rng(SEED_BASE + index + 1000 * salt)


# ----------------------------------------------------------------------------
# image generators
# ----------------------------------------------------------------------------

def _radial(n):
    t = (np.arange(n) + 0.5 - n / 2) / (n / 2)
    v, u = np.meshgrid(t, t, indexing="ij")
    return np.sqrt(u * u + v * v)


def disc_mask(n):
    """Smooth fundus disc: 1 inside radius 0.92 (of the half-width), 0 outside."""
    r = _radial(n)
    return 1.0 / (1.0 + np.exp((r - 0.92) / 0.015))


def vignette(n):
    return 1.0 - 0.4 * _radial(n) ** 2


def uniform_images(rng, b, c, n):
    return rng.random((b, c, n, n), dtype=np.float32)


def disc_images(rng, b, c, n):
    """U[0,1) texture under the disc mask and vignette (fundus-like disc on black)."""
    base = (disc_mask(n) * vignette(n)).astype(np.float32)
    return rng.random((b, c, n, n), dtype=np.float32) * base


def fundus_images(rng, b, c, n, blobs=64):
    """Disc + vignette at 0.55 plus sparse Gaussian blobs (2-6 px radius), clipped to [0, 1].

    Half the blobs are bright (amplitude +U[0.15, 0.35]), half dark (-U[0.15, 0.35]);
    blob centres are uniform in the disc of radius 0.85.
    """
    mask = disc_mask(n)
    base = 0.55 * mask * vignette(n)
    out = np.empty((b, c, n, n), dtype=np.float32)
    for bi in range(b):
        for ci in range(c):
            img = base.copy()
            radius = np.sqrt(rng.random(blobs)) * 0.85
            theta = rng.random(blobs) * 2 * np.pi
            rho = rng.uniform(2.0, 6.0, blobs)
            amp = rng.uniform(0.15, 0.35, blobs)
            amp[blobs // 2:] *= -1.0
            cy = (radius * np.sin(theta) + 1.0) * n / 2 - 0.5
            cx = (radius * np.cos(theta) + 1.0) * n / 2 - 0.5
            for i in range(blobs):
                half = int(np.ceil(4 * rho[i]))
                y0, y1 = max(0, int(cy[i]) - half), min(n, int(cy[i]) + half + 1)
                x0, x1 = max(0, int(cx[i]) - half), min(n, int(cx[i]) + half + 1)
                yy = np.arange(y0, y1)[:, None] - cy[i]
                xx = np.arange(x0, x1)[None, :] - cx[i]
                img[y0:y1, x0:x1] += mask[y0:y1, x0:x1] * amp[i] * np.exp(
                    -(yy * yy + xx * xx) / (2 * rho[i] ** 2))
            out[bi, ci] = np.clip(img, 0.0, 1.0)
    return out


def spectral_kernels(rng, s, n, std=0.1):
    """Complex kernels at the rfft2 spectrum shape [S][n][n/2+1]; Re and Im independently N(0, std^2)."""
    ri = rng.standard_normal((s, n, n // 2 + 1, 2), dtype=np.float32) * np.float32(std)
    return ri.view(np.complex64)[..., 0]


def he_normal_weights(rng, cout, cin, n):
    """Kaiming/He-normal spatial weights: N(0, 2 / (cin n^2))."""
    std = np.float32(np.sqrt(2.0 / (cin * n * n)))
    return rng.standard_normal((cout, cin, n, n), dtype=np.float32) * std


def normal(rng, shape):
    return rng.standard_normal(shape, dtype=np.float32)


# ----------------------------------------------------------------------------
# whole-workload draws
# ----------------------------------------------------------------------------

@dataclass
class CicStackInputs:
    x: np.ndarray                 # [B][C0][N0][N0] float32
    kernels: list = field(default_factory=list)   # per layer [S][N][N/2+1] complex64
    grad: np.ndarray = None       # [B][S_last][M_last][M_last] float32


def make_cic_stack(wl: CicStack, batch=None):
    """Draw x, every layer's kernels and the upstream gradient for a CIC stack workload."""
    b = wl.batch if batch is None else batch
    rng = rng_for(wl.index)
    n0, c0 = wl.sizes[0], wl.channels[0]
    if wl.image == "uniform":
        x = uniform_images(rng, b, c0, n0)
    elif wl.image == "disc":
        x = disc_images(rng, b, c0, n0)
    else:
        x = fundus_images(rng, b, c0, n0)
    kernels = [spectral_kernels(rng, wl.channels[i + 1], wl.sizes[i]) for i in range(wl.layers)]
    grad = normal(rng, (b, wl.channels[-1], wl.sizes[-1], wl.sizes[-1]))
    return CicStackInputs(x, kernels, grad)


@dataclass
class FullFdcInputs:
    x: np.ndarray   # [B][Cin][P][P]
    w: np.ndarray   # [Cout][Cin][n][n]
    grad: np.ndarray  # [B][Cout][P-n+1][P-n+1]


def make_full_fdc(wl: FullFdcLayer, batch=None):
    b = wl.batch if batch is None else batch
    rng = rng_for(wl.index, salt=wl.size * 1000 + wl.cin)
    x = normal(rng, (b, wl.cin, wl.size, wl.size))
    w = he_normal_weights(rng, wl.cout, wl.cin, wl.n)
    o = wl.size - wl.n + 1
    grad = normal(rng, (b, wl.cout, o, o))
    return FullFdcInputs(x, w, grad)


@dataclass
class CicSpatialInputs:
    x: np.ndarray            # [B][C0][N0][N0] float32
    weights: list = field(default_factory=list)   # per layer [S][n][n] float32
    grad: np.ndarray = None  # [B][S_last][M_last][M_last] float32


def make_cic_spatial(wl: CicStack, n, batch=None):
    """A CIC stack workload with n x n spatial kernels instead of spectra: the same
    images, He-normal depthwise weights N(0, 2 / n^2) per layer (fan-in n^2: each
    output channel convolves one input channel), and the upstream gradient."""
    b = wl.batch if batch is None else batch
    rng = rng_for(wl.index, salt=100 + n)
    n0, c0 = wl.sizes[0], wl.channels[0]
    if wl.image == "uniform":
        x = uniform_images(rng, b, c0, n0)
    elif wl.image == "disc":
        x = disc_images(rng, b, c0, n0)
    else:
        x = fundus_images(rng, b, c0, n0)
    std = np.float32(np.sqrt(2.0 / (n * n)))
    weights = [rng.standard_normal((wl.channels[i + 1], n, n), dtype=np.float32) * std for i in range(wl.layers)]
    grad = normal(rng, (b, wl.channels[-1], wl.sizes[-1], wl.sizes[-1]))
    return CicSpatialInputs(x, weights, grad)


@dataclass
class FullCicInputs:
    x: np.ndarray     # [B][Cin][P][P]
    w: np.ndarray     # [Cout][n][n]
    grad: np.ndarray  # [B][Cout][P-n+1][P-n+1]


def make_full_cic(wl: FullCicLayer, batch=None):
    """Activations N(0,1), He-normal depthwise weights N(0, 2 / n^2), upstream gradient N(0,1)."""
    b = wl.batch if batch is None else batch
    rng = rng_for(wl.index, salt=wl.cin * 1000 + wl.cout)
    x = normal(rng, (b, wl.cin, wl.size, wl.size))
    w = rng.standard_normal((wl.cout, wl.n, wl.n), dtype=np.float32) * np.float32(np.sqrt(2.0 / (wl.n * wl.n)))
    o = wl.size - wl.n + 1
    grad = normal(rng, (b, wl.cout, o, o))
    return FullCicInputs(x, w, grad)

