"""Torch-facing wrappers of libfdc: plans, workspaces and calls on the current stream.

PyTorch only provides device memory and the stream; every step of the
computation runs in libfdc's HIP kernels.  Tensors must be contiguous CUDA
(HIP) tensors: float32 for images, complex64 for spectra.
"""

import ctypes
import weakref

import torch

from . import _lib
from ._lib import ARTIFACT_CROP, ARTIFACT_NONE, ARTIFACT_ROLL, call  # noqa: F401

_ARTIFACTS = {"none": ARTIFACT_NONE, "crop": ARTIFACT_CROP, "roll": ARTIFACT_ROLL}


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _check(t, dtype, shape=None, name="tensor"):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype} (got {t.dtype})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")


def _workspace(nbytes, device):
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def _own(obj, destroy):
    """Destroy obj's plan handle `obj._p` with the C function `destroy` when obj is
    collected or at interpreter exit; the function object is bound now, so the call
    does not depend on module state during shutdown."""
    weakref.finalize(obj, getattr(_lib.lib(), destroy), ctypes.c_void_p(obj._p.value))


def _check_saved(saved, nbytes, name="saved"):
    """A saved-spectrum buffer: contiguous complex64 of exactly nbytes bytes."""
    _check(saved, torch.complex64, (nbytes // 8,), name)


class FftPlan:
    """Batched 2-D real FFT of `count` h x w images (fdc_rfft2 and friends)."""

    def __init__(self, count, h, w):
        self.count, self.h, self.w = count, h, w
        self._p = ctypes.c_void_p()
        call("fdc_fft_plan_create", ctypes.byref(self._p), count, h, w)
        _own(self, "fdc_fft_plan_destroy")
        n = ctypes.c_size_t()
        call("fdc_fft_workspace_size", self._p, ctypes.byref(n))
        self.ws_bytes = n.value

    def _spec_shape(self, lead):
        return lead + (self.h, self.w // 2 + 1)

    def _run(self, name, src, dst, ws):
        call(name, self._p, _ptr(src), _ptr(dst), _ptr(ws), ws.numel() if ws is not None else 0, _stream())
        return dst

    def rfft2(self, x):
        _check(x, torch.float32, name="x")
        out = torch.empty(self._spec_shape(tuple(x.shape[:-2])), dtype=torch.complex64, device=x.device)
        return self._run("fdc_rfft2", x, out, None)

    def rfft2_pooled(self, x, mh, mw, out=None, ws=None):
        """fdc_rfft2_pooled into `out` (a new tensor if None): the bins an FDP to
        mh x mw keeps; the others are undefined.  With a workspace `ws` (a uint8
        tensor of at least count * h * (mw/2 + 1) * 8 bytes), fdc_rfft2_pooled_ws."""
        _check(x, torch.float32, name="x")
        if out is None:
            out = torch.empty(self._spec_shape(tuple(x.shape[:-2])), dtype=torch.complex64, device=x.device)
        _check(out, torch.complex64, self._spec_shape(tuple(x.shape[:-2])), "out")
        if ws is None:
            call("fdc_rfft2_pooled", self._p, _ptr(x), _ptr(out), mh, mw, _stream())
        else:
            call("fdc_rfft2_pooled_ws", self._p, _ptr(x), _ptr(out), mh, mw, _ptr(ws), ws.numel() * ws.element_size(),
                 _stream())
        return out

    def irfft2(self, X):
        _check(X, torch.complex64, name="X")
        out = torch.empty(tuple(X.shape[:-2]) + (self.h, self.w), dtype=torch.float32, device=X.device)
        return self._run("fdc_irfft2", X, out, _workspace(self.ws_bytes, X.device))

    def rfft2_backward(self, gX):
        _check(gX, torch.complex64, name="gX")
        out = torch.empty(tuple(gX.shape[:-2]) + (self.h, self.w), dtype=torch.float32, device=gX.device)
        return self._run("fdc_rfft2_backward", gX, out, _workspace(self.ws_bytes, gX.device))

    def irfft2_backward(self, gx):
        _check(gx, torch.float32, name="gx")
        out = torch.empty(self._spec_shape(tuple(gx.shape[:-2])), dtype=torch.complex64, device=gx.device)
        return self._run("fdc_irfft2_backward", gx, out, None)


def cic_forward(X, K):
    """Spectral CIC (Eq. 5): X [B][C][H][Wf], K [S][H][Wf] -> [B][S][H][Wf]."""
    _check(X, torch.complex64, name="X")
    _check(K, torch.complex64, name="K")
    B, C, H, Wf = X.shape
    S = K.shape[0]
    Y = torch.empty((B, S, H, Wf), dtype=torch.complex64, device=X.device)
    call("fdc_cic_forward", _ptr(X), _ptr(K), _ptr(Y), B, C, S, H, Wf, _stream())
    return Y


def cic_backward(gY, X, K, need_gx=True, need_gk=True):
    _check(gY, torch.complex64, name="gY")
    B, S, H, Wf = gY.shape
    C = X.shape[1]
    gX = torch.empty_like(X) if need_gx else None
    gK = torch.empty_like(K) if need_gk else None
    call("fdc_cic_backward", _ptr(gY), _ptr(X), _ptr(K), _ptr(gX), _ptr(gK), B, C, S, H, Wf, _stream())
    return gX, gK


def fdp_forward(X, mh, mw):
    """FDP crop: [.., H, W/2+1] -> [.., mh, mw/2+1] (W taken as 2 * (Wf - 1))."""
    _check(X, torch.complex64, name="X")
    H, Wf = X.shape[-2:]
    W = 2 * (Wf - 1)
    count = X.numel() // (H * Wf)
    Y = torch.empty(tuple(X.shape[:-2]) + (mh, mw // 2 + 1), dtype=torch.complex64, device=X.device)
    call("fdp_forward", _ptr(X), _ptr(Y), count, H, W, mh, mw, _stream())
    return Y


def fdp_backward(gY, h, w):
    _check(gY, torch.complex64, name="gY")
    mh, mwf = gY.shape[-2:]
    count = gY.numel() // (mh * mwf)
    gX = torch.empty(tuple(gY.shape[:-2]) + (h, w // 2 + 1), dtype=torch.complex64, device=gY.device)
    call("fdp_backward", _ptr(gY), _ptr(gX), count, h, w, mh, 2 * (mwf - 1), _stream())
    return gX


class _LayerPlan:
    def _sizes(self):
        f, s, b = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
        call("fdc_layer_workspace_size", self._p, ctypes.byref(f), ctypes.byref(s), ctypes.byref(b))
        o = ctypes.c_int()
        call("fdc_layer_output_size", self._p, ctypes.byref(o))
        self.fwd_ws_bytes, self.saved_bytes, self.bwd_ws_bytes = f.value, s.value, b.value
        self.out = o.value


class CicLayer(_LayerPlan):
    """Fused CIC + FDP layer: x [B][C][N][N] -> y [B][S][O][O] (fdc_cic_layer_*).

    Workspaces are allocated once per layer object and reused by every call,
    so a layer object must not run concurrently on two streams.
    """

    def __init__(self, B, C, S, N, M, artifact="none", kernel_n=1, device="cuda"):
        self.B, self.C, self.S, self.N, self.M = B, C, S, N, M
        self._p = ctypes.c_void_p()
        call("fdc_cic_layer_plan_create", ctypes.byref(self._p), B, C, S, N, M, _ARTIFACTS[artifact], kernel_n)
        _own(self, "fdc_layer_plan_destroy")
        self._sizes()
        self.device = torch.device(device)
        self.fwd_ws = _workspace(self.fwd_ws_bytes, self.device)
        self.bwd_ws = _workspace(self.bwd_ws_bytes, self.device)

    def new_saved(self):
        """Buffer for the pooled input spectrum (see fdc_cic_layer_forward for its layout)."""
        return torch.empty(self.saved_bytes // 8, dtype=torch.complex64, device=self.device)

    def dk_ranges(self):
        """Image ranges the backward's dK step sums separately (fdc_cic_layer_dk_ranges)."""
        r = ctypes.c_int()
        call("fdc_cic_layer_dk_ranges", self._p, ctypes.byref(r))
        return r.value

    def saved_spectrum(self, saved):
        """The M x (M/2+1) kept bins held in a saved buffer, as a [B][C][M][M/2+1] tensor:
        columns 0..M/2-1 come from the main block (8-column tiles [M/16][M][8] per
        image and channel when M/2 is a multiple of 8), column M/2 from the block after it."""
        B, C, M = self.B, self.C, self.M
        h = M // 2
        if h % 8 == 0:
            main = saved[: B * C * M * h].view(B, C, h // 8, M, 8).permute(0, 1, 3, 2, 4).reshape(B, C, M, h)
        else:
            main = saved[: B * C * M * h].view(B, C, M, h)
        side = saved[B * C * M * h:].view(B, C, M, 1)
        return torch.cat([main, side], dim=-1)

    def new_output(self):
        return torch.empty((self.B, self.S, self.out, self.out), dtype=torch.float32, device=self.device)

    def forward(self, x, K, y=None, saved=None):
        _check(x, torch.float32, (self.B, self.C, self.N, self.N), "x")
        _check(K, torch.complex64, (self.S, self.N, self.N // 2 + 1), "K")
        y = self.new_output() if y is None else y
        _check(y, torch.float32, (self.B, self.S, self.out, self.out), "y")
        if saved is not None:
            _check_saved(saved, self.saved_bytes)
        call("fdc_cic_layer_forward", self._p, _ptr(x), _ptr(K), _ptr(y), _ptr(saved), _ptr(self.fwd_ws),
             self.fwd_ws.numel(), _stream())
        return y

    def backward(self, gy, saved, K, need_gx=True, need_gk=True, gx=None, gK=None):
        _check(gy, torch.float32, (self.B, self.S, self.out, self.out), "gy")
        if need_gx and gx is None:
            gx = torch.empty((self.B, self.C, self.N, self.N), dtype=torch.float32, device=self.device)
        if need_gk and gK is None:
            gK = torch.empty((self.S, self.N, self.N // 2 + 1), dtype=torch.complex64, device=self.device)
        if need_gx:
            _check(gx, torch.float32, (self.B, self.C, self.N, self.N), "gx")
            _check(K, torch.complex64, (self.S, self.N, self.N // 2 + 1), "K")
        if need_gk:
            _check(gK, torch.complex64, (self.S, self.N, self.N // 2 + 1), "gK")
            _check_saved(saved, self.saved_bytes)
        call("fdc_cic_layer_backward", self._p, _ptr(gy), _ptr(saved), _ptr(K), _ptr(gx if need_gx else None),
             _ptr(gK if need_gk else None), _ptr(self.bwd_ws), self.bwd_ws.numel(), _stream())
        return (gx if need_gx else None), (gK if need_gk else None)


def full_row(P):
    """FDC_FULL_ROW(P) of fdc.h: complex elements per plane row in a Full FDC spectrum's main block."""
    return P // 2 + 16


def full_side_plane(P):
    """FDC_FULL_SIDE_PLANE(P) of fdc.h: complex elements per Nyquist-column plane."""
    return P + 8


class FullLayer(_LayerPlan):
    """Full FDC layer: x [B][Cin][P][P], w [Cout][Cin][n][n] -> y [B][Cout][O][O]
    (fdc_full_layer_*).  Workspaces are allocated once per layer object."""

    def __init__(self, B, Cin, Cout, P, kernel_n=3, artifact="crop", device="cuda"):
        self.B, self.Cin, self.Cout, self.P, self.n = B, Cin, Cout, P, kernel_n
        self._p = ctypes.c_void_p()
        call("fdc_full_layer_plan_create", ctypes.byref(self._p), B, Cin, Cout, P, kernel_n, _ARTIFACTS[artifact])
        _own(self, "fdc_layer_plan_destroy")
        self._sizes()
        self.device = torch.device(device)
        self.fwd_ws = _workspace(self.fwd_ws_bytes, self.device)
        self.bwd_ws = _workspace(self.bwd_ws_bytes, self.device)

    def new_saved(self):
        """Buffer for rfft2(x) (see fdc_full_forward for its layout)."""
        return torch.empty(self.saved_bytes // 8, dtype=torch.complex64, device=self.device)

    def saved_spectrum(self, saved):
        """rfft2(x) held in a saved buffer (layout in fdc_full_forward's header entry),
        as a [B][Cin][P][P/2+1] tensor."""
        B, C, P = self.B, self.Cin, self.P
        h, R, SS = P // 2, full_row(P), full_side_plane(P)
        n = B * C
        main = saved[: P * n * R].view(P, B, C, R)[..., :h].permute(1, 2, 0, 3)
        side = saved[P * n * R:].view(B, C, SS)[..., :P].reshape(B, C, P, 1)
        return torch.cat([main, side], dim=-1)

    def new_output(self):
        return torch.empty((self.B, self.Cout, self.out, self.out), dtype=torch.float32, device=self.device)

    def forward(self, x, w, y=None, saved=None):
        _check(x, torch.float32, (self.B, self.Cin, self.P, self.P), "x")
        _check(w, torch.float32, (self.Cout, self.Cin, self.n, self.n), "w")
        if saved is not None:
            _check(saved, torch.complex64, (self.saved_bytes // 8,), "saved")
        y = self.new_output() if y is None else y
        _check(y, torch.float32, (self.B, self.Cout, self.out, self.out), "y")
        call("fdc_full_forward", self._p, _ptr(x), _ptr(w), _ptr(y), _ptr(saved), _ptr(self.fwd_ws),
             self.fwd_ws.numel(), _stream())
        return y

    def backward(self, gy, saved, w, need_gx=True, need_gw=True, gx=None, gw=None):
        _check(gy, torch.float32, (self.B, self.Cout, self.out, self.out), "gy")
        if need_gx and gx is None:
            gx = torch.empty((self.B, self.Cin, self.P, self.P), dtype=torch.float32, device=self.device)
        if need_gw and gw is None:
            gw = torch.empty((self.Cout, self.Cin, self.n, self.n), dtype=torch.float32, device=self.device)
        if need_gx:
            _check(gx, torch.float32, (self.B, self.Cin, self.P, self.P), "gx")
            _check(w, torch.float32, (self.Cout, self.Cin, self.n, self.n), "w")
        if need_gw:
            _check(gw, torch.float32, (self.Cout, self.Cin, self.n, self.n), "gw")
            _check_saved(saved, self.saved_bytes)
        call("fdc_full_backward", self._p, _ptr(gy), _ptr(saved), _ptr(w), _ptr(gx if need_gx else None),
             _ptr(gw if need_gw else None), _ptr(self.bwd_ws), self.bwd_ws.numel(), _stream())
        return (gx if need_gx else None), (gw if need_gw else None)


class CicSpatialLayer(CicLayer):
    """The CIC + FDP layer with spatial n x n kernels w [S][n][n], transformed on every
    call (fdc_cic_spatial_layer_*); n is the plan's kernel_n."""

    def __init__(self, B, C, S, N, M, kernel_n, artifact="roll", device="cuda"):
        super().__init__(B, C, S, N, M, artifact=artifact, kernel_n=kernel_n, device=device)
        self.n = kernel_n
        f, b = ctypes.c_size_t(), ctypes.c_size_t()
        call("fdc_cic_spatial_workspace_size", self._p, ctypes.byref(f), ctypes.byref(b))
        self.fwd_ws = _workspace(f.value, self.device)
        self.bwd_ws = _workspace(b.value, self.device)

    def forward(self, x, w, y=None, saved=None):
        _check(x, torch.float32, (self.B, self.C, self.N, self.N), "x")
        _check(w, torch.float32, (self.S, self.n, self.n), "w")
        y = self.new_output() if y is None else y
        _check(y, torch.float32, (self.B, self.S, self.out, self.out), "y")
        if saved is not None:
            _check_saved(saved, self.saved_bytes)
        call("fdc_cic_spatial_layer_forward", self._p, _ptr(x), _ptr(w), _ptr(y), _ptr(saved), _ptr(self.fwd_ws),
             self.fwd_ws.numel(), _stream())
        return y

    def backward(self, gy, saved, w, need_gx=True, need_gw=True, gx=None, gw=None):
        _check(gy, torch.float32, (self.B, self.S, self.out, self.out), "gy")
        if need_gx and gx is None:
            gx = torch.empty((self.B, self.C, self.N, self.N), dtype=torch.float32, device=self.device)
        if need_gw and gw is None:
            gw = torch.empty((self.S, self.n, self.n), dtype=torch.float32, device=self.device)
        if need_gx:
            _check(gx, torch.float32, (self.B, self.C, self.N, self.N), "gx")
            _check(w, torch.float32, (self.S, self.n, self.n), "w")
        if need_gw:
            _check(gw, torch.float32, (self.S, self.n, self.n), "gw")
            _check_saved(saved, self.saved_bytes)
        call("fdc_cic_spatial_layer_backward", self._p, _ptr(gy), _ptr(saved), _ptr(w),
             _ptr(gx if need_gx else None), _ptr(gw if need_gw else None), _ptr(self.bwd_ws), self.bwd_ws.numel(),
             _stream())
        return (gx if need_gx else None), (gw if need_gw else None)


class CicSpatialStack:
    """A stack of spatial-kernel CIC + FDP layers (ROLL artifact handling, so sizes
    stay powers of two) with preallocated activations, saved spectra and gradients."""

    def __init__(self, batch, sizes, channels, kernel_n, device="cuda"):
        self.layers = [CicSpatialLayer(batch, channels[i], channels[i + 1], sizes[i], sizes[i + 1], kernel_n,
                                       artifact="roll", device=device) for i in range(len(sizes) - 1)]
        self.saved = [layer.new_saved() for layer in self.layers]
        self.acts = [layer.new_output() for layer in self.layers]
        self.gacts = [None] + [torch.empty((batch, channels[i], sizes[i], sizes[i]), dtype=torch.float32,
                                           device=device) for i in range(1, len(sizes) - 1)]
        self.gws = [torch.empty((channels[i + 1], kernel_n, kernel_n), dtype=torch.float32, device=device)
                    for i in range(len(sizes) - 1)]

    def forward(self, x, weights):
        h = x
        for layer, w, y, sv in zip(self.layers, weights, self.acts, self.saved):
            layer.forward(h, w, y=y, saved=sv)
            h = y
        return h

    def dk_ranges(self):
        return [layer.dk_ranges() for layer in self.layers]

    def backward(self, gy, weights, input_grad=None):
        g = gy
        for i in reversed(range(len(self.layers))):
            gx = self.gacts[i] if i > 0 else input_grad
            self.layers[i].backward(g, self.saved[i], weights[i], need_gx=gx is not None, need_gw=True, gx=gx,
                                    gw=self.gws[i])
            g = gx
        return self.gws


class CicStack:
    """A stack of fused CIC + FDP layers with preallocated activations, saved
    spectra and gradients, so that one forward + backward step allocates nothing."""

    def __init__(self, batch, sizes, channels, device="cuda"):
        self.layers = [CicLayer(batch, channels[i], channels[i + 1], sizes[i], sizes[i + 1], device=device)
                       for i in range(len(sizes) - 1)]
        self.saved = [layer.new_saved() for layer in self.layers]
        self.acts = [layer.new_output() for layer in self.layers]
        self.gacts = [None] + [torch.empty((batch, channels[i], sizes[i], sizes[i]), dtype=torch.float32,
                                           device=device) for i in range(1, len(sizes) - 1)]
        self.gks = [torch.empty((channels[i + 1], sizes[i], sizes[i] // 2 + 1), dtype=torch.complex64,
                                device=device) for i in range(len(sizes) - 1)]

    def forward(self, x, kernels):
        h = x
        for layer, K, y, sv in zip(self.layers, kernels, self.acts, self.saved):
            layer.forward(h, K, y=y, saved=sv)
            h = y
        return h

    def dk_ranges(self):
        return [layer.dk_ranges() for layer in self.layers]

    def backward(self, gy, kernels, input_grad=None):
        """Gradients of every kernel (and of the input if `input_grad` is a tensor to fill)."""
        g = gy
        for i in reversed(range(len(self.layers))):
            layer = self.layers[i]
            if i > 0:
                gx = self.gacts[i]
            else:
                gx = input_grad
            layer.backward(g, self.saved[i], kernels[i], need_gx=gx is not None, need_gk=True, gx=gx,
                           gK=self.gks[i])
            g = gx
        return self.gks


def _ptr_array(tensors):
    arr = (ctypes.c_void_p * len(tensors))()
    for i, t in enumerate(tensors):
        arr[i] = t.data_ptr() if t is not None else None
    return arr


class CicStackFused:
    """The same stack as CicStack run through fdc_cic_stack_*: one plan, the
    activations between layers never written to memory.  Kernel gradients, saved
    spectra, the last activation and workspaces are preallocated."""

    def __init__(self, batch, sizes, channels, device="cuda"):
        self.batch, self.sizes, self.channels = batch, tuple(sizes), tuple(channels)
        self.layers = len(sizes) - 1
        self.device = torch.device(device)
        self._sizes = (ctypes.c_int * len(sizes))(*sizes)
        self._chans = (ctypes.c_int * len(channels))(*channels)
        self._p = ctypes.c_void_p()
        call("fdc_cic_stack_plan_create", ctypes.byref(self._p), batch, self.layers, self._sizes, self._chans)
        _own(self, "fdc_cic_stack_plan_destroy")
        f, b = ctypes.c_size_t(), ctypes.c_size_t()
        call("fdc_cic_stack_workspace_size", self._p, ctypes.byref(f), ctypes.byref(b))
        self.fwd_ws = _workspace(f.value, self.device)
        self.bwd_ws = _workspace(b.value, self.device)
        self.saved = []
        for i in range(self.layers):
            n = ctypes.c_size_t()
            call("fdc_cic_stack_saved_size", self._p, i, ctypes.byref(n))
            self.saved.append(torch.empty(n.value // 8, dtype=torch.complex64, device=self.device))
        self.out = torch.empty((batch, channels[-1], sizes[-1], sizes[-1]), dtype=torch.float32, device=self.device)
        # zero once: the backward (fdc_cic_stack_backward_kept) writes only the bins FDP
        # keeps, and the gradient is exactly zero at the others
        self.gks = [torch.zeros((channels[i + 1], sizes[i], sizes[i] // 2 + 1), dtype=torch.complex64,
                                device=self.device) for i in range(self.layers)]
        self._saved_arr = _ptr_array(self.saved)
        self._gk_arr = _ptr_array(self.gks)

    def tail(self):
        """First layer of the LDS-resident tail (fdc_cic_stack_tail), or -1."""
        r = ctypes.c_int()
        call("fdc_cic_stack_tail", self._p, ctypes.byref(r))
        return r.value

    def dk_ranges(self):
        """Image ranges each layer's dK step sums separately (fdc_cic_stack_dk_ranges)."""
        out = []
        for i in range(self.layers):
            r = ctypes.c_int()
            call("fdc_cic_stack_dk_ranges", self._p, i, ctypes.byref(r))
            out.append(r.value)
        return out

    def _kernels(self, kernels):
        if len(kernels) != self.layers:
            raise ValueError(f"{self.layers} kernel tensors expected")
        for i, K in enumerate(kernels):
            _check(K, torch.complex64, (self.channels[i + 1], self.sizes[i], self.sizes[i] // 2 + 1), f"K[{i}]")
        return _ptr_array(kernels)

    def forward(self, x, kernels):
        _check(x, torch.float32, (self.batch, self.channels[0], self.sizes[0], self.sizes[0]), "x")
        call("fdc_cic_stack_forward", self._p, _ptr(x), self._kernels(kernels), _ptr(self.out), self._saved_arr,
             _ptr(self.fwd_ws), self.fwd_ws.numel(), _stream())
        return self.out

    def backward(self, gy, kernels, input_grad=None):
        """Kernel gradients of every layer (and the input gradient into `input_grad` if given).
        The returned tensors are the module's own buffers, rewritten at the kept bins by
        every call; their other bins hold the zeros set at construction, so callers must
        not write into them."""
        _check(gy, torch.float32, tuple(self.out.shape), "gy")
        if input_grad is not None:
            _check(input_grad, torch.float32, (self.batch, self.channels[0], self.sizes[0], self.sizes[0]),
                   "input_grad")
        call("fdc_cic_stack_backward_kept", self._p, _ptr(gy), self._saved_arr, self._kernels(kernels), _ptr(input_grad),
             self._gk_arr, _ptr(self.bwd_ws), self.bwd_ws.numel(), _stream())
        return self.gks


class CicSpatialStackFused(CicStackFused):
    """The stack of CicSpatialStack (n x n spatial kernels, ROLL in every layer) run
    through fdc_cic_spatial_stack_*: every layer's kernel spectra in one launch, the
    stack executor, every layer's dL/dw in one launch."""

    def __init__(self, batch, sizes, channels, kernel_n, device="cuda"):
        super().__init__(batch, sizes, channels, device=device)
        self.kernel_n = kernel_n
        f, b = ctypes.c_size_t(), ctypes.c_size_t()
        call("fdc_cic_spatial_stack_workspace_size", self._p, kernel_n, ctypes.byref(f), ctypes.byref(b))
        self.fwd_ws = _workspace(f.value, self.device)
        self.bwd_ws = _workspace(b.value, self.device)
        self.gks = None
        self.gws = [torch.empty((channels[i + 1], kernel_n, kernel_n), dtype=torch.float32, device=self.device)
                    for i in range(self.layers)]
        self._gw_arr = _ptr_array(self.gws)

    def _weights(self, weights):
        if len(weights) != self.layers:
            raise ValueError(f"{self.layers} weight tensors expected")
        n = self.kernel_n
        for i, w in enumerate(weights):
            _check(w, torch.float32, (self.channels[i + 1], n, n), f"w[{i}]")
        return _ptr_array(weights)

    def forward(self, x, weights):
        _check(x, torch.float32, (self.batch, self.channels[0], self.sizes[0], self.sizes[0]), "x")
        call("fdc_cic_spatial_stack_forward", self._p, self.kernel_n, _ptr(x), self._weights(weights), _ptr(self.out),
             self._saved_arr, _ptr(self.fwd_ws), self.fwd_ws.numel(), _stream())
        return self.out

    def backward(self, gy, weights, input_grad=None):
        """dL/dw of every layer (and the input gradient into `input_grad` if given)."""
        _check(gy, torch.float32, tuple(self.out.shape), "gy")
        if input_grad is not None:
            _check(input_grad, torch.float32, (self.batch, self.channels[0], self.sizes[0], self.sizes[0]),
                   "input_grad")
        call("fdc_cic_spatial_stack_backward", self._p, self.kernel_n, _ptr(gy), self._saved_arr,
             self._weights(weights), _ptr(input_grad), self._gw_arr, _ptr(self.bwd_ws), self.bwd_ws.numel(),
             _stream())
        return self.gws



def hermitian_project(Y):
    """Pi_H in place on half spectra [..][H][W/2+1] (fdc_hermitian_project); returns Y."""
    if Y.dtype != torch.complex64 or not Y.is_cuda or not Y.is_contiguous() or Y.dim() < 2:
        raise ValueError("Y must be a contiguous complex64 CUDA tensor [..][H][W/2+1]")
    H, Wf = Y.shape[-2], Y.shape[-1]
    call("fdc_hermitian_project", _ptr(Y), Y.numel() // (H * Wf), H, 2 * (Wf - 1), _stream())
    return Y


def cic_fdp_forward(X, K, M, project=False):
    """FDC layer of the FDCNN on spectra followed by FDP: [B][C][N][N/2+1] -> [B][S][M][M/2+1]
    (with project=True, Pi_H of the result: fdc_cic_fdp_forward_projected)."""
    _check(X, torch.complex64, name="X")
    _check(K, torch.complex64, name="K")
    B, C, N, _ = X.shape
    S = K.shape[0]
    Y = torch.empty((B, S, M, M // 2 + 1), dtype=torch.complex64, device=X.device)
    fn = "fdc_cic_fdp_forward_projected" if project else "fdc_cic_fdp_forward"
    call(fn, _ptr(X), _ptr(K), _ptr(Y), B, C, S, N, M, _stream())
    return Y


def cic_fdp_backward(gY, X, K, need_gx=True, need_gk=True, project=False):
    """Its backward (with project=True, Pi_H of gX: fdc_cic_fdp_backward_projected)."""
    _check(gY, torch.complex64, name="gY")
    B, S, M, _ = gY.shape
    C, N = X.shape[1], X.shape[2]
    gX = torch.empty_like(X) if need_gx else None
    gK = torch.empty_like(K) if need_gk else None
    fn = "fdc_cic_fdp_backward_projected" if project else "fdc_cic_fdp_backward"
    call(fn, _ptr(gY), _ptr(X), _ptr(K), _ptr(gX), _ptr(gK), B, C, S, N, M, _stream())
    return gX, gK


class CicChain:
    """The FDCNN data flow of section 2.5.1 on a CIC + FDP stack: one rfft2 of the
    input, every FDC (CIC) + FDP layer on spectra (fdc_cic_fdp_*), one irfft2 of the
    last spectrum.  All buffers are preallocated, so a step allocates nothing.

    The gradient spectra `gspecs` and kernel gradients `gks` are zero from allocation at
    the bins each FDP drops, and the backward (fdc_cic_fdp_backward_kept) writes only the
    kept bins, so they stay zero there: a caller that replaces `gks` (as FdcnnClassifier
    does, with views of its zeroed gradient buffer) must keep that so.

    The input transform forms only the bins the first FDP keeps (fdc_rfft2_pooled_ws, in
    the chain's transform workspace): the first layer reads no others, forward or backward.

    With hermitian=True, Pi_H follows every layer but the last (the projected form of
    fdc_cic_fdp_forward), and its adjoint (itself) precedes their backward (the projected
    form of the next layer's fdc_cic_fdp_backward): the irfft2 of one layer and the
    rfft2 of the next reduce to Pi_H, so this computes the per-layer stack of
    CicStack / CicStackFused (artifact NONE) with one transform at each end."""

    def __init__(self, batch, sizes, channels, device="cuda", hermitian=False):
        self.hermitian = bool(hermitian)
        self.batch, self.sizes, self.channels = batch, tuple(sizes), tuple(channels)
        self.layers = len(sizes) - 1
        self.device = torch.device(device)
        B = batch
        self.plan_in = FftPlan(B * channels[0], sizes[0], sizes[0])
        self.plan_out = FftPlan(B * channels[-1], sizes[-1], sizes[-1])
        self.ws = _workspace(max(self.plan_in.ws_bytes, self.plan_out.ws_bytes), self.device)
        cd = torch.complex64
        self.specs = [torch.empty((B, channels[i], sizes[i], sizes[i] // 2 + 1), dtype=cd, device=self.device)
                      for i in range(self.layers + 1)]
        # zero from allocation: the backward writes only the bins each FDP keeps
        # (fdc_cic_fdp_backward_kept), and the others are never written
        self.gspecs = [torch.zeros_like(t) for t in self.specs]
        self.out = torch.empty((B, channels[-1], sizes[-1], sizes[-1]), dtype=torch.float32, device=self.device)
        self.gks = [torch.zeros((channels[i + 1], sizes[i], sizes[i] // 2 + 1), dtype=cd, device=self.device)
                    for i in range(self.layers)]

    def forward(self, x, kernels):
        _check(x, torch.float32, (self.batch, self.channels[0], self.sizes[0], self.sizes[0]), "x")
        s = _stream()
        # the first FDP keeps only some bins of the input spectrum, and the first layer
        # (forward and backward) reads no others
        m = self.sizes[1]
        call("fdc_rfft2_pooled_ws", self.plan_in._p, _ptr(x), _ptr(self.specs[0]), m, m, _ptr(self.ws),
             self.ws.numel() * self.ws.element_size(), s)
        B = self.batch
        for i, K in enumerate(kernels):
            _check(K, torch.complex64, (self.channels[i + 1], self.sizes[i], self.sizes[i] // 2 + 1), f"K[{i}]")
            # Pi_H on every layer's output but the last, in the layer's own launch
            fn = "fdc_cic_fdp_forward_projected" if self.hermitian and i + 1 < self.layers else "fdc_cic_fdp_forward"
            call(fn, _ptr(self.specs[i]), _ptr(K), _ptr(self.specs[i + 1]), B, self.channels[i],
                 self.channels[i + 1], self.sizes[i], self.sizes[i + 1], s)
        call("fdc_irfft2", self.plan_out._p, _ptr(self.specs[-1]), _ptr(self.out), _ptr(self.ws), self.ws.numel(), s)
        return self.out

    def backward(self, gy, kernels, input_grad=None):
        """Kernel gradients of every layer (and the input gradient into `input_grad` if given)."""
        _check(gy, torch.float32, tuple(self.out.shape), "gy")
        s = _stream()
        B = self.batch
        call("fdc_irfft2_backward", self.plan_out._p, _ptr(gy), _ptr(self.gspecs[-1]), None, 0, s)
        for i in reversed(range(self.layers)):
            need_gx = i > 0 or input_grad is not None
            # Pi_H (its own adjoint) on the input gradient of every layer but the first,
            # in the layer's own launch
            # (the kept-bins forms: the bins the FDP drops stay zero in gspecs and gks)
            fn = "fdc_cic_fdp_backward_projected_kept" if self.hermitian and i > 0 else "fdc_cic_fdp_backward_kept"
            call(fn, _ptr(self.gspecs[i + 1]), _ptr(self.specs[i]), _ptr(kernels[i]),
                 _ptr(self.gspecs[i] if need_gx else None), _ptr(self.gks[i]), B, self.channels[i],
                 self.channels[i + 1], self.sizes[i], self.sizes[i + 1], s)
        if input_grad is not None:
            _check(input_grad, torch.float32, (B, self.channels[0], self.sizes[0], self.sizes[0]), "input_grad")
            call("fdc_rfft2_backward", self.plan_in._p, _ptr(self.gspecs[0]), _ptr(input_grad), _ptr(self.ws),
                 self.ws.numel(), s)
        return self.gks


class FdcnnClassifier:
    """The FDCNN of section 2.5.1 (Fig. 3) as a classifier, trained as section 3.1
    describes: the spectral chain (CicChain: one rfft2, every FDC + FDP layer on
    spectra, one irfft2), a ReLU, one fully connected layer to `classes` outputs
    (fdc_head_*), the mean softmax cross-entropy, and Adam with weight decay
    (fdc_adam_step; the paper's learning rate 1e-5 and weight decay 1e-6 by default).

    All parameters (each layer's kernel spectra, then W [classes][F], then bias) live in
    one flat fp32 buffer, their gradients and the Adam moments in three more, so that
    one launch updates them all; `kernels`, `W` and `bias` are views of it.  The step
    count lives on the device, so a captured step advances on every replay."""

    def __init__(self, batch, sizes, channels, classes=2, lr=1e-5, weight_decay=1e-6, betas=(0.9, 0.999),
                 eps=1e-8, device="cuda"):
        self.chain = CicChain(batch, sizes, channels, device=device)
        self.batch, self.classes = batch, classes
        self.lr, self.weight_decay, self.betas, self.eps = lr, weight_decay, betas, eps
        dev = self.chain.device
        kshapes = [(channels[i + 1], sizes[i], sizes[i] // 2 + 1) for i in range(len(sizes) - 1)]
        self.features = channels[-1] * sizes[-1] * sizes[-1]
        F = self.features
        sizes_f = [2 * s[0] * s[1] * s[2] for s in kshapes] + [classes * F, classes]
        offs = [0]
        for n in sizes_f:
            offs.append(offs[-1] + n)
        self.n_params = offs[-1]
        self.params = torch.zeros(self.n_params, dtype=torch.float32, device=dev)
        self.grads = torch.zeros_like(self.params)
        self.m = torch.zeros_like(self.params)
        self.v = torch.zeros_like(self.params)
        self.step_count = torch.zeros(1, dtype=torch.int32, device=dev)

        def views(buf):
            ks = [buf[offs[i]:offs[i + 1]].view(torch.complex64).view(s) for i, s in enumerate(kshapes)]
            n = len(kshapes)
            return ks, buf[offs[n]:offs[n + 1]].view(classes, F), buf[offs[n + 1]:offs[n + 2]]

        self.kernels, self.W, self.bias = views(self.params)
        gks, self.gW, self.gbias = views(self.grads)
        self.chain.gks = gks  # the chain's backward writes dL/dK straight into the gradient buffer
        self.logits = torch.empty((batch, classes), dtype=torch.float32, device=dev)
        self.loss = torch.empty(1, dtype=torch.float32, device=dev)
        self.gy = torch.empty_like(self.chain.out)
        n = ctypes.c_size_t()
        call("fdc_head_workspace_size", batch, F, classes, ctypes.byref(n))
        self.head_ws = _workspace(n.value, dev)

    def load(self, kernels, W, bias):
        """Copy initial parameters in and clear the optimiser state."""
        for dst, src in zip(self.kernels, kernels):
            dst.copy_(src)
        self.W.copy_(W)
        self.bias.copy_(bias)
        self.m.zero_()
        self.v.zero_()
        self.step_count.zero_()

    def forward(self, x, labels):
        """Chain, ReLU, fully connected layer and loss; returns (logits, loss)."""
        _check(labels, torch.int32, (self.batch,), "labels")
        y = self.chain.forward(x, self.kernels)
        call("fdc_head_forward", _ptr(y), _ptr(self.W), _ptr(self.bias), _ptr(labels), _ptr(self.logits),
             _ptr(self.loss), self.batch, self.features, self.classes, _ptr(self.head_ws), self.head_ws.numel(),
             _stream())
        return self.logits, self.loss

    def backward(self, labels):
        """Gradients of the last forward's loss into `grads` (dL/dK, dL/dW, dL/dbias)."""
        call("fdc_head_backward", _ptr(self.chain.out), _ptr(self.W), _ptr(self.logits), _ptr(labels),
             _ptr(self.gy), _ptr(self.gW), _ptr(self.gbias), self.batch, self.features, self.classes, _stream())
        self.chain.backward(self.gy, self.kernels)

    def optimizer_step(self):
        b1, b2 = self.betas
        call("fdc_adam_step", _ptr(self.params), _ptr(self.grads), _ptr(self.m), _ptr(self.v), self.n_params,
             _ptr(self.step_count), self.lr, b1, b2, self.eps, self.weight_decay, _stream())

    def train_step(self, x, labels):
        self.forward(x, labels)
        self.backward(labels)
        self.optimizer_step()
        return self.loss

    def state(self):
        """A copy of the training state (parameters, moments, step count)."""
        return [t.clone() for t in (self.params, self.m, self.v, self.step_count)]

    def set_state(self, st):
        for dst, src in zip((self.params, self.m, self.v, self.step_count), st):
            dst.copy_(src)
