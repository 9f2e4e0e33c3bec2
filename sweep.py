#!/usr/bin/env python3
"""Layer execution-time sweeps in the manner of the paper's speed experiments
(section 3.2, Figs. 5-7: channels, kernel size, image size; section 3.3, Fig. 8:
pooling), on one GPU, forward only, with this library's layers beside the
framework's own convolution and pooling as comparators.  Context only: the
paper's figures were taken on another GPU with another library and are not
reproduced here.

Convolution sweeps (B images, C -> S = 2C channels, N x N inputs, n x n kernels):
  fdc_spectral   FDC as section 3.1 times it: the input is already a spectrum
                 [B][C][N][N/2+1]; each call transforms the S zero-padded n x n
                 kernels (fdc_rfft2) and forms the CIC product (fdc_cic_forward),
                 leaving the output a spectrum [B][S][N][N/2+1]
  fdc_layer      the CIC layer with spatial kernels, spatial in and out
                 (fdc_cic_spatial_layer_forward: rfft2, kernel spectra, product,
                 irfft2, CROP; no pooling), n <= 8
  full_fdc       the Full FDC layer, spatial in and out (fdc_full_forward, CROP), n <= 5
  conv2d         torch conv2d over all C input channels (MIOpen), the conventional
                 convolution the paper compares against
  conv2d_native  the same with MIOpen disabled (the framework's own im2col + GEMM),
                 the paper's "spatial convolution"; skipped above --native-max-gflop
  conv2d_dw      depthwise conv2d (groups = C, S outputs): what CIC computes
                 (CROP = a valid convolution with flipped kernels), for reference
Pooling sweep (B images of C channels, N x N -> N/2 x N/2):
  fdp            fdp_forward on spectra [B][C][N][N/2+1] -> [B][C][N/2][N/4+1]
  max_pool2d, avg_pool2d   2 x 2 windows on the spatial images

Every input is seeded and synthetic (N(0, 1) activations, He-normal kernels); times
are HIP-event averages over repeated calls after warm-up, on torch's current stream.
Prints one JSON line per case and a markdown table per sweep.
"""

import argparse
import json
import math
import os
import sys

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

CHANNELS = [(c, 2 * c) for c in (1, 2, 4, 8, 16, 32, 64, 128, 256)]
KERNELS = [1, 3, 5, 7, 9, 11]
SIZES = [32, 64, 128, 256, 512, 1024]
CONV_METHODS = ["fdc_spectral", "fdc_layer", "full_fdc", "conv2d", "conv2d_native", "conv2d_dw"]
POOL_METHODS = ["fdp", "max_pool2d", "avg_pool2d"]


def time_call(torch, fn, target_ms=150.0, max_reps=50):
    """Average milliseconds per call of fn (HIP events on the current stream)."""
    stream = torch.cuda.current_stream()
    fn()
    fn()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    fn()
    b.record(stream)
    torch.cuda.synchronize()
    first = max(a.elapsed_time(b), 1e-3)
    reps = max(3, min(max_reps, int(math.ceil(target_ms / first))))
    a.record(stream)
    for _ in range(reps):
        fn()
    b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / reps, reps


def conv_case(torch, F, layers, _lib, B, C, S, N, n, methods, native_max_gflop, seed):
    """{method: ms or None (unsupported / skipped)} for one convolution case."""
    g = torch.Generator(device="cuda").manual_seed(seed)
    dev = torch.device("cuda")
    x = torch.randn((B, C, N, N), generator=g, device=dev)
    std = math.sqrt(2.0 / (n * n))
    w_dw = torch.randn((S, n, n), generator=g, device=dev) * std          # CIC / depthwise: one n x n per output
    w_full = torch.randn((S, C, n, n), generator=g, device=dev) * math.sqrt(2.0 / (C * n * n))
    out = {}
    nf = N // 2 + 1
    s = layers._stream()
    for m in methods:
        fn = None
        if m == "fdc_spectral":
            X = torch.randn((B, C, N, nf), generator=g, device=dev, dtype=torch.complex64)
            wpad = torch.zeros((S, N, N), device=dev)
            wpad[:, :n, :n] = w_dw
            K = torch.empty((S, N, nf), device=dev, dtype=torch.complex64)
            Y = torch.empty((B, S, N, nf), device=dev, dtype=torch.complex64)
            plan = layers.FftPlan(S, N, N)

            def fn(plan=plan, wpad=wpad, K=K, X=X, Y=Y):
                _lib.call("fdc_rfft2", plan._p, layers._ptr(wpad), layers._ptr(K), None, 0, s)
                _lib.call("fdc_cic_forward", layers._ptr(X), layers._ptr(K), layers._ptr(Y), B, C, S, N, nf, s)
        elif m == "fdc_layer":
            if n > 8 or n > N:
                out[m] = None
                continue
            lay = layers.CicSpatialLayer(B, C, S, N, N, n, artifact="crop")
            y = lay.new_output()

            def fn(lay=lay, y=y):
                lay.forward(x, w_dw, y=y)
        elif m == "full_fdc":
            if n > 5 or n > N:
                out[m] = None
                continue
            lay = layers.FullLayer(B, C, S, N, kernel_n=n, artifact="crop")
            y = lay.new_output()

            def fn(lay=lay, y=y):
                lay.forward(x, w_full, y=y)
        elif m == "conv2d":
            def fn():
                F.conv2d(x, w_full)
        elif m == "conv2d_native":
            gflop = 2.0 * B * S * C * n * n * (N - n + 1) ** 2 / 1e9
            if gflop > native_max_gflop:
                out[m] = None
                continue

            def fn():
                with torch.backends.cudnn.flags(enabled=False):
                    F.conv2d(x, w_full)
        elif m == "conv2d_dw":
            w4 = w_dw.view(S, 1, n, n)

            def fn(w4=w4):
                F.conv2d(x, w4, groups=C)
        ms, reps = time_call(torch, fn)
        out[m] = ms
        torch.cuda.empty_cache()
    return out


def pool_case(torch, F, layers, _lib, B, C, N, seed):
    g = torch.Generator(device="cuda").manual_seed(seed)
    dev = torch.device("cuda")
    x = torch.randn((B, C, N, N), generator=g, device=dev)
    X = torch.randn((B, C, N, N // 2 + 1), generator=g, device=dev, dtype=torch.complex64)
    M = N // 2
    Y = torch.empty((B, C, M, M // 2 + 1), device=dev, dtype=torch.complex64)
    s = layers._stream()
    fns = {
        "fdp": lambda: _lib.call("fdp_forward", layers._ptr(X), layers._ptr(Y), B * C, N, N, M, M, s),
        "max_pool2d": lambda: F.max_pool2d(x, 2),
        "avg_pool2d": lambda: F.avg_pool2d(x, 2),
    }
    return {m: time_call(torch, f)[0] for m, f in fns.items()}


def table(title, key, rows, methods):
    lines = [f"### {title}", "", f"| {key} | " + " | ".join(methods) + " |",
             "|---|" + "---|" * len(methods)]
    for label, res in rows:
        cells = [("—" if res.get(m) is None else f"{res[m]:.3f}") for m in methods]
        lines.append(f"| {label} | " + " | ".join(cells) + " |")
    return "\n".join(lines) + "\n"


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--sweep", choices=["channels", "kernel", "size", "pool", "all"], default="all")
    ap.add_argument("--batch", type=int, default=4, help="images per call (the paper's batch size of section 3.1)")
    ap.add_argument("--native-max-gflop", type=float, default=2000.0,
                    help="skip conv2d_native above this many GFLOP per call")
    args = ap.parse_args()

    import torch
    import torch.nn.functional as F

    from paper_2106_12736_amd import _lib, layers

    if not torch.cuda.is_available():
        sys.exit("sweep.py needs a GPU")
    torch.cuda.set_device(0)
    _lib.lib()  # fails loudly if libfdc.so is not built
    torch.backends.cudnn.benchmark = False
    B = args.batch
    md = []

    def emit(sweep, case, res):
        print(json.dumps({"sweep": sweep, **case, "ms": res}), flush=True)

    if args.sweep in ("channels", "all"):
        rows = []
        for C, S in CHANNELS:
            case = {"batch": B, "cin": C, "cout": S, "size": 512, "kernel": 3}
            res = conv_case(torch, F, layers, _lib, B, C, S, 512, 3, CONV_METHODS, args.native_max_gflop, 1)
            emit("channels", case, res)
            rows.append((f"{C}/{S}", res))
        md.append(table(f"Channels (cf. Fig. 5): {B} images of 512 x 512, 3 x 3 kernels, ms per forward call",
                        "Cin/Cout", rows, CONV_METHODS))
    if args.sweep in ("kernel", "all"):
        rows = []
        for n in KERNELS:
            case = {"batch": B, "cin": 8, "cout": 16, "size": 512, "kernel": n}
            res = conv_case(torch, F, layers, _lib, B, 8, 16, 512, n, CONV_METHODS, args.native_max_gflop, 2)
            emit("kernel", case, res)
            rows.append((f"{n} x {n}", res))
        md.append(table(f"Kernel size (cf. Fig. 6): {B} images of 512 x 512, 8 -> 16 channels, ms per forward call",
                        "kernel", rows, CONV_METHODS))
    if args.sweep in ("size", "all"):
        for n in (3, 5):
            rows = []
            for N in SIZES:
                case = {"batch": B, "cin": 8, "cout": 16, "size": N, "kernel": n}
                res = conv_case(torch, F, layers, _lib, B, 8, 16, N, n, CONV_METHODS, args.native_max_gflop, 3)
                emit("size", case, res)
                rows.append((f"{N} x {N}", res))
            md.append(table(f"Image size (cf. Fig. 7), {n} x {n} kernels: {B} images, 8 -> 16 channels, "
                            "ms per forward call", "input", rows, CONV_METHODS))
    if args.sweep in ("pool", "all"):
        rows = []
        for N in SIZES:
            case = {"batch": B, "channels": 16, "size": N}
            res = pool_case(torch, F, layers, _lib, B, 16, N, 4)
            emit("pool", case, res)
            rows.append((f"{N} x {N}", res))
        md.append(table(f"Pooling to half size (cf. Fig. 8): {B} images of 16 channels, ms per call",
                        "input", rows, POOL_METHODS))
    print("\n" + "\n".join(md), flush=True)


if __name__ == "__main__":
    main()
