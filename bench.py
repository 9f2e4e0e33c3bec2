#!/usr/bin/env python3
"""Throughput of the fused CIC + FDP layer stack, forward + backward, on one GPU.

Workload (the paper's large-image setting, section 2.5.1 / 3.2, with synthetic
fundus-like inputs in place of the APTOS 2019 photographs): batch 8 of 1024 x 1024
grayscale images, five CIC + FDP layers with channel fan-out
1 -> 8 -> 16 -> 32 -> 64 -> 128 and FDP halving the size after each layer
(1024 -> 512 -> 256 -> 128 -> 64 -> 32).  One step = every layer forward
(rfft2 -> CIC -> FDP -> irfft2) and every layer backward (kernel gradients of
all layers, activation gradients of layers 2..5; the gradient of the input
image is not part of a training step).  Inputs are resident in HBM before the
timed region starts.  The step runs through the stack executor (fdc_cic_stack_*),
which performs every layer's transforms but keeps the activations between layers
in registers; --per-layer times the layer-by-layer calls instead (same results up
to fp32 rounding).

With --workload full_fdc_<P>_c<C> it times one Full FDC layer instead (16 images of
P x P, C -> C channels, 3 x 3 weights, crop): forward, then dL/dx and dL/dw; the
roofline of its dominant kernel is then taken against the fp32 matrix-core peak.

Prints ONE JSON line (see --help).  The step is captured once as a HIP graph
and the timed region replays it K times (--eager times plain launches).  Besides
the step time it reports, for the kernel that takes most of the step, its
algorithmic bytes per launch divided by its average launch duration (HIP events
around that kernel's launches on the stream it runs on, over a second timed
region of K eager steps), and the float64 CPU oracle timed on a bounded sample
of the same workload.
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, published peak
MFMA_F32_PEAK_TFLOPS = 157.3  # MI355X dense fp32 matrix-core peak
METRIC = "images/sec fwd+bwd of FDC/FDP stack at 1024² fp32; % peak HBM GB/s (and MFMA %)"
C64, F32 = 8, 4


# ----------------------------------------------------------------------------
# algorithmic bytes: each tensor a kernel must read or write, counted once
# ----------------------------------------------------------------------------

def layer_dims(wl, i):
    N, M = wl.sizes[i], wl.sizes[i + 1]
    C, S = wl.channels[i], wl.channels[i + 1]
    return wl.batch, C, S, N, M, M // 2 + 1, N // 2 + 1


def fwd_col_launches(B, C, S, N, M, L):
    """The forward's column work of one layer: the column DFT with the FDP crop (writes
    the saved spectrum) and the CIC product with the inverse column DFT, in one kernel
    when an input channel has 1, 2 or 4 output channels (or 8, at N <= 256), else in two.
    At 8 the kernel's two channel groups each read the input columns; the model counts
    them once (algorithmic bytes)."""
    if S // C in (1, 2, 4) or (S // C == 8 and N <= 256):
        return [(f"col_fwd_cic_{N}_{M}", C64 * (B * C * N * L + B * C * M * L + S * M * L + B * S * M * L))]
    return [(f"col_fwd_crop_{N}_{M}", C64 * (B * C * N * L + B * C * M * L)),
            (f"col_cic_inv_{N}_{M}", C64 * (B * C * M * L + S * M * L + B * S * M * L))]


def gk_launches(B, C, S, N, M, L, NF, ranges=1, zeros=True):
    """dK of one layer: one launch that reads the upstream and saved spectra and writes
    all of gK (zeros where FDP drops; with zeros=False only the kept bins, the zeros
    coming from the launch before or already in the buffer), or, with the batch cut
    into R ranges, the range sums written by that launch and added in order by a
    second one."""
    gk_bytes = S * N * NF if zeros else S * M * L
    if ranges <= 1:
        return [(f"col_bwd_gk_{M}", C64 * (B * S * M * L + B * C * M * L + gk_bytes))]
    R = ranges
    return [(f"col_bwd_gk_{M}", C64 * (B * S * M * L + B * C * M * L + R * S * M * L)),
            ("gk_reduce", C64 * (R * S * M * L + gk_bytes))]


def step_launches(wl, input_grad=False, ranges=None):
    """(kernel name, algorithmic bytes) of every launch of one step, in launch order;
    ranges[i]: dK batch ranges of layer i (fdc_cic_layer_dk_ranges, default 1)."""
    ranges = ranges or [1] * wl.layers
    out = []
    for i in range(wl.layers):
        B, C, S, N, M, L, _ = layer_dims(wl, i)
        out.append((f"row_r2c_{N}", F32 * B * C * N * N + C64 * B * C * N * L))
        out += fwd_col_launches(B, C, S, N, M, L)
        out.append((f"row_c2r_{M}", C64 * B * S * M * L + F32 * B * S * M * M))
    for i in reversed(range(wl.layers)):
        B, C, S, N, M, L, NF = layer_dims(wl, i)
        out.append((f"row_r2c_{M}", F32 * B * S * M * M + C64 * B * S * M * L))
        out += gk_launches(B, C, S, N, M, L, NF, ranges[i])
        if i > 0 or input_grad:
            out.append((f"col_bwd_gx_{N}_{M}", C64 * (B * S * M * L + S * M * L + B * C * N * L)))
            out.append((f"row_c2r_{N}", C64 * B * C * N * L + F32 * B * C * N * N))
    return out


def tail_launches(wl, a, input_grad=False, kept=False):
    """The stack's last two layers (a, a + 1) run by the LDS-resident tail kernels:
    (forward launch, [backward launch, in-order dK sums of both layers]).
    Bytes: what crosses HBM -- the previous layer's column-inverted spectra (or the
    input image), both kernels at the kept bins, both saved spectra, the output;
    backward the upstream gradient, both saved spectra and kernels, the per-image dK
    products (written, then read by the in-order sums) and the previous layer's
    upstream-gradient spectrum (or the input gradient); kept: the dK sums write the
    kept bins of gK only."""
    B, C, S, N, M, L, NF = layer_dims(wl, a)
    _, _, S2, _, M2, L2, NF2 = layer_dims(wl, a + 1)
    k_bytes = C64 * (S * M * L + S2 * M2 * L2)
    saved_bytes = C64 * (B * C * M * L + B * S * M2 * L2)
    out_bytes = F32 * B * S2 * M2 * M2
    in_bytes = C64 * B * C * N * NF if a > 0 else F32 * B * C * N * N
    part_a, part_b = C64 * B * S * M * L, C64 * B * S2 * M2 * L2
    name = f"{N}_{M}_{M2}"
    fwd = (f"tail_fwd_{name}", in_bytes + k_bytes + saved_bytes + out_bytes)
    dx_bytes = in_bytes if (a > 0 or input_grad) else 0
    bwd = [(f"tail_bwd_{name}", out_bytes + saved_bytes + k_bytes + part_a + part_b + dx_bytes),
           ("gk_reduce", part_a + part_b + (k_bytes if kept else C64 * (S * N * NF + S2 * M * NF2)))]
    return fwd, bwd


def fused_step_launches(wl, input_grad=False, ranges=None, tail=-1, kept=False):
    """(kernel name, algorithmic bytes) of every launch of one step of the fused stack
    executor: as step_launches, with each layer boundary's inverse rows and the next
    layer's forward rows (and the backward's adjoint pair) in one kernel, a layer's
    dK and dX columns in one launch when dK uses one batch range, and the last two
    layers in the LDS-resident tail kernels from layer `tail` on (-1: none); kept: the
    backward writes only the kept bins of gK (fdc_cic_stack_backward_kept)."""
    return fused_fwd_launches(wl, tail) + fused_bwd_launches(wl, input_grad, ranges, tail, kept)


def fused_fwd_launches(wl, tail=-1):
    out = []
    n = wl.layers
    for i in range(n):
        B, C, S, N, M, L, _ = layer_dims(wl, i)
        if i == tail:
            out.append(tail_launches(wl, tail, False)[0])
            break
        if i == 0:
            out.append((f"row_r2c_{N}", F32 * B * C * N * N + C64 * B * C * N * L))
        out += fwd_col_launches(B, C, S, N, M, L)
        if i + 1 == tail:
            continue
        if i + 1 < n:
            _, _, _, N2, M2, L2, _ = layer_dims(wl, i + 1)
            out.append((f"row_c2r_r2c_{M}", C64 * B * S * M * L + C64 * B * S * N2 * L2))
        else:
            out.append((f"row_c2r_{M}", C64 * B * S * M * L + F32 * B * S * M * M))
    return out


def fused_bwd_launches(wl, input_grad=False, ranges=None, tail=-1, kept=False):
    ranges = ranges or [1] * wl.layers
    out = []
    n = wl.layers

    def merged(i):  # dK and dX of layer i in one launch
        N = wl.sizes[i]
        return (i > 0 or input_grad) and ranges[i] <= 1 and N <= 256

    def zeros_early(i):  # layer i's gK zeros written by layer i + 1's boundary rows
        return not kept and i + 1 < n and not (tail >= 0 and i + 1 >= tail) and not merged(i) and ranges[i] <= 1

    for i in reversed(range(n)):
        B, C, S, N, M, L, NF = layer_dims(wl, i)
        if tail >= 0 and i >= tail:
            if i == tail + 1:
                out += tail_launches(wl, tail, input_grad, kept)[1]
            continue
        if i == n - 1:
            out.append((f"row_r2c_{M}", F32 * B * S * M * M + C64 * B * S * M * L))
        dx = i > 0 or input_grad
        gx_bytes = C64 * (B * S * M * L + S * M * L + B * C * N * L)
        if merged(i):
            # dK and dX columns in one launch (layers of at most 256 points): the bytes of both
            (_, gk_bytes), = gk_launches(B, C, S, N, M, L, NF, 1, zeros=not kept)
            out.append((f"col_bwd_dk_dx_{N}_{M}", gk_bytes + gx_bytes))
        else:
            out += gk_launches(B, C, S, N, M, L, NF, ranges[i], zeros=not kept and not zeros_early(i))
            if dx:
                out.append((f"col_bwd_gx_{N}_{M}", gx_bytes))
        if dx:
            if i > 0:
                _, _, Sp, Np, Mp, Lp, NFp = layer_dims(wl, i - 1)
                zero_bytes = C64 * (Sp * Np * NFp - Sp * Mp * Lp) if zeros_early(i - 1) else 0
                out.append((f"row_c2r_r2c_{N}", C64 * B * C * N * L + C64 * B * C * Mp * Lp + zero_bytes))
            else:
                out.append((f"row_c2r_{N}", C64 * B * C * N * L + F32 * B * C * N * N))
    return out


def fft2_launches(n, planes, inverse):
    """(kernel name, algorithmic bytes) of one n x n rfft2 (or irfft2, inverse=True) of
    `planes` planes: one launch for square planes up to 64 x 64, else rows then columns."""
    nf = n // 2 + 1
    real, spec = F32 * planes * n * n, C64 * planes * n * nf
    if n in (16, 32, 64):
        return [(f"fft2_small_{'inv' if inverse else 'fwd'}_{n}", real + spec)]
    if inverse:
        return [(f"col_fft_inv_{n}", 2 * spec), (f"row_c2r_{n}", spec + real)]
    return [(f"row_r2c_{n}", real + spec), (f"col_fft_fwd_{n}", 2 * spec)]


def pooled_rfft2_launches(n, m, planes):
    """(kernel name, algorithmic bytes) of fdc_rfft2_pooled_ws: n x n planes to the bins an
    FDP to m x m keeps (m/2+1 columns of every row into the workspace, then m rows of
    those columns)."""
    if n in (16, 32, 64):
        return fft2_launches(n, planes, inverse=False)
    L = m // 2 + 1
    real = F32 * planes * n * n
    return [(f"row_r2c_{n}", real + C64 * planes * n * L), (f"col_fft_keep_{n}", C64 * planes * (n + m) * L)]


def chain_step_launches(wl, input_grad=False, hermitian=False):
    """(kernel name, algorithmic bytes) of every launch of one step of the FDCNN chain
    (one rfft2, every FDC + FDP layer on spectra, one irfft2, and the backward); with
    hermitian=True the layers' launches also apply Pi_H, with the same launches (the
    backward also writing columns 0 and N/2 of dX over every row)."""
    out = []
    n = wl.layers
    B = wl.batch
    N0, C0 = wl.sizes[0], wl.channels[0]
    NF0 = N0 // 2 + 1
    ML, CL = wl.sizes[-1], wl.channels[-1]
    MFL = ML // 2 + 1
    out += pooled_rfft2_launches(N0, wl.sizes[1], B * C0)
    for i in range(n):
        B, C, S, N, M, L, NF = layer_dims(wl, i)
        # (with hermitian=True, Pi_H of the output is part of the same launch)
        out.append(("cic_fdp_fwd", C64 * (B * C * M * L + S * M * L + B * S * M * L)))
    out += fft2_launches(ML, B * CL, inverse=True)
    out += fft2_launches(ML, B * CL, inverse=False)  # the irfft2 adjoint has the forward's launches
    for i in reversed(range(n)):
        B, C, S, N, M, L, NF = layer_dims(wl, i)
        # dX and dK in one launch (fdc_cic_fdp_backward_kept; with hermitian=True and
        # i > 0, Pi_H of dX in it too): gY, and X at the kept bins, read; gK written at the
        # kept bins (the chain's buffers hold zeros at the others); with dX also K at the
        # kept bins read and gX written at the kept bins (projected: also columns 0 and
        # N/2 of the other rows)
        nb = C64 * (B * S * M * L + B * C * M * L + S * M * L)
        if i > 0 or input_grad:
            nb += C64 * (S * M * L + B * C * M * L)
            if hermitian and i > 0:
                nb += C64 * B * C * ((N - M) + (N if M < N else 0))
        out.append(("cic_fdp_bwd", nb))
    if input_grad:
        out += fft2_launches(N0, B * C0, inverse=True)
    return out


def classifier_step_launches(wl, classes, n_params):
    """One training step of the FDCNN classifier: the chain forward, the head forward
    (ReLU + fully connected layer, then the loss), the head backward, the chain backward
    (no input gradient), and the Adam update of every parameter (plus its step count)."""
    chain = chain_step_launches(wl, False)
    # rfft2, the layers, irfft2
    n_fwd = (len(fft2_launches(wl.sizes[0], 1, False)) + wl.layers +
             len(fft2_launches(wl.sizes[-1], 1, True)))
    B, F = wl.batch, wl.channels[-1] * wl.sizes[-1] ** 2
    chunks = -(-F // 1024)
    head = [
        ("head_fwd", F32 * (B * F + classes * F + B * chunks * classes)),
        ("head_loss", F32 * (B * chunks * classes + classes + 2 * B * classes)),
        ("head_bwd", F32 * (2 * B * F + 2 * classes * F + B * classes)),
    ]
    return chain[:n_fwd] + head + chain[n_fwd:] + [("adam", 7 * F32 * n_params), ("adam_count", 8)]


def spatial_step_launches(wl, n, input_grad=False, ranges=None):
    """(kernel name, algorithmic bytes) of every launch of one step of the stack with
    n x n spatial kernels (layer by layer, ROLL): step_launches plus the kernel-spectrum
    formation before each layer's product and the weight-gradient projection."""
    ranges = ranges or [1] * wl.layers
    out = []
    for i in range(wl.layers):
        B, C, S, N, M, L, _ = layer_dims(wl, i)
        out.append(("cic_kspec", F32 * S * n * n + C64 * S * M * L))
        out.append((f"row_r2c_{N}", F32 * B * C * N * N + C64 * B * C * N * L))
        out += fwd_col_launches(B, C, S, N, M, L)
        out.append((f"row_c2r_{M}", C64 * B * S * M * L + F32 * B * S * M * M))
    for i in reversed(range(wl.layers)):
        B, C, S, N, M, L, NF = layer_dims(wl, i)
        gx = i > 0 or input_grad
        if gx:
            out.append(("cic_kspec", F32 * S * n * n + C64 * S * M * L))
        out.append((f"row_r2c_{M}", F32 * B * S * M * M + C64 * B * S * M * L))
        out += gk_launches(B, C, S, N, M, L, NF, ranges[i])
        if gx:
            out.append((f"col_bwd_gx_{N}_{M}", C64 * (B * S * M * L + S * M * L + B * C * N * L)))
            out.append((f"row_c2r_{N}", C64 * B * C * N * L + F32 * B * C * N * N))
        out.append(("cic_wgrad", C64 * S * M * L))
        out.append(("cic_wgrad_reduce", F32 * S * n * n))
    return out


def spatial_fused_step_launches(wl, n, input_grad=False, ranges=None, tail=-1):
    """(kernel name, algorithmic bytes) of every launch of one step of the stack with
    n x n spatial kernels through the stack executor (fdc_cic_spatial_stack_*): every
    layer's kernel spectra in one launch before the forward and before the backward,
    the fused executor's launches, and every layer's dL/dw in one launch plus the sum
    of its partials."""
    kspec = wgrad = reduce_ = 0
    for i in range(wl.layers):
        B, C, S, N, M, L, _ = layer_dims(wl, i)
        rb = 32 if M >= 256 else (16 if M >= 64 else 4)
        kspec += F32 * S * n * n + C64 * S * M * L
        wgrad += C64 * S * M * L + F32 * S * rb * n * n
        reduce_ += F32 * S * rb * n * n + F32 * S * n * n
    return ([("cic_kspec_stack", kspec)] + fused_fwd_launches(wl, tail) + [("cic_kspec_stack", kspec)] +
            fused_bwd_launches(wl, input_grad, ranges, tail) +
            [("cic_wgrad_stack", wgrad), ("cic_wgrad_stack_reduce", reduce_)])


def step_api_bytes(wl, input_grad=False):
    """Bytes of the tensors that cross the layer interface in one step, each counted once:
    forward x, K at the kept bins, y; backward g, K, the saved pooled spectrum, gx, gK at kept bins."""
    total = 0
    for i in range(wl.layers):
        B, C, S, N, M, L, _ = layer_dims(wl, i)
        total += F32 * B * C * N * N + C64 * S * M * L + F32 * B * S * M * M
        total += F32 * B * S * M * M + C64 * S * M * L + C64 * B * C * M * L + C64 * S * M * L
        if i > 0 or input_grad:
            total += F32 * B * C * N * N
    return total


def full_step_launches(wl):
    """(kernel name, algorithmic amount, unit) of every launch of one Full FDC step
    (forward, dL/dw, dL/dx).  Matrix-core kernels count flops (8 per complex
    multiply-add of the per-bin contraction), the others HBM bytes."""
    B, Ci, Co, P, n = wl.batch, wl.cin, wl.cout, wl.size, wl.n
    NB = P * (P // 2 + 1)
    O = P - n + 1
    wbytes = F32 * Co * Ci * n * n
    flops = 8 * B * Ci * Co * NB
    return [
        (f"row_r2c_{P}", F32 * B * Ci * P * P + C64 * B * Ci * NB, "B"),
        (f"col_fft_fwd_{P}", 2 * C64 * B * Ci * NB, "B"),
        ("full_weights", 2 * wbytes, "B"),
        ("full_contract_fwd", flops, "flop"),
        (f"col_fft_inv_{P}", 2 * C64 * B * Co * NB, "B"),
        (f"row_c2r_{P}", C64 * B * Co * NB + F32 * B * Co * O * O, "B"),
        (f"row_r2c_{P}", F32 * B * Co * O * O + C64 * B * Co * NB, "B"),
        (f"col_fft_fwd_{P}", 2 * C64 * B * Co * NB, "B"),
        ("full_gw", flops, "flop"),
        ("full_gw_reduce", wbytes, "B"),  # dL/dw written once; its per-chunk partial sums are scratch
        ("full_weights", 2 * wbytes, "B"),
        ("full_contract_gx", flops, "flop"),
        (f"col_fft_inv_{P}", 2 * C64 * B * Ci * NB, "B"),
        (f"row_c2r_{P}", C64 * B * Ci * NB + F32 * B * Ci * P * P, "B"),
    ]


def full_api_bytes(wl):
    """x, w, y forward; gy, saved rfft2(x), w, gx, gw backward."""
    B, Ci, Co, P, n = wl.batch, wl.cin, wl.cout, wl.size, wl.n
    O = P - n + 1
    w = F32 * Co * Ci * n * n
    spec = C64 * B * Ci * P * (P // 2 + 1)
    return (F32 * B * Ci * P * P + w + F32 * B * Co * O * O) + (F32 * B * Co * O * O + spec + 2 * w + F32 * B * Ci * P * P)


def kernel_source_digest():
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2106_12736_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        if f.endswith((".hip", ".h")):
            with open(os.path.join(csrc, f), "rb") as fh:
                h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()


def measured_traffic(kernel, workload):
    """HBM bytes per launch from the committed rocprofv3 counter summary of this kernel,
    or None when there is none or the kernel sources changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_sha256") != kernel_source_digest():
        return None
    return rec["hbm_bytes_per_launch"]


# ----------------------------------------------------------------------------
# CPU baseline: the float64 oracle on the host cores
# ----------------------------------------------------------------------------

def cpu_baseline(wl, data, min_seconds=10.0, max_reps=50, chain=False):
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import fdc

    x = data.x.astype(np.float64)
    kd = [k.astype(np.complex128) for k in data.kernels]
    g = data.grad.astype(np.float64)
    reps, t0 = 0, time.perf_counter()
    fwd, bwd = (fdc.cic_chain_forward, fdc.cic_chain_backward) if chain else (fdc.cic_stack_forward,
                                                                              fdc.cic_stack_backward)
    while True:
        _, saved = fwd(x, kd, wl.sizes)
        bwd(g, saved, kd, wl.sizes, want_input_grad=False)
        reps += 1
        el = time.perf_counter() - t0
        if el >= min_seconds or reps >= max_reps:
            break
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    return {
        "value": reps * wl.batch / el,
        "unit": "images/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"{reps} full step(s) of the same workload (batch {wl.batch}, all {wl.layers} layers, "
                  f"fwd+bwd, float64) in {el:.1f} s on {os.cpu_count()} host CPUs visible",
    }


def spatial_cpu_baseline(wl, data, min_seconds=10.0, max_reps=50):
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import fdc

    x = data.x.astype(np.float64)
    ws = [w.astype(np.float64) for w in data.weights]
    g0 = data.grad.astype(np.float64)
    reps, t0 = 0, time.perf_counter()
    while True:
        h, saved = x, []
        for i in range(wl.layers):
            h, xs = fdc.cic_spatial_layer_forward(h, ws[i], wl.sizes[i + 1], fdc.ARTIFACT_ROLL)
            saved.append(xs)
        g = g0
        for i in reversed(range(wl.layers)):
            g, _ = fdc.cic_spatial_layer_backward(g, saved[i], ws[i], wl.sizes[i + 1], fdc.ARTIFACT_ROLL,
                                                  want_gx=i > 0)
        reps += 1
        el = time.perf_counter() - t0
        if el >= min_seconds or reps >= max_reps:
            break
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    return {"value": reps * wl.batch / el, "unit": "images/s", "cores": threads, "kind": "oracle",
            "sample": f"{reps} full step(s) of the same workload (batch {wl.batch}, all {wl.layers} layers, "
                      f"fwd+bwd, float64) in {el:.1f} s on {os.cpu_count()} host CPUs visible"}


# ----------------------------------------------------------------------------
# main
# ----------------------------------------------------------------------------

def classifier_cpu_baseline(wl, data, W, bias, labels, min_seconds=10.0, max_reps=50):
    """The oracle's training step of the classifier (chain, head, Adam) on the same
    inputs, repeated to about min_seconds."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import classifier

    x = data.x.astype(np.float64)
    kd = [k.astype(np.complex128) for k in data.kernels]
    reps, t0 = 0, time.perf_counter()
    while True:
        _, _, gks, gW, gb = classifier.classifier_gradients(x, kd, W, bias, labels, wl.sizes)
        flat_p = np.concatenate([np.concatenate([k.view(np.float64).ravel() for k in kd]), W.ravel(), bias])
        flat_g = np.concatenate([np.concatenate([g.view(np.float64).ravel() for g in gks]), gW.ravel(), gb])
        classifier.adam_step(flat_p, flat_g, 0 * flat_p, 0 * flat_p, 1, 1e-5, 0.9, 0.999, 1e-8, 1e-6)
        reps += 1
        el = time.perf_counter() - t0
        if el >= min_seconds or reps >= max_reps:
            break
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    return {
        "value": reps * wl.batch / el,
        "unit": "images/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"{reps} full training step(s) of the same workload (batch {wl.batch}, chain of {wl.layers} "
                  f"layers, head, Adam, float64) in {el:.1f} s on {os.cpu_count()} host CPUs visible",
    }


class CicStackRun:
    """The CIC + FDP stack step on preallocated buffers: the fused stack executor
    (fdc_cic_stack_*), or the layer-by-layer calls with --per-layer."""

    def __init__(self, wl, args, dev):
        import torch

        from paper_2106_12736_amd import inputs, layers
        self.wl = wl
        self.data = inputs.make_cic_stack(wl)
        self.x = torch.from_numpy(self.data.x).to(dev)
        self.Ks = [torch.from_numpy(k).to(dev) for k in self.data.kernels]
        self.g = torch.from_numpy(self.data.grad).to(dev)
        self.per_layer = args.per_layer
        self.executor = "chain" if args.chain else ("per_layer" if args.per_layer else "fused_stack")
        self.clf = None
        self.spatial = args.spatial_kernel
        if self.spatial:
            self.data = inputs.make_cic_spatial(wl, self.spatial)
            self.x = torch.from_numpy(self.data.x).to(dev)
            self.Ks = [torch.from_numpy(w).to(dev) for w in self.data.weights]
            self.g = torch.from_numpy(self.data.grad).to(dev)
            if self.per_layer:
                self.stack = layers.CicSpatialStack(wl.batch, wl.sizes, wl.channels, self.spatial, device=dev)
                model = lambda w_, ig: spatial_step_launches(w_, self.spatial, ig, self.stack.dk_ranges())  # noqa: E731
            else:
                self.executor = "fused_stack"
                self.stack = layers.CicSpatialStackFused(wl.batch, wl.sizes, wl.channels, self.spatial, device=dev)
                model = lambda w_, ig: spatial_fused_step_launches(  # noqa: E731
                    w_, self.spatial, ig, self.stack.dk_ranges(), self.stack.tail())
        elif args.classifier:
            import numpy as np
            self.executor = "classifier"
            classes = 2
            self.clf = layers.FdcnnClassifier(wl.batch, wl.sizes, wl.channels, classes=classes, device=dev)
            self.stack = self.clf.chain
            F = self.clf.features
            rng = np.random.default_rng(20210700 + wl.index)
            self.W = (rng.standard_normal((classes, F)) * np.sqrt(2.0 / F)).astype(np.float32)
            self.bias = np.zeros(classes, np.float32)
            self.labels = (np.arange(wl.batch) % classes).astype(np.int32)
            self.clf.load(self.Ks, torch.from_numpy(self.W).to(dev), torch.from_numpy(self.bias).to(dev))
            self.labels_d = torch.from_numpy(self.labels).to(dev)
            model = lambda w_, ig: classifier_step_launches(w_, classes, self.clf.n_params)  # noqa: E731
        elif args.chain or args.folded:
            self.executor = "folded_chain" if args.folded else "chain"
            self.stack = layers.CicChain(wl.batch, wl.sizes, wl.channels, device=dev, hermitian=args.folded)
            model = lambda w_, ig: chain_step_launches(w_, ig, hermitian=args.folded)  # noqa: E731
        elif self.per_layer:
            self.stack = layers.CicStack(wl.batch, wl.sizes, wl.channels, device=dev)
            model = lambda w_, ig: step_launches(w_, ig, self.stack.dk_ranges())  # noqa: E731
        else:
            self.stack = layers.CicStackFused(wl.batch, wl.sizes, wl.channels, device=dev)
            model = lambda w_, ig: fused_step_launches(w_, ig, self.stack.dk_ranges(), self.stack.tail(),  # noqa: E731
                                                       kept=True)
        self.gin = (torch.empty((wl.batch, wl.channels[0], wl.sizes[0], wl.sizes[0]), dtype=torch.float32,
                                device=dev) if args.input_grad else None)
        self.input_grad = args.input_grad
        self.launches = [(name, nbytes, "B") for name, nbytes in model(wl, args.input_grad)]
        self.api_bytes = step_api_bytes(wl, args.input_grad)

    def step(self):
        if self.clf is not None:
            self.clf.train_step(self.x, self.labels_d)
            return
        self.stack.forward(self.x, self.Ks)
        self.stack.backward(self.g, self.Ks, input_grad=self.gin)

    def outputs(self):
        if self.clf is not None:
            return [self.clf.loss, self.clf.logits, self.clf.params, self.clf.m, self.clf.v, self.clf.step_count]
        last = self.stack.acts[-1] if self.executor == "per_layer" else self.stack.out
        return [last] + list(self.stack.gws if self.spatial else self.stack.gks)

    def save_state(self):
        """Training state a step changes (classifier only), for the graph replay check."""
        return self.clf.state() if self.clf is not None else None

    def restore_state(self, st):
        if st is not None:
            self.clf.set_state(st)

    def config(self):
        wl = self.wl
        cfg = {"workload": wl.name, "batch": wl.batch, "sizes": list(wl.sizes), "channels": list(wl.channels),
               "input_grad": bool(self.input_grad),
               "executor": self.executor,
               "kernels": f"spatial {self.spatial}x{self.spatial}, roll" if self.spatial else "spectral"}
        if self.executor == "fused_stack":
            cfg["lds_tail_from_layer"] = self.stack.tail()
        if self.clf is not None:
            cfg["head"] = (f"relu, fully connected {self.clf.features} -> {self.clf.classes}, softmax cross-entropy; "
                           f"adam lr {self.clf.lr:g}, weight decay {self.clf.weight_decay:g}")
        return cfg

    def cpu_baseline(self):
        if self.spatial:
            return spatial_cpu_baseline(self.wl, self.data)
        if self.clf is not None:
            return classifier_cpu_baseline(self.wl, self.data, self.W.astype("float64"), self.bias.astype("float64"),
                                           self.labels)
        return cpu_baseline(self.wl, self.data, chain=self.executor == "chain")


def full_cic_step_launches(wl, ranges=1):
    """One step of the Full FDC layer with CIC (spatial kernels, no pooling, crop):
    forward, dL/dx and dL/dw."""
    B, C, S, P, n = wl.batch, wl.cin, wl.cout, wl.size, wl.n
    L = P // 2 + 1
    O = P - n + 1
    return [
        ("cic_kspec", F32 * S * n * n + C64 * S * P * L),
        (f"row_r2c_{P}", F32 * B * C * P * P + C64 * B * C * P * L),
        *fwd_col_launches(B, C, S, P, P, L),
        (f"row_c2r_{P}", C64 * B * S * P * L + F32 * B * S * O * O),
        ("cic_kspec", F32 * S * n * n + C64 * S * P * L),
        (f"row_r2c_{P}", F32 * B * S * O * O + C64 * B * S * P * L),
        *gk_launches(B, C, S, P, P, L, L, ranges),
        (f"col_bwd_gx_{P}_{P}", C64 * (B * S * P * L + S * P * L + B * C * P * L)),
        (f"row_c2r_{P}", C64 * B * C * P * L + F32 * B * C * P * P),
        ("cic_wgrad", C64 * S * P * L),
        ("cic_wgrad_reduce", F32 * S * n * n),
    ]


class FullCicRun:
    """One Full FDC layer with CIC (the paper's VGG16 Conv Block 4 variant): forward,
    dL/dx and dL/dw through fdc_cic_spatial_layer_*."""

    def __init__(self, wl, args, dev):
        import torch

        from paper_2106_12736_amd import inputs, layers
        self.wl = wl
        self.data = inputs.make_full_cic(wl)
        self.x = torch.from_numpy(self.data.x).to(dev)
        self.w = torch.from_numpy(self.data.w).to(dev)
        self.g = torch.from_numpy(self.data.grad).to(dev)
        self.layer = layers.CicSpatialLayer(wl.batch, wl.cin, wl.cout, wl.size, wl.size, wl.n, artifact="crop",
                                            device=dev)
        self.saved = self.layer.new_saved()
        self.y = self.layer.new_output()
        self.gx = torch.empty_like(self.x)
        self.gw = torch.empty_like(self.w)
        self.launches = [(nm, b, "B") for nm, b in full_cic_step_launches(wl, self.layer.dk_ranges())]
        B, C, S, P, n = wl.batch, wl.cin, wl.cout, wl.size, wl.n
        O = P - n + 1
        self.api_bytes = F32 * (2 * B * C * P * P + 2 * B * S * O * O + 3 * S * n * n) + C64 * B * C * P * (P // 2 + 1)

    def step(self):
        self.layer.forward(self.x, self.w, y=self.y, saved=self.saved)
        self.layer.backward(self.g, self.saved, self.w, gx=self.gx, gw=self.gw)

    def outputs(self):
        return [self.y, self.gx, self.gw]

    def config(self):
        wl = self.wl
        return {"workload": wl.name, "batch": wl.batch, "size": wl.size, "cin": wl.cin, "cout": wl.cout,
                "kernel": wl.n, "artifact": "crop", "product": "cic"}

    def cpu_baseline(self, min_seconds=10.0):
        import numpy as np
        from threadpoolctl import threadpool_info

        from oracle import fdc

        wl = self.wl
        x = self.data.x[:1].astype(np.float64)
        w = self.data.w.astype(np.float64)
        g = self.data.grad[:1].astype(np.float64)
        reps, t0 = 0, time.perf_counter()
        while True:
            _, xs = fdc.cic_spatial_layer_forward(x, w, wl.size, fdc.ARTIFACT_CROP)
            fdc.cic_spatial_layer_backward(g, xs, w, wl.size, fdc.ARTIFACT_CROP)
            reps += 1
            el = time.perf_counter() - t0
            if el >= min_seconds or reps >= 50:
                break
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
        return {"value": reps / el, "unit": "images/s", "cores": threads, "kind": "oracle",
                "sample": f"{reps} step(s) of one image of the same layer (fwd, dL/dx, dL/dw, float64) in {el:.1f} s; "
                          f"{os.cpu_count()} host CPUs visible"}


class FullFdcRun:
    """One Full FDC layer step (forward, dL/dx, dL/dw) on preallocated buffers."""

    def __init__(self, wl, args, dev):
        import torch

        from paper_2106_12736_amd import inputs, layers
        self.wl = wl
        self.data = inputs.make_full_fdc(wl)
        self.x = torch.from_numpy(self.data.x).to(dev)
        self.w = torch.from_numpy(self.data.w).to(dev)
        self.g = torch.from_numpy(self.data.grad).to(dev)
        self.layer = layers.FullLayer(wl.batch, wl.cin, wl.cout, wl.size, kernel_n=wl.n, artifact="crop",
                                      device=dev)
        self.saved = self.layer.new_saved()
        self.y = self.layer.new_output()
        self.gx = torch.empty_like(self.x)
        self.gw = torch.empty_like(self.w)
        self.launches = full_step_launches(wl)
        self.api_bytes = full_api_bytes(wl)

    def step(self):
        self.layer.forward(self.x, self.w, y=self.y, saved=self.saved)
        self.layer.backward(self.g, self.saved, self.w, gx=self.gx, gw=self.gw)

    def outputs(self):
        return [self.y, self.gx, self.gw]

    def config(self):
        wl = self.wl
        return {"workload": wl.name, "batch": wl.batch, "size": wl.size, "cin": wl.cin, "cout": wl.cout,
                "kernel": wl.n, "artifact": "crop"}

    def cpu_baseline(self, min_seconds=10.0):
        """The oracle on one image and a slice of the output channels (the layer's work
        grows linearly with the output channels), scaled to the whole layer."""
        import numpy as np
        from threadpoolctl import threadpool_info

        from oracle import fdc

        wl = self.wl
        cs = max(1, wl.cout // 32)
        x = self.data.x[:1].astype(np.float64)
        w = self.data.w[:cs].astype(np.float64)
        g = self.data.grad[:1, :cs].astype(np.float64)
        reps, t0 = 0, time.perf_counter()
        while True:
            _, xs = fdc.full_fdc_forward(x, w, fdc.ARTIFACT_CROP)
            fdc.full_fdc_backward(g, xs, w, fdc.ARTIFACT_CROP)
            reps += 1
            el = time.perf_counter() - t0
            if el >= min_seconds or reps >= 50:
                break
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
        return {
            "value": reps * (cs / wl.cout) / el,
            "unit": "images/s",
            "cores": threads,
            "kind": "oracle",
            "sample": f"{reps} step(s) of one image with {cs} of {wl.cout} output channels (fwd, dL/dx, dL/dw, "
                      f"float64) in {el:.1f} s, scaled by {wl.cout // cs} to all output channels; "
                      f"{os.cpu_count()} host CPUs visible",
        }


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="cic_stack_1024",
                    help="CIC stack (cic_stack_1024 [default], cic_stack_512, ...) or Full FDC layer "
                         "(full_fdc_512_c256, ...) workload")
    ap.add_argument("--no-cpu-baseline", action="store_true", help="skip the oracle timing")
    ap.add_argument("--input-grad", action="store_true", help="CIC stack: also compute the input-image gradient")
    ap.add_argument("--per-layer", action="store_true",
                    help="CIC stack: run the layer-by-layer calls instead of the fused stack executor")
    ap.add_argument("--spatial-kernel", type=int, default=0, metavar="n",
                    help="CIC stack: n x n spatial kernels transformed on every call (ROLL), through the stack "
                         "executor (with --per-layer: layer by layer)")
    ap.add_argument("--chain", action="store_true",
                    help="CIC stack: the FDCNN data flow of section 2.5.1 (one rfft2, FDC + FDP layers on spectra, "
                         "one irfft2); a different function from the per-layer transforms")
    ap.add_argument("--folded", action="store_true",
                    help="CIC stack: the per-layer stack's function (the default workload) computed as the chain of "
                         "--chain with Pi_H between layers, since irfft2 followed by rfft2 is Pi_H")
    ap.add_argument("--classifier", action="store_true",
                    help="CIC stack: one training step of the FDCNN classifier (the chain of --chain, a ReLU, a "
                         "fully connected layer to 2 classes, softmax cross-entropy, Adam)")
    ap.add_argument("--eager", action="store_true", help="time eager launches instead of HIP graph replays")
    ap.add_argument("--flush-mib", type=int, default=512, metavar="MIB",
                    help="buffer written between the individually timed steps of the step-time "
                         "distribution (evicts the last-level cache; 0: no flush)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="after the timed region, run one plain streaming copy kernel (dst = src * 1) over "
                         "MIB MiB, a known-size reference for the HBM traffic counters of a profiler run")
    ap.add_argument("--launch-table", action="store_true",
                    help="print every launch of the instrumented step (work, duration, rate) to stderr")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the method shards over the batch "
              "with one all-reduce of the kernel gradients per layer, which this build does not run.",
              file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2106_12736_amd import _lib, inputs

    workloads = {w.name: w for w in inputs.CIC_WORKLOADS + inputs.FULL_FDC_WORKLOADS + inputs.FULL_CIC_WORKLOADS}
    if args.workload not in workloads:
        sys.exit(f"unknown workload {args.workload}; one of {sorted(workloads)}")
    wl = workloads[args.workload]
    if not torch.cuda.is_available():
        sys.exit("bench.py needs a GPU")
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    _lib.lib()  # fails loudly if libfdc.so is not built

    if isinstance(wl, inputs.FullFdcLayer):
        run = FullFdcRun(wl, args, dev)
    elif isinstance(wl, inputs.FullCicLayer):
        run = FullCicRun(wl, args, dev)
    else:
        run = CicStackRun(wl, args, dev)
    step = run.step
    stream = torch.cuda.current_stream()

    for _ in range(max(args.warmup, 1)):
        step()
    torch.cuda.synchronize()

    # one instrumented step: per-kernel durations, to find the kernel that dominates
    launches = run.launches
    _lib.call("fdc_kernel_timing_enable", len(launches) + 8, None)
    step()
    torch.cuda.synchronize()
    buf = ctypes_buf(1 << 16)
    _lib.call("fdc_kernel_timing_launches", buf, len(buf))
    _lib.call("fdc_kernel_timing_disable")
    recs = [ln.rsplit(" ", 1) for ln in buf.value.decode().strip().splitlines()]
    names = [r[0] for r in recs]
    if names != [n for n, _, _ in launches]:
        sys.exit(f"launch sequence differs from the work model:\n{names}\n{[n for n, _, _ in launches]}")
    per_name = {}
    for (name, amount, unit), (_, ms) in zip(launches, recs):
        t, a, n, _ = per_name.get(name, (0.0, 0, 0, unit))
        per_name[name] = (t + float(ms), a + amount, n + 1, unit)
    if args.launch_table:
        for i, ((name, amount, unit), (_, ms)) in enumerate(zip(launches, recs)):
            rate = amount / (float(ms) * 1e-3) / (1e12 if unit == "flop" else 1e9)
            print(f"launch {i:3d} {name:32s} {amount:14.0f} {unit:6s} {float(ms) * 1e3:9.2f} us "
                  f"{rate:9.1f} {'TFLOP/s' if unit == 'flop' else 'GB/s'}", file=sys.stderr)
    dominant = max(per_name, key=lambda k: per_name[k][0])
    dom_amount_per_step, dom_launches_per_step, dom_unit = per_name[dominant][1:]

    t_start, t_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    # the step captured once as a HIP graph (all buffers are preallocated, so the
    # captured launches reuse them); a replay must reproduce the eager step exactly
    graph = None
    if not args.eager:
        state = run.save_state() if hasattr(run, "save_state") else None
        step()
        torch.cuda.synchronize()
        ref = [t.clone() for t in run.outputs()]
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        if state is not None:  # a training step changes its own state: replay from the same one
            run.restore_state(state)
        graph.replay()
        torch.cuda.synchronize()
        if not all(torch.equal(a, b) for a, b in zip(ref, run.outputs())):
            sys.exit("graph replay does not reproduce the eager step")
        del ref
        for _ in range(max(args.warmup, 1)):
            graph.replay()

    def timed(fn):
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        t_start.record(stream)
        for _ in range(args.steps):
            fn()
        t_end.record(stream)
        torch.cuda.synchronize()
        return t_start.elapsed_time(t_end) / args.steps, (time.perf_counter() - w0) * 1e3 / args.steps

    # timed region 1: K steps (graph replays unless --eager)
    ms_per_step, wall_ms = timed(graph.replay if graph is not None else step)

    # timed region 1b: the same steps bracketed one by one, for the distribution (p10,
    # median, p90); back to back, and with a --flush-mib buffer written between steps
    # (outside the brackets) so that every step starts with its data in HBM, not in the
    # 256 MB last-level cache
    def distribution(fn, flush):
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(args.steps)]
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(evs):
            if flush is not None:
                flush.fill_(float(i & 7))
            a.record(stream)
            fn()
            b.record(stream)
        torch.cuda.synchronize()
        ts = sorted(a.elapsed_time(b) for a, b in evs)
        q = lambda f: ts[min(len(ts) - 1, int(round(f * (len(ts) - 1))))]
        return {"p10": q(0.1), "median": q(0.5), "p90": q(0.9)}

    stepfn = graph.replay if graph is not None else step
    dist = {"back_to_back": distribution(stepfn, None)}
    if args.flush_mib > 0:
        flush = torch.empty(args.flush_mib * (1 << 20) // 4, dtype=torch.float32, device=dev)
        dist["flushed"] = distribution(stepfn, flush)
        dist["flushed"]["flush_mib"] = args.flush_mib
        del flush

    # timed region 2: K eager steps, the dominant kernel's launches bracketed by HIP events
    # on the stream they run on (events cannot be placed inside a replayed graph)
    _lib.call("fdc_kernel_timing_enable", args.steps * dom_launches_per_step, dominant.encode())
    eager_ms_per_step, _ = timed(step)
    _lib.call("fdc_kernel_timing_disable")
    buf = ctypes_buf(1 << 20)
    _lib.call("fdc_kernel_timing_launches", buf, len(buf))
    dom_ms = [float(ln.rsplit(" ", 1)[1]) for ln in buf.value.decode().strip().splitlines()]

    dom_avg_ms = sum(dom_ms) / len(dom_ms)
    per_launch = dom_amount_per_step / dom_launches_per_step
    if dom_unit == "flop":
        achieved = per_launch / (dom_avg_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "kernel": dominant, "achieved": achieved, "peak": MFMA_F32_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": achieved / MFMA_F32_PEAK_TFLOPS, "traffic": None,
                "flops_per_launch": per_launch}
    else:
        achieved = per_launch / (dom_avg_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "kernel": dominant, "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBPS, "traffic": measured_traffic(dominant, wl.name),
                "bytes_per_launch": per_launch}
    roof["avg_launch_ms"] = dom_avg_ms
    roof["share_of_step"] = sum(dom_ms) / args.steps / eager_ms_per_step

    cfg = run.config()
    cfg.update({"launches_per_step": len(launches), "hip_graph": graph is not None})
    out = {
        "metric": METRIC,
        "value": wl.batch / (ms_per_step * 1e-3),
        "unit": "images/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": cfg,
        "roofline": roof,
        "step_api_bytes": run.api_bytes,
        "step_effective_gbps": run.api_bytes / (ms_per_step * 1e-3) / 1e9,
        "step_kernel_ms": {k: round(v[0], 5) for k, v in sorted(per_name.items(), key=lambda kv: -kv[1][0])},
        "step_ms_dist": dist,
        "wall_ms_per_step": wall_ms,
        "eager_ms_per_step": eager_ms_per_step,
    }
    if args.copy_calibration > 0:
        n = args.copy_calibration * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        out["copy_calibration_bytes"] = 2 * 4 * n
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = run.cpu_baseline()
    print(json.dumps(out), flush=True)


def ctypes_buf(n):
    import ctypes
    return ctypes.create_string_buffer(n)


if __name__ == "__main__":
    main()
