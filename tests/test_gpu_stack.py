"""GPU tests of the fused stack executor (fdc_cic_stack_*).  It runs the same
kernels on the same rows as the layer-by-layer calls, with the activations between
layers kept in registers; the compiler may contract multiply-adds differently inside
the fused boundary kernel, so the two agree to fp32 rounding (not bit for bit).  Every
CIC workload runs at full size, including the input-image gradient: against the
layer-by-layer path at a tight tolerance and against the oracle at the parity bar;
the fused step also replays identically as a HIP graph."""

import numpy as np
import pytest
import torch

from _parity import assert_parity, to_np
from oracle import fdc
from paper_2106_12736_amd import inputs, layers

pytestmark = pytest.mark.gpu


def _run_both(wl):
    d = inputs.make_cic_stack(wl)
    x = torch.from_numpy(d.x).cuda()
    Ks = [torch.from_numpy(k).cuda() for k in d.kernels]
    g = torch.from_numpy(d.grad).cuda()
    ref = layers.CicStack(wl.batch, wl.sizes, wl.channels)
    gin_ref = torch.empty_like(x)
    ref.forward(x, Ks)
    ref.backward(g, Ks, input_grad=gin_ref)
    fused = layers.CicStackFused(wl.batch, wl.sizes, wl.channels)
    gin = torch.empty_like(x)
    fused.forward(x, Ks)
    fused.backward(g, Ks, input_grad=gin)
    torch.cuda.synchronize()
    return d, ref, gin_ref, fused, gin


def _close(got, ref, name, rel=1e-6):
    d = (got - ref).abs()
    r = (d.norm() / ref.norm()).item()
    print(f"  {name}: max |d| {d.max().item():.3e}, rel-L2 {r:.3e}", flush=True)
    assert r <= rel, f"{name}: rel-L2 {r:.3e} against the layer-by-layer path"


@pytest.mark.parametrize("wl", inputs.CIC_WORKLOADS, ids=lambda w: w.name)
def test_fused_stack_matches_layer_calls_and_oracle(wl):
    print(f"fused stack {wl.name}", flush=True)
    d, ref, gin_ref, fused, gin = _run_both(wl)
    _close(fused.out, ref.acts[-1], "y")
    for i in range(wl.layers):
        _close(fused.saved[i], ref.saved[i], f"saved[{i}]")
        _close(fused.gks[i], ref.gks[i], f"dK[{i}]")
    _close(gin, gin_ref, "gx")
    x64 = d.x.astype(np.float64)
    kd = [k.astype(np.complex128) for k in d.kernels]
    y_ref, saved = fdc.cic_stack_forward(x64, kd, wl.sizes)
    gks_ref, gx_ref = fdc.cic_stack_backward(d.grad.astype(np.float64), saved, kd, wl.sizes, want_input_grad=True)
    assert_parity(to_np(fused.out), y_ref, "y")
    for i in range(wl.layers):
        assert_parity(to_np(fused.gks[i]), gks_ref[i], f"dK[{i}]")
    assert_parity(to_np(gin), gx_ref, "gx")


def test_fused_stack_graph_replays():
    wl = inputs.STACK512
    d = inputs.make_cic_stack(wl)
    x = torch.from_numpy(d.x).cuda()
    Ks = [torch.from_numpy(k).cuda() for k in d.kernels]
    g = torch.from_numpy(d.grad).cuda()
    st = layers.CicStackFused(wl.batch, wl.sizes, wl.channels)

    def step():
        st.forward(x, Ks)
        st.backward(g, Ks)

    step()
    torch.cuda.synchronize()
    ref = [st.out.clone()] + [k.clone() for k in st.gks]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for rep in range(3):
        torch.randn(1 << 20, device="cuda").mul_(2.0).sum().item()
        for t in [st.out] + st.gks:
            t.zero_()
        graph.replay()
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(ref, [st.out] + st.gks)):
            assert torch.equal(a, b), f"replay {rep}: output {i}"


def _fused(wl, x, Ks, g, input_grad, tail_env=None):
    import os
    old = os.environ.get("FDC_STACK_TAIL")
    if tail_env is not None:
        os.environ["FDC_STACK_TAIL"] = tail_env
    try:
        st = layers.CicStackFused(wl.batch, wl.sizes, wl.channels)
    finally:
        if tail_env is not None:
            if old is None:
                del os.environ["FDC_STACK_TAIL"]
            else:
                os.environ["FDC_STACK_TAIL"] = old
    gin = torch.empty_like(x) if input_grad else None
    st.forward(x, Ks)
    st.backward(g, Ks, input_grad=gin)
    torch.cuda.synchronize()
    return st, gin


@pytest.mark.parametrize("wl", inputs.CIC_WORKLOADS[1:], ids=lambda w: w.name)
def test_stack_tail_matches_per_layer_kernels(wl):
    """The LDS-resident tail (the last two layers in one launch each way) against the
    same stack with every layer on the per-layer kernels."""
    print(f"stack tail {wl.name}", flush=True)
    d = inputs.make_cic_stack(wl)
    x = torch.from_numpy(d.x).cuda()
    Ks = [torch.from_numpy(k).cuda() for k in d.kernels]
    g = torch.from_numpy(d.grad).cuda()
    on, gin_on = _fused(wl, x, Ks, g, True)
    off, gin_off = _fused(wl, x, Ks, g, True, tail_env="0")
    assert on.tail() == wl.layers - 2 and off.tail() == -1
    _close(on.out, off.out, "y")
    for i in range(wl.layers):
        _close(on.saved[i], off.saved[i], f"saved[{i}]")
        _close(on.gks[i], off.gks[i], f"dK[{i}]")
    _close(gin_on, gin_off, "gx")
    # exact zeros at the bins FDP drops
    for i in range(wl.layers):
        N, M = wl.sizes[i], wl.sizes[i + 1]
        gk = to_np(on.gks[i])
        assert np.all(gk[:, M // 2:N - M // 2, :] == 0) and np.all(gk[:, :, M // 2 + 1:] == 0)


@pytest.mark.parametrize("input_grad", [True, False])
def test_stack_that_is_only_a_tail(input_grad):
    """A two-layer stack 128 -> 64 -> 32 is all tail: the forward starts from the input
    images and the backward ends in the input gradient (or in nothing)."""
    wl = inputs.CicStack("tail_only_128", 77, 3, (128, 64, 32), (2, 4, 8), "disc")
    print(f"tail-only stack, input grad {input_grad}", flush=True)
    d = inputs.make_cic_stack(wl)
    x = torch.from_numpy(d.x).cuda()
    Ks = [torch.from_numpy(k).cuda() for k in d.kernels]
    g = torch.from_numpy(d.grad).cuda()
    st, gin = _fused(wl, x, Ks, g, input_grad)
    assert st.tail() == 0
    x64 = d.x.astype(np.float64)
    kd = [k.astype(np.complex128) for k in d.kernels]
    y_ref, saved = fdc.cic_stack_forward(x64, kd, wl.sizes)
    gks_ref, gx_ref = fdc.cic_stack_backward(d.grad.astype(np.float64), saved, kd, wl.sizes,
                                             want_input_grad=input_grad)
    assert_parity(to_np(st.out), y_ref, "y")
    for i in range(wl.layers):
        assert_parity(to_np(st.gks[i]), gks_ref[i], f"dK[{i}]")
    if input_grad:
        assert_parity(to_np(gin), gx_ref, "gx")


def _stack_backward(fn, st, g, Ks, gks, gin):
    from paper_2106_12736_amd._lib import call
    from paper_2106_12736_amd.layers import _ptr, _ptr_array, _stream
    call(fn, st._p, _ptr(g), st._saved_arr, _ptr_array(Ks), _ptr(gin), _ptr_array(gks), _ptr(st.bwd_ws),
         st.bwd_ws.numel(), _stream())
    torch.cuda.synchronize()


_TAIL_ONLY = inputs.CicStack("tail_only_128", 77, 3, (128, 64, 32), (2, 4, 8), "disc")


@pytest.mark.parametrize("input_grad", [True, False])
@pytest.mark.parametrize("wl", list(inputs.CIC_WORKLOADS) + [_TAIL_ONLY], ids=lambda w: w.name)
def test_stack_backward_kept_matches_full(wl, input_grad):
    """fdc_cic_stack_backward_kept writes the kept bins of every gK only: on buffers
    that hold zeros elsewhere it equals fdc_cic_stack_backward bit for bit (dK of every
    layer path: one batch range, ranges summed by a second launch, dK and dX merged, the
    tail's sums), and NaN planted at the dropped bins stays there."""
    print(f"stack backward kept {wl.name}, input grad {input_grad}", flush=True)
    d = inputs.make_cic_stack(wl)
    x = torch.from_numpy(d.x).cuda()
    Ks = [torch.from_numpy(k).cuda() for k in d.kernels]
    g = torch.from_numpy(d.grad).cuda()
    st = layers.CicStackFused(wl.batch, wl.sizes, wl.channels)
    st.forward(x, Ks)
    shapes = [(wl.channels[i + 1], wl.sizes[i], wl.sizes[i] // 2 + 1) for i in range(wl.layers)]
    nan = complex(float("nan"), float("nan"))

    def bufs(fill):
        return [torch.full(s, fill, dtype=torch.complex64, device="cuda") for s in shapes]

    gin_full = torch.full_like(x, float("nan")) if input_grad else None
    gin_kept = torch.full_like(x, float("nan")) if input_grad else None
    full, kept0, kept_nan = bufs(nan), bufs(0), bufs(nan)
    _stack_backward("fdc_cic_stack_backward", st, g, Ks, full, gin_full)
    _stack_backward("fdc_cic_stack_backward_kept", st, g, Ks, kept0, gin_kept)
    _stack_backward("fdc_cic_stack_backward_kept", st, g, Ks, kept_nan, None)
    for i in range(wl.layers):
        N, M = wl.sizes[i], wl.sizes[i + 1]
        assert not torch.isnan(full[i]).any(), f"dK[{i}]: full form left a bin unwritten"
        assert torch.equal(kept0[i], full[i]), f"dK[{i}]: kept form differs from the full form"
        kn = kept_nan[i]
        keep = torch.zeros(shapes[i], dtype=torch.bool, device="cuda")
        keep[:, :M // 2, :M // 2 + 1] = True
        keep[:, N - M // 2:, :M // 2 + 1] = True
        assert torch.equal(kn[keep], full[i][keep]), f"dK[{i}]: kept bins"
        assert torch.isnan(kn[~keep]).all(), f"dK[{i}]: a dropped bin was written"
    if input_grad:
        assert torch.equal(gin_kept, gin_full), "gx differs"
