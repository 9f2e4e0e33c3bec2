"""GPU parity of the FDCNN data flow of section 2.5.1 (one rfft2, every FDC + FDP layer
on spectra, one irfft2) against the float64 oracle: the fused spectral CIC + FDP op on
its own, and the whole chain forward and backward on every CIC workload at full size."""

import ctypes
import zlib

import numpy as np
import pytest
import torch

from _parity import assert_parity, to_np
from oracle import dft, fdc
from paper_2106_12736_amd import inputs, layers
from paper_2106_12736_amd._lib import call

pytestmark = pytest.mark.gpu


def _rng(*key):
    return np.random.default_rng(zlib.crc32(repr(key).encode()))


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _p(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _c64(rng, shape):
    return (rng.standard_normal(shape) + 1j * rng.standard_normal(shape)).astype(np.complex64)


@pytest.mark.parametrize("B,C,S,N,M", [
    (1, 1, 1, 4, 2), (2, 1, 4, 8, 4), (3, 2, 6, 16, 16), (2, 4, 4, 32, 8), (1, 3, 9, 64, 32), (2, 2, 4, 224, 112),
    # batches past one group of in-flight images, with a ragged rest; odd row lengths
    (11, 2, 4, 16, 8), (9, 1, 8, 32, 16), (17, 3, 3, 8, 8),
])
def test_cic_fdp_op(B, C, S, N, M):
    rng = _rng("cic_fdp", B, C, S, N, M)
    X = _c64(rng, (B, C, N, N // 2 + 1))
    K = _c64(rng, (S, N, N // 2 + 1))
    gY = _c64(rng, (B, S, M, M // 2 + 1))
    Xd, Kd = torch.from_numpy(X).cuda(), torch.from_numpy(K).cuda()
    Y = layers.cic_fdp_forward(Xd, Kd, M)
    gX, gK = layers.cic_fdp_backward(torch.from_numpy(gY).cuda(), Xd, Kd)
    torch.cuda.synchronize()
    X64, K64, g64 = X.astype(np.complex128), K.astype(np.complex128), gY.astype(np.complex128)
    assert_parity(to_np(Y), fdc.fdp(fdc.cic(X64, K64), M, M), "Y")
    gz = fdc.fdp_backward(g64, N, N)
    gx_ref, gk_ref = fdc.cic_backward(gz, X64, K64)
    assert_parity(to_np(gX), gx_ref, "gX")
    assert_parity(to_np(gK), gk_ref, "gK")
    assert np.all(to_np(gK)[np.abs(gk_ref) == 0] == 0), "dropped bins must be exact zeros"


@pytest.mark.parametrize("B,C,S,N,M", [
    (1, 1, 1, 4, 2), (2, 1, 4, 8, 4), (3, 2, 6, 16, 16), (2, 4, 4, 32, 8), (1, 3, 9, 64, 32), (2, 2, 4, 224, 112),
    (11, 2, 4, 16, 8), (9, 1, 8, 32, 16), (17, 3, 3, 8, 8), (8, 1, 8, 1024, 512),
])
def test_cic_fdp_projected_op(B, C, S, N, M):
    """The projected forms equal the plain calls followed by Pi_H, bit for bit (same
    arithmetic), and the oracle's Pi_H of the oracle's layer; columns 0 and N/2 of dX
    include the unpooled case (M = N, both columns kept)."""
    print(f"cic_fdp projected B={B} C={C} S={S} N={N} M={M}", flush=True)
    rng = _rng("cic_fdp_proj", B, C, S, N, M)
    X = _c64(rng, (B, C, N, N // 2 + 1))
    K = _c64(rng, (S, N, N // 2 + 1))
    gY = _c64(rng, (B, S, M, M // 2 + 1))
    Xd, Kd, gYd = (torch.from_numpy(a).cuda() for a in (X, K, gY))
    Y = layers.cic_fdp_forward(Xd, Kd, M)
    Yp = layers.cic_fdp_forward(Xd, Kd, M, project=True)
    gX, gK = layers.cic_fdp_backward(gYd, Xd, Kd)
    gXp, gKp = layers.cic_fdp_backward(gYd, Xd, Kd, project=True)
    layers.hermitian_project(Y)
    layers.hermitian_project(gX)
    torch.cuda.synchronize()
    assert torch.equal(Yp, Y) and torch.equal(gXp, gX) and torch.equal(gKp, gK)
    X64, K64, g64 = X.astype(np.complex128), K.astype(np.complex128), gY.astype(np.complex128)
    assert_parity(to_np(Yp), dft.hermitian_projection(fdc.fdp(fdc.cic(X64, K64), M, M)), "Pi_H Y")
    gx_ref, _ = fdc.cic_backward(fdc.fdp_backward(g64, N, N), X64, K64)
    assert_parity(to_np(gXp), dft.hermitian_projection(gx_ref), "Pi_H gX")


@pytest.mark.parametrize("B,C,S,N,M", [
    (1, 1, 1, 4, 2), (2, 1, 4, 8, 4), (3, 2, 6, 16, 16), (2, 4, 4, 32, 8), (1, 3, 9, 64, 32), (2, 2, 4, 224, 112),
    (11, 2, 4, 16, 8), (9, 1, 8, 32, 16), (8, 1, 8, 1024, 512), (8, 8, 16, 512, 256),
])
@pytest.mark.parametrize("project", [False, True])
def test_cic_fdp_backward_kept(B, C, S, N, M, project):
    """The kept-bins forms on zeroed gX and gK equal the full calls, bit for bit at every
    bin (the projected form also over columns 0 and N/2 of the dropped rows), and leave
    every dropped bin of gK and every dropped bin of gX outside those columns untouched."""
    print(f"cic_fdp kept B={B} C={C} S={S} N={N} M={M} project={project}", flush=True)
    rng = _rng("cic_fdp_kept", B, C, S, N, M)
    X = _c64(rng, (B, C, N, N // 2 + 1))
    K = _c64(rng, (S, N, N // 2 + 1))
    gY = _c64(rng, (B, S, M, M // 2 + 1))
    Xd, Kd, gYd = (torch.from_numpy(a).cuda() for a in (X, K, gY))
    gX, gK = layers.cic_fdp_backward(gYd, Xd, Kd, project=project)
    gX0, gK0 = torch.zeros_like(Xd), torch.zeros_like(Kd)
    fn = "fdc_cic_fdp_backward_projected_kept" if project else "fdc_cic_fdp_backward_kept"
    call(fn, _p(gYd), _p(Xd), _p(Kd), _p(gX0), _p(gK0), B, C, S, N, M, _stream())
    # a sentinel in every dropped bin: the kept forms must not write there
    nan = float("nan")
    kept = np.zeros((N, N // 2 + 1), bool)
    kept[np.r_[0:M // 2, N - M // 2:N], :M // 2 + 1] = True
    gxw = kept.copy()
    if project:
        gxw[:, 0] = gxw[:, N // 2] = True
    gXs, gKs = torch.zeros_like(Xd), torch.zeros_like(Kd)
    gXs[..., torch.from_numpy(~gxw)] = complex(nan, nan)
    gKs[..., torch.from_numpy(~kept)] = complex(nan, nan)
    call(fn, _p(gYd), _p(Xd), _p(Kd), _p(gXs), _p(gKs), B, C, S, N, M, _stream())
    # dK alone (gX NULL): the output channels of an input channel may then run in
    # separate threads
    gKn = torch.full_like(Kd, complex(nan, nan))
    gKn[..., torch.from_numpy(kept)] = 0
    call(fn, _p(gYd), _p(Xd), _p(Kd), None, _p(gKn), B, C, S, N, M, _stream())
    torch.cuda.synchronize()
    assert torch.equal(gKn[..., torch.from_numpy(kept)], gK[..., torch.from_numpy(kept)])
    assert np.all(np.isnan(to_np(gKn)[..., ~kept]))
    assert torch.equal(gX0, gX) and torch.equal(gK0, gK)
    assert np.all(np.isnan(to_np(gXs)[..., ~gxw])) and np.all(np.isnan(to_np(gKs)[..., ~kept]))
    assert torch.equal(gXs[..., torch.from_numpy(gxw)], gX[..., torch.from_numpy(gxw)])
    assert torch.equal(gKs[..., torch.from_numpy(kept)], gK[..., torch.from_numpy(kept)])


@pytest.mark.parametrize("wl", inputs.CIC_WORKLOADS, ids=lambda w: w.name)
def test_chain_forward_backward(wl):
    print(f"chain {wl.name}", flush=True)
    d = inputs.make_cic_stack(wl)
    x = torch.from_numpy(d.x).cuda()
    Ks = [torch.from_numpy(k).cuda() for k in d.kernels]
    ch = layers.CicChain(wl.batch, wl.sizes, wl.channels)
    gin = torch.empty_like(x)
    ch.forward(x, Ks)
    ch.backward(torch.from_numpy(d.grad).cuda(), Ks, input_grad=gin)
    torch.cuda.synchronize()
    kd = [k.astype(np.complex128) for k in d.kernels]
    y_ref, saved = fdc.cic_chain_forward(d.x.astype(np.float64), kd, wl.sizes)
    gks_ref, gx_ref = fdc.cic_chain_backward(d.grad.astype(np.float64), saved, kd, wl.sizes, want_input_grad=True)
    assert_parity(to_np(ch.out), y_ref, "y")
    for i in range(wl.layers):
        assert_parity(to_np(ch.gks[i]), gks_ref[i], f"dK[{i}]")
    assert_parity(to_np(gin), gx_ref, "gx")


@pytest.mark.parametrize("wl", inputs.CIC_WORKLOADS, ids=lambda w: w.name)
def test_chain_with_projection_is_the_stack(wl):
    """The chain with Pi_H after every layer but the last computes the per-layer stack
    (rfft2 -> CIC -> FDP -> irfft2 for every layer): against the oracle's layer-by-layer
    stack, and against the GPU's stack executor on the same inputs."""
    print(f"chain + Pi_H {wl.name}", flush=True)
    d = inputs.make_cic_stack(wl)
    x = torch.from_numpy(d.x).cuda()
    Ks = [torch.from_numpy(k).cuda() for k in d.kernels]
    g = torch.from_numpy(d.grad).cuda()
    ch = layers.CicChain(wl.batch, wl.sizes, wl.channels, hermitian=True)
    gin = torch.empty_like(x)
    ch.forward(x, Ks)
    ch.backward(g, Ks, input_grad=gin)
    st = layers.CicStackFused(wl.batch, wl.sizes, wl.channels)
    gin_st = torch.empty_like(x)
    st.forward(x, Ks)
    st.backward(g, Ks, input_grad=gin_st)
    torch.cuda.synchronize()
    kd = [k.astype(np.complex128) for k in d.kernels]
    y_ref, saved = fdc.cic_stack_forward(d.x.astype(np.float64), kd, wl.sizes)
    gks_ref, gx_ref = fdc.cic_stack_backward(d.grad.astype(np.float64), saved, kd, wl.sizes, want_input_grad=True)
    assert_parity(to_np(ch.out), y_ref, "y")
    assert_parity(to_np(st.out), y_ref, "y (stack executor)")
    for i in range(wl.layers):
        assert_parity(to_np(ch.gks[i]), gks_ref[i], f"dK[{i}]")
        assert_parity(to_np(st.gks[i]), gks_ref[i], f"dK[{i}] (stack executor)")
    assert_parity(to_np(gin), gx_ref, "gx")
    assert_parity(to_np(gin_st), gx_ref, "gx (stack executor)")


def test_chain_graph_replays():
    wl = inputs.STACK512
    d = inputs.make_cic_stack(wl)
    x = torch.from_numpy(d.x).cuda()
    Ks = [torch.from_numpy(k).cuda() for k in d.kernels]
    g = torch.from_numpy(d.grad).cuda()
    ch = layers.CicChain(wl.batch, wl.sizes, wl.channels)

    def step():
        ch.forward(x, Ks)
        ch.backward(g, Ks)

    step()
    torch.cuda.synchronize()
    ref = [ch.out.clone()] + [k.clone() for k in ch.gks]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for rep in range(3):
        torch.randn(1 << 20, device="cuda").mul_(2.0).sum().item()
        for t in [ch.out] + ch.gks:
            t.zero_()
        graph.replay()
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(ref, [ch.out] + ch.gks)):
            assert torch.equal(a, b), f"replay {rep}: output {i}"
