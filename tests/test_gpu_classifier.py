"""GPU parity of the FDCNN classifier (section 2.5.1, Fig. 3; section 3.1's loss and
optimiser) against the float64 oracle: the head (ReLU, fully connected layer, softmax
cross-entropy, forward and backward), the Adam step, and a whole training step of the
spectral chain with the head."""

import ctypes
import zlib

import numpy as np
import pytest
import torch

from _parity import assert_parity, to_np
from oracle import classifier, fdc
from paper_2106_12736_amd import inputs, layers
from paper_2106_12736_amd._lib import call

pytestmark = pytest.mark.gpu


def _rng(*key):
    return np.random.default_rng(zlib.crc32(repr(key).encode()))


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _p(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


@pytest.mark.parametrize("B,F,classes", [
    (1, 1, 1), (3, 7, 2), (2, 4096, 5), (4, 5000, 2), (8, 131072, 2), (5, 9000, 16),
])
def test_head_forward_backward(B, F, classes):
    print(f"head B={B} F={F} classes={classes}", flush=True)
    rng = _rng("head", B, F, classes)
    y = rng.standard_normal((B, F)).astype(np.float32)
    W = (rng.standard_normal((classes, F)) / np.sqrt(F)).astype(np.float32)
    bias = rng.standard_normal(classes).astype(np.float32)
    labels = rng.integers(0, classes, B).astype(np.int32)
    yd, Wd, bd, ld = (torch.from_numpy(a).cuda() for a in (y, W, bias, labels))
    logits = torch.empty((B, classes), dtype=torch.float32, device="cuda")
    loss = torch.empty(1, dtype=torch.float32, device="cuda")
    n = ctypes.c_size_t()
    call("fdc_head_workspace_size", B, F, classes, ctypes.byref(n))
    ws = torch.empty(n.value, dtype=torch.uint8, device="cuda")
    call("fdc_head_forward", _p(yd), _p(Wd), _p(bd), _p(ld), _p(logits), _p(loss), B, F, classes, _p(ws),
         ws.numel(), _stream())
    gy, gW = torch.empty_like(yd), torch.empty_like(Wd)
    gb = torch.empty_like(bd)
    call("fdc_head_backward", _p(yd), _p(Wd), _p(logits), _p(ld), _p(gy), _p(gW), _p(gb), B, F, classes,
         _stream())
    torch.cuda.synchronize()
    ref_logits, ref_loss = classifier.head_forward(y.astype(np.float64), W, bias, labels)
    assert_parity(to_np(logits), ref_logits, "logits")
    assert abs(to_np(loss)[0] - ref_loss) <= 1e-5 * max(1.0, abs(ref_loss)), (to_np(loss)[0], ref_loss)
    # the backward works from the GPU's logits, so both sides take the same softmax
    rgy, rgW, rgb = classifier.head_backward(y.astype(np.float64), W, to_np(logits).astype(np.float64), labels)
    assert_parity(to_np(gy), rgy, "gy")
    assert_parity(to_np(gW), rgW, "gW")
    assert_parity(to_np(gb), rgb, "gbias")
    assert np.all(to_np(gy)[y <= 0] == 0), "the ReLU blocks the gradient where y <= 0"


@pytest.mark.parametrize("B,F,classes", [(3, 7, 5), (5, 9000, 16), (16, 4096, 16), (8, 131072, 2)])
def test_head_backward_from_oracle_logits(B, F, classes):
    """The head backward on its own: the GPU takes the oracle's logits (rounded to fp32),
    so its gradients are checked against the oracle independently of the GPU forward."""
    print(f"head backward B={B} F={F} classes={classes}", flush=True)
    rng = _rng("head-bwd", B, F, classes)
    y = rng.standard_normal((B, F)).astype(np.float32)
    W = (rng.standard_normal((classes, F)) / np.sqrt(F)).astype(np.float32)
    bias = rng.standard_normal(classes).astype(np.float32)
    labels = rng.integers(0, classes, B).astype(np.int32)
    ref_logits, _ = classifier.head_forward(y.astype(np.float64), W, bias, labels)
    logits32 = ref_logits.astype(np.float32)
    yd, Wd, ld, lg = (torch.from_numpy(a).cuda() for a in (y, W, labels, logits32))
    gy, gW = torch.empty_like(yd), torch.empty_like(Wd)
    gb = torch.empty(classes, dtype=torch.float32, device="cuda")
    call("fdc_head_backward", _p(yd), _p(Wd), _p(lg), _p(ld), _p(gy), _p(gW), _p(gb), B, F, classes, _stream())
    torch.cuda.synchronize()
    rgy, rgW, rgb = classifier.head_backward(y.astype(np.float64), W, logits32.astype(np.float64), labels)
    assert_parity(to_np(gy), rgy, "gy")
    assert_parity(to_np(gW), rgW, "gW")
    assert_parity(to_np(gb), rgb, "gbias")


@pytest.mark.parametrize("n", [1, 1000, 262147, (1 << 24) + 5])
def test_adam_step(n):
    print(f"adam n={n}", flush=True)
    rng = _rng("adam", n)
    p = rng.standard_normal(n).astype(np.float32)
    g = rng.standard_normal(n).astype(np.float32)
    m = (0.1 * rng.standard_normal(n)).astype(np.float32)
    v = (0.01 * rng.random(n)).astype(np.float32)
    lr, b1, b2, eps, wd = 1e-2, 0.9, 0.999, 1e-8, 1e-3
    pd, gd, md, vd = (torch.from_numpy(a.copy()).cuda() for a in (p, g, m, v))
    count = torch.tensor([3], dtype=torch.int32, device="cuda")
    call("fdc_adam_step", _p(pd), _p(gd), _p(md), _p(vd), n, _p(count), lr, b1, b2, eps, wd, _stream())
    torch.cuda.synchronize()
    rp, rm, rv = classifier.adam_step(p, g, m, v, 4, lr, b1, b2, eps, wd)
    assert int(count.item()) == 4
    assert_parity(to_np(md), rm, "m")
    assert_parity(to_np(vd), rv, "v")
    # the update itself (p1 - p0), so that the check is not swamped by p0
    assert_parity(to_np(pd).astype(np.float64) - p, rp - p, "update")


def _classifier_setup(wl, classes=2, lr=1e-5):
    d = inputs.make_cic_stack(wl)
    rng = _rng("classifier", wl.name)
    clf = layers.FdcnnClassifier(wl.batch, wl.sizes, wl.channels, classes=classes, lr=lr)
    F = clf.features
    W = (rng.standard_normal((classes, F)) * np.sqrt(2.0 / F)).astype(np.float32)
    bias = np.zeros(classes, np.float32)
    labels = (np.arange(wl.batch) % classes).astype(np.int32)
    clf.load([torch.from_numpy(k).cuda() for k in d.kernels], torch.from_numpy(W).cuda(),
             torch.from_numpy(bias).cuda())
    return d, clf, W, bias, labels


# Chain outputs within this fraction of the largest |output| of zero: the ReLU's
# decision there is within the fp32 error of the chain (rel-L2 about 1e-7 at 1024^2).
RELU_AMBIGUOUS = 1e-5


def _reference_gradients(d, kd, W, bias, labels, wl, out_gpu):
    """classifier.classifier_gradients, with the ReLU decision (y > 0, a per-element
    choice) taken from the GPU's fp32 chain output where the float64 output is within
    the fp32 error of zero, and checked against the float64 decision everywhere else."""
    y, saved = fdc.cic_chain_forward(d.x.astype(np.float64), kd, wl.sizes)
    amb = np.abs(y) <= RELU_AMBIGUOUS * np.abs(y).max()
    assert amb.sum() <= 1e-3 * amb.size, int(amb.sum())
    assert np.array_equal((out_gpu > 0)[~amb], (y > 0)[~amb]), "ReLU decisions differ away from zero"
    y_dec = np.where(amb, out_gpu.astype(np.float64), y)  # same decisions as the GPU, |change| <= the threshold
    B = y.shape[0]
    logits, loss = classifier.head_forward(y_dec.reshape(B, -1), W.astype(np.float64), bias.astype(np.float64),
                                           labels)
    gy, gW, gbias = classifier.head_backward(y_dec.reshape(B, -1), W.astype(np.float64), logits, labels)
    gks, _ = fdc.cic_chain_backward(gy.reshape(y.shape), saved, kd, wl.sizes)
    return loss, logits, gks, gW, gbias


@pytest.mark.parametrize("wl", inputs.CIC_WORKLOADS, ids=lambda w: w.name)
def test_classifier_step(wl):
    """One training step at full size on every CIC workload (cic_stack_1024 is the one
    bench.py --classifier times): loss, logits, every gradient, and the Adam update."""
    print(f"classifier {wl.name}", flush=True)
    d, clf, W, bias, labels = _classifier_setup(wl, lr=1e-2)
    x = torch.from_numpy(d.x).cuda()
    ld = torch.from_numpy(labels).cuda()
    p0 = to_np(clf.params).astype(np.float64)
    clf.forward(x, ld)
    clf.backward(ld)
    torch.cuda.synchronize()
    grads = to_np(clf.grads).copy()
    logits, loss = to_np(clf.logits), to_np(clf.loss)[0]
    gks = [to_np(t) for t in clf.chain.gks]
    gW, gb = to_np(clf.gW), to_np(clf.gbias)
    clf.optimizer_step()
    torch.cuda.synchronize()

    kd = [k.astype(np.complex128) for k in d.kernels]
    r_loss, r_logits, r_gks, r_gW, r_gb = _reference_gradients(d, kd, W, bias, labels, wl, to_np(clf.chain.out))
    assert_parity(logits, r_logits, "logits")
    assert abs(loss - r_loss) <= 1e-5 * max(1.0, abs(r_loss)), (loss, r_loss)
    for i, (g, r) in enumerate(zip(gks, r_gks)):
        assert_parity(g, r, f"dK[{i}]")
    assert_parity(gW, r_gW, "dW")
    assert_parity(gb, r_gb, "dbias", max_abs_frac=1e-3)
    # Adam on the GPU's own gradients: the update against the oracle's on the same inputs
    rp, rm, rv = classifier.adam_step(p0, grads, 0.0 * p0, 0.0 * p0, 1, clf.lr, *clf.betas, clf.eps,
                                      clf.weight_decay)
    assert int(clf.step_count.item()) == 1
    assert_parity(to_np(clf.params).astype(np.float64) - p0, rp - p0, "update")
    assert_parity(to_np(clf.m), rm, "m")
    assert_parity(to_np(clf.v), rv, "v")


def test_classifier_steps_repeat_exactly():
    """Three training steps, the state restored, the same three again: bit-identical
    (every sum runs in a fixed order), and the loss moves."""
    wl = inputs.LAYER64
    d, clf, W, bias, labels = _classifier_setup(wl, lr=1e-3)
    x = torch.from_numpy(d.x).cuda()
    ld = torch.from_numpy(labels).cuda()
    st = clf.state()
    losses = []
    for _ in range(3):
        losses.append(float(clf.train_step(x, ld).item()))
    first = [t.clone() for t in (clf.params, clf.m, clf.v)]
    clf.set_state(st)
    for i in range(3):
        assert float(clf.train_step(x, ld).item()) == losses[i]
    for a, b in zip(first, (clf.params, clf.m, clf.v)):
        assert torch.equal(a, b)
    assert int(clf.step_count.item()) == 3
    assert losses[2] != losses[0]
