"""fdc_head_forward_noalloc (the head forward with the library's static scratch array
instead of a caller workspace) against fdc_head_forward on the same inputs: two calls
in a row, the second with a smaller input, each bit for bit equal to the workspace
form (both run the same kernels in the same order)."""

import ctypes
import zlib

import numpy as np
import pytest
import torch

from paper_2106_12736_amd._lib import FDC_EUNSUPPORTED, call, status

pytestmark = pytest.mark.gpu


def _p(t):
    return ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _inputs(B, F, classes):
    rng = np.random.default_rng(zlib.crc32(repr(("noalloc", B, F, classes)).encode()))
    y = rng.standard_normal((B, F)).astype(np.float32)
    W = (rng.standard_normal((classes, F)) / np.sqrt(F)).astype(np.float32)
    bias = rng.standard_normal(classes).astype(np.float32)
    labels = rng.integers(0, classes, B).astype(np.int32)
    return [torch.from_numpy(a).cuda() for a in (y, W, bias, labels)]


def _both(B, F, classes):
    print(f"no-alloc head B={B} F={F} classes={classes}", flush=True)
    y, W, bias, labels = _inputs(B, F, classes)
    out = []
    for noalloc in (True, False):
        logits = torch.full((B, classes), float("nan"), dtype=torch.float32, device="cuda")
        loss = torch.full((1,), float("nan"), dtype=torch.float32, device="cuda")
        if noalloc:
            call("fdc_head_forward_noalloc", _p(y), _p(W), _p(bias), _p(labels), _p(logits), _p(loss), B, F,
                 classes, _stream())
        else:
            n = ctypes.c_size_t()
            call("fdc_head_workspace_size", B, F, classes, ctypes.byref(n))
            ws = torch.empty(n.value, dtype=torch.uint8, device="cuda")
            call("fdc_head_forward", _p(y), _p(W), _p(bias), _p(labels), _p(logits), _p(loss), B, F, classes,
                 _p(ws), ws.numel(), _stream())
        torch.cuda.synchronize()
        out.append((logits.cpu().numpy(), loss.cpu().numpy()))
    return out


def test_noalloc_head_forward_equals_workspace_form():
    # a large call, then a smaller one: the second must not see the first's partial logits
    for B, F, classes in ((16, 200000, 16), (3, 5000, 5)):
        (lg_a, ls_a), (lg_b, ls_b) = _both(B, F, classes)
        assert np.all(np.isfinite(lg_a)) and np.isfinite(ls_a[0])
        assert np.array_equal(lg_a, lg_b), np.abs(lg_a - lg_b).max()
        assert np.array_equal(ls_a, ls_b)


def test_noalloc_head_forward_refuses_oversize():
    y, W, bias, labels = _inputs(2, 8, 2)
    # ceil(F / 1024) * B * classes = 64 * 2 * 16 * 64 > 2^18 partial logits
    st = status("fdc_head_forward_noalloc", _p(y), _p(W), _p(bias), _p(labels), _p(y), _p(y), 64, 1 << 21, 16,
                _stream())
    assert st == FDC_EUNSUPPORTED
