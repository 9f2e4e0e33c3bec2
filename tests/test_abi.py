"""Host-side tests of the C ABI: the library loads, exports every declared symbol,
and rejects bad arguments with the documented status before touching the GPU.

None of these calls enqueues work: each returns from host-side validation.
"""

import ctypes

import pytest

from paper_2106_12736_amd import _lib, layers
from paper_2106_12736_amd._lib import FDC_EHIP, FDC_EINVAL, FDC_EUNSUPPORTED, FDC_EWORKSPACE, FDC_OK


def test_library_exports_every_declared_function():
    declared = _lib.header_functions()
    assert len(declared) >= 25
    lib = _lib.lib()
    missing = [n for n in declared if not hasattr(lib, n)]
    assert not missing, missing
    assert set(_lib._SIGS) == set(declared), "binding signatures out of sync with include/fdc.h"


def test_status_strings_and_version():
    lib = _lib.lib()
    for st in range(5):
        assert lib.fdc_status_string(st)
    assert lib.fdc_version() >= 100


def _fft_plan(count, h, w):
    p = ctypes.c_void_p()
    st = _lib.status("fdc_fft_plan_create", ctypes.byref(p), count, h, w)
    return st, p


@pytest.mark.parametrize("count,h,w,expect", [
    (1, 8, 8, FDC_OK), (3, 224, 224, FDC_OK), (2, 1024, 16, FDC_OK),
    (0, 8, 8, FDC_EINVAL), (1, 7, 8, FDC_EINVAL), (1, 8, -4, FDC_EINVAL),
    (1, 2048, 8, FDC_EUNSUPPORTED), (1, 96, 96, FDC_EUNSUPPORTED), (1, 22, 8, FDC_EUNSUPPORTED),
])
def test_fft_plan_validation(count, h, w, expect):
    st, p = _fft_plan(count, h, w)
    assert st == expect, _lib.last_error()
    if st == FDC_OK:
        n = ctypes.c_size_t()
        assert _lib.status("fdc_fft_workspace_size", p, ctypes.byref(n)) == FDC_OK
        assert n.value == count * h * (w // 2 + 1) * 8
        assert _lib.status("fdc_fft_plan_destroy", p) == FDC_OK
    else:
        assert _lib.last_error()


def test_fft_calls_reject_bad_arguments_before_launch():
    st, p = _fft_plan(2, 16, 16)
    assert st == FDC_OK
    dummy = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first
    assert _lib.status("fdc_rfft2", p, None, dummy, None, 0, None) == FDC_EINVAL
    assert _lib.status("fdc_irfft2", p, dummy, dummy, None, 0, None) == FDC_EWORKSPACE
    assert _lib.status("fdc_irfft2", p, dummy, dummy, dummy, 10, None) == FDC_EWORKSPACE
    assert _lib.status("fdc_rfft2_backward", p, dummy, None, dummy, 1 << 20, None) == FDC_EINVAL
    assert _lib.status("fdc_rfft2", None, dummy, dummy, None, 0, None) == FDC_EINVAL
    for mh, mw in ((0, 16), (16, 0), (15, 16), (16, 17), (66, 16), (16, 66), (-2, 16)):
        assert _lib.status("fdc_rfft2_pooled", p, dummy, dummy, mh, mw, None) == FDC_EINVAL, (mh, mw)
    assert _lib.status("fdc_rfft2_pooled", p, None, dummy, 16, 16, None) == FDC_EINVAL
    assert _lib.status("fdc_rfft2_pooled", None, dummy, dummy, 16, 16, None) == FDC_EINVAL
    for mh, mw in ((0, 16), (16, 0), (15, 16), (16, 17), (66, 16), (16, 66), (-2, 16)):
        assert _lib.status("fdc_rfft2_pooled_ws", p, dummy, dummy, mh, mw, dummy, 1 << 20, None) == FDC_EINVAL
    assert _lib.status("fdc_rfft2_pooled_ws", p, None, dummy, 16, 16, dummy, 1 << 20, None) == FDC_EINVAL
    _lib.status("fdc_fft_plan_destroy", p)
    # above the one-launch sizes the pooled transform needs count * h * (mw/2 + 1) complex values
    st, q = _fft_plan(2, 128, 128)
    assert st == FDC_OK
    need = 2 * 128 * 33 * 8
    assert _lib.status("fdc_rfft2_pooled_ws", q, dummy, dummy, 64, 64, None, need, None) == FDC_EWORKSPACE
    assert _lib.status("fdc_rfft2_pooled_ws", q, dummy, dummy, 64, 64, dummy, need - 1, None) == FDC_EWORKSPACE
    _lib.status("fdc_fft_plan_destroy", q)


@pytest.mark.parametrize("args,expect", [
    ((2, 1, 4, 64, 32, 0, 1), FDC_OK),
    ((1, 2, 6, 16, 8, 1, 3), FDC_OK),          # crop with 3x3 support
    ((1, 2, 6, 1024, 256, 2, 3), FDC_OK),
    ((0, 1, 4, 64, 32, 0, 1), FDC_EINVAL),     # B = 0
    ((2, 3, 4, 64, 32, 0, 1), FDC_EINVAL),     # S mod C != 0
    ((2, 1, 4, 64, 31, 0, 1), FDC_EINVAL),     # odd M
    ((2, 1, 4, 32, 64, 0, 1), FDC_EINVAL),     # M > N
    ((2, 1, 4, 64, 32, 1, 0), FDC_EINVAL),     # crop needs kernel_n >= 1
    ((2, 1, 4, 64, 32, 1, 33), FDC_EINVAL),    # kernel_n > M
    ((2, 1, 4, 64, 32, 7, 1), FDC_EINVAL),     # bad artifact mode
    ((2, 1, 4, 64, 24, 0, 1), FDC_EUNSUPPORTED),  # M not N / 2^k
    ((2, 1, 4, 64, 8, 0, 1), FDC_EUNSUPPORTED),   # N/8: outside the fused set
    ((2, 1, 4, 2048, 1024, 0, 1), FDC_EUNSUPPORTED),
])
def test_cic_layer_plan_validation(args, expect):
    p = ctypes.c_void_p()
    st = _lib.status("fdc_cic_layer_plan_create", ctypes.byref(p), *args)
    assert st == expect, _lib.last_error()
    if st == FDC_OK:
        f, s, b = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
        assert _lib.status("fdc_layer_workspace_size", p, ctypes.byref(f), ctypes.byref(s), ctypes.byref(b)) == 0
        B, C, S, N, M, art, kn = args
        assert s.value == B * C * M * (M // 2 + 1) * 8
        o = ctypes.c_int()
        assert _lib.status("fdc_layer_output_size", p, ctypes.byref(o)) == FDC_OK
        assert o.value == (M - kn + 1 if art == 1 else M)
        assert _lib.status("fdc_layer_plan_destroy", p) == FDC_OK


def test_layer_calls_reject_bad_arguments():
    p = ctypes.c_void_p()
    assert _lib.status("fdc_cic_layer_plan_create", ctypes.byref(p), 2, 1, 4, 64, 32, 0, 1) == FDC_OK
    d = ctypes.c_void_p(0x1000)
    assert _lib.status("fdc_cic_layer_forward", p, d, d, None, None, d, 1 << 30, None) == FDC_EINVAL
    assert _lib.status("fdc_cic_layer_forward", p, d, d, d, None, None, 0, None) == FDC_EWORKSPACE
    assert _lib.status("fdc_cic_layer_backward", p, d, None, d, None, d, d, 1 << 30, None) == FDC_EINVAL
    assert _lib.status("fdc_cic_layer_backward", p, None, d, d, d, d, d, 1 << 30, None) == FDC_EINVAL
    assert _lib.status("fdc_cic_layer_backward", p, d, d, d, d, None, None, 8, None) == FDC_EWORKSPACE
    # a plan of the other kind is refused
    assert _lib.status("fdc_full_forward", p, d, d, d, d, d, 1 << 30, None) == FDC_EINVAL
    assert _lib.status("fdc_layer_plan_destroy", p) == FDC_OK


@pytest.mark.parametrize("args,expect", [
    ((2, 3, 4, 16, 6, 1), FDC_EUNSUPPORTED),   # kernel_n beyond the generated-spectrum set
    ((2, 3, 4, 15, 3, 1), FDC_EINVAL),         # odd P
    ((2, 3, 4, 16, 17, 1), FDC_EINVAL),        # kernel larger than the image
    ((2, 3, 4, 16, 0, 1), FDC_EINVAL),
    ((2, 3, 4, 16, 3, 7), FDC_EINVAL),         # artifact mode
    ((0, 3, 4, 16, 3, 1), FDC_EINVAL),
    ((2, 0, 4, 16, 3, 1), FDC_EINVAL),
    ((2, 3, 0, 16, 3, 1), FDC_EINVAL),
    ((2, 3, 4, 2048, 3, 1), FDC_EUNSUPPORTED),  # outside the FFT length set
    ((2, 3, 4, 4, 3, 1), FDC_EUNSUPPORTED),     # not a multiple of 8
])
def test_full_plan_validation(args, expect):
    """Arguments are checked before the plan touches the device."""
    p = ctypes.c_void_p(0x1234)
    assert _lib.status("fdc_full_layer_plan_create", ctypes.byref(p), *args) == expect
    assert p.value is None


def test_full_plan_valid_sizes_reach_the_device():
    """Valid sizes pass validation; without a device the twiddle-table allocation fails
    with FDC_EHIP, with a device the plan is made and reports its sizes."""
    p = ctypes.c_void_p()
    st = _lib.status("fdc_full_layer_plan_create", ctypes.byref(p), 2, 3, 4, 16, 3, 1)
    assert st in (FDC_OK, FDC_EHIP)
    if st == FDC_EHIP:
        assert "twiddle" in _lib.last_error()
        return
    f, sv, b = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
    assert _lib.status("fdc_layer_workspace_size", p, ctypes.byref(f), ctypes.byref(sv), ctypes.byref(b)) == FDC_OK
    assert sv.value == 2 * 3 * (16 * layers.full_row(16) + layers.full_side_plane(16)) * 8
    o = ctypes.c_int()
    assert _lib.status("fdc_layer_output_size", p, ctypes.byref(o)) == FDC_OK
    assert o.value == 14
    d = ctypes.c_void_p(0x1000)
    # a plan of the other kind is refused
    assert _lib.status("fdc_cic_layer_forward", p, d, d, d, None, d, 1 << 30, None) == FDC_EINVAL
    assert _lib.status("fdc_full_forward", p, d, d, d, None, None, 0, None) == FDC_EWORKSPACE
    assert _lib.status("fdc_full_backward", p, d, None, d, None, d, d, 1 << 30, None) == FDC_EINVAL
    assert _lib.status("fdc_layer_plan_destroy", p) == FDC_OK


@pytest.mark.parametrize("args,expect", [
    ((1, 8, 8, 4, 4), FDC_OK), ((3, 10, 12, 6, 8), FDC_OK),
    ((0, 8, 8, 4, 4), FDC_EINVAL), ((1, 8, 8, 10, 4), FDC_EINVAL), ((1, 8, 8, 3, 4), FDC_EINVAL),
])
def test_fdp_validation(args, expect):
    count, H, W, Mh, Mw = args
    if expect == FDC_OK:
        # valid sizes with NULL tensors still fail, but on the tensor check
        assert _lib.status("fdp_forward", None, None, count, H, W, Mh, Mw, None) == FDC_EINVAL
        assert "NULL" in _lib.last_error()
    else:
        assert _lib.status("fdp_forward", None, None, count, H, W, Mh, Mw, None) == expect
        assert "NULL" not in _lib.last_error()


def test_cic_spectral_validation():
    d = ctypes.c_void_p(0x1000)
    assert _lib.status("fdc_cic_forward", d, d, d, 2, 3, 4, 8, 5, None) == FDC_EINVAL
    assert _lib.status("fdc_cic_forward", d, d, d, 0, 1, 4, 8, 5, None) == FDC_EINVAL
    assert _lib.status("fdc_cic_backward", None, d, d, d, d, 2, 1, 4, 8, 5, None) == FDC_EINVAL


def test_timing_api_arguments():
    assert _lib.status("fdc_kernel_timing_enable", 0, None) == FDC_EINVAL
    assert _lib.status("fdc_kernel_timing_enable", -3, b"row_r2c_64") == FDC_EINVAL
    assert _lib.status("fdc_kernel_timing_report", None, 0) == FDC_EINVAL
    assert _lib.status("fdc_kernel_timing_launches", None, 0) == FDC_EINVAL


def test_destroyed_plan_is_refused():
    """Handles are looked up in the library's registry of live plans before they are
    read: a destroyed handle, a never-created one and a plan of another type are all
    refused with FDC_EINVAL, without touching freed memory."""
    st, p = _fft_plan(1, 8, 8)
    assert st == FDC_OK
    n = ctypes.c_size_t()
    bogus = ctypes.create_string_buffer(64)
    assert _lib.status("fdc_fft_workspace_size", ctypes.cast(bogus, ctypes.c_void_p), ctypes.byref(n)) == FDC_EINVAL
    # an fft plan is not a layer or stack plan
    assert _lib.status("fdc_layer_workspace_size", p, None, None, None) == FDC_EINVAL
    assert _lib.status("fdc_cic_stack_workspace_size", p, None, None) == FDC_EINVAL
    assert _lib.status("fdc_fft_plan_destroy", p) == FDC_OK
    assert _lib.status("fdc_fft_workspace_size", p, ctypes.byref(n)) == FDC_EINVAL
    assert _lib.status("fdc_rfft2", p, ctypes.c_void_p(0x1000), ctypes.c_void_p(0x1000), None, 0, None) == FDC_EINVAL
    assert _lib.status("fdc_fft_plan_destroy", p) == FDC_EINVAL  # a second destroy
    assert _lib.status("fdc_fft_plan_destroy", None) == FDC_OK


def test_destroyed_layer_and_stack_plans_are_refused():
    lp = ctypes.c_void_p()
    assert _lib.status("fdc_cic_layer_plan_create", ctypes.byref(lp), 2, 1, 4, 64, 32, 0, 1) == FDC_OK
    assert _lib.status("fdc_layer_plan_destroy", lp) == FDC_OK
    d = ctypes.c_void_p(0x1000)
    assert _lib.status("fdc_layer_output_size", lp, ctypes.byref(ctypes.c_int())) == FDC_EINVAL
    assert _lib.status("fdc_cic_layer_forward", lp, d, d, d, None, d, 1 << 30, None) == FDC_EINVAL
    assert _lib.status("fdc_layer_plan_destroy", lp) == FDC_EINVAL
    st, sp = _stack(2, (64, 32), (1, 4))
    assert st == FDC_OK
    assert _lib.status("fdc_layer_workspace_size", sp, None, None, None) == FDC_EINVAL  # not a layer plan
    assert _lib.status("fdc_cic_stack_plan_destroy", sp) == FDC_OK
    assert _lib.status("fdc_cic_stack_plan_destroy", sp) == FDC_EINVAL


def test_oversize_counts_fail_before_any_launch():
    """Sizes beyond the kernels' 32-bit row and grid indexing are refused with
    FDC_EUNSUPPORTED when the plan is made (or at the top of a call without a plan),
    so no later call can enqueue part of its work and then fail.  On a machine
    without a GPU any launch would return FDC_EHIP instead, so these statuses also
    show that nothing was launched."""
    p = ctypes.c_void_p()
    assert _lib.status("fdc_fft_plan_create", ctypes.byref(p), 1 << 30, 2, 2) == FDC_EUNSUPPORTED
    assert _lib.status("fdc_fft_plan_create", ctypes.byref(p), (1 << 31) // 1024, 1024, 16) == FDC_EUNSUPPORTED
    st, q = _fft_plan((1 << 30) - 1, 2, 2)  # the largest count of 2 x 2 images
    assert st == FDC_OK
    assert _lib.status("fdc_fft_plan_destroy", q) == FDC_OK
    assert _lib.status("fdc_cic_layer_plan_create", ctypes.byref(p), 1 << 21, 1, 1, 1024, 512, 0, 1) == FDC_EUNSUPPORTED
    assert _lib.status("fdc_cic_layer_plan_create", ctypes.byref(p), 1 << 16, 1, 1024, 64, 32, 0, 1) == FDC_EUNSUPPORTED
    st, _ = _stack(1 << 21, (1024, 512), (1, 1))
    assert st == FDC_EUNSUPPORTED
    assert _lib.status("fdc_full_layer_plan_create", ctypes.byref(p), 16, 1 << 20, 64, 512, 3, 1) == FDC_EUNSUPPORTED
    d = ctypes.c_void_p(0x1000)
    assert _lib.status("fdc_cic_fdp_forward", d, d, d, 1, 1, 1, 8192, 4096, None) == FDC_EUNSUPPORTED
    assert _lib.status("fdc_cic_fdp_backward", d, d, d, d, d, 1, 1, 1, 8192, 4096, None) == FDC_EUNSUPPORTED
    n = ctypes.c_size_t()
    assert _lib.status("fdc_head_workspace_size", 1, 1 << 38, 2, ctypes.byref(n)) == FDC_EUNSUPPORTED


def test_full_plane_strides_match_header():
    """The binding's copy of the saved-spectrum strides equals the header's macros."""
    import os
    import re
    hdr = open(os.path.join(os.path.dirname(__file__), "..", "include", "fdc.h")).read()
    m = re.search(r"#define FDC_FULL_ROW\(P\) \(\(int64_t\)\(P\) / 2 \+ (\d+)\)", hdr)
    s = re.search(r"#define FDC_FULL_SIDE_PLANE\(P\) \(\(int64_t\)\(P\) \+ (\d+)\)", hdr)
    assert m and s
    for P in (8, 224, 512):
        assert layers.full_row(P) == P // 2 + int(m.group(1))
        assert layers.full_side_plane(P) == P + int(s.group(1))


def _stack(B, sizes, chans):
    p = ctypes.c_void_p()
    st = _lib.status("fdc_cic_stack_plan_create", ctypes.byref(p), B, len(sizes) - 1,
                     (ctypes.c_int * len(sizes))(*sizes), (ctypes.c_int * len(chans))(*chans))
    return st, p


@pytest.mark.parametrize("B,sizes,chans,expect", [
    (8, (64, 32, 16), (1, 4, 8), FDC_OK),
    (0, (64, 32), (1, 4), FDC_EINVAL),
    (2, (64,), (1,), FDC_EINVAL),              # no layer
    (2, (64, 32), (2, 3), FDC_EINVAL),         # S mod C != 0
    (2, (32, 64), (1, 2), FDC_EINVAL),         # growing size
    (2, (64, 30), (1, 2), FDC_EUNSUPPORTED),   # a valid FDP size, but not a pooling the fused layer has
    (2, (2048, 1024), (1, 2), FDC_EUNSUPPORTED),
])
def test_stack_plan_validation(B, sizes, chans, expect):
    st, p = _stack(B, sizes, chans)
    assert st == expect
    if st == FDC_OK:
        assert _lib.status("fdc_cic_stack_plan_destroy", p) == FDC_OK


def test_stack_plan_sizes_and_argument_checks():
    """Saved sizes equal the layer plans'; workspaces cover every layer's spectra;
    bad arguments are refused before anything is enqueued."""
    B, sizes, chans = 4, (256, 128, 64), (1, 8, 16)
    st, p = _stack(B, sizes, chans)
    assert st == FDC_OK
    f, b = ctypes.c_size_t(), ctypes.c_size_t()
    assert _lib.status("fdc_cic_stack_workspace_size", p, ctypes.byref(f), ctypes.byref(b)) == FDC_OK
    tmax = 0
    for i in range(2):
        N, M, C, S = sizes[i], sizes[i + 1], chans[i], chans[i + 1]
        L = M // 2 + 1
        tmax = max(tmax, B * C * N * L, B * S * M * L)
        n = ctypes.c_size_t()
        assert _lib.status("fdc_cic_stack_saved_size", p, i, ctypes.byref(n)) == FDC_OK
        lp = ctypes.c_void_p()
        assert _lib.status("fdc_cic_layer_plan_create", ctypes.byref(lp), B, C, S, N, M, 0, 1) == FDC_OK
        sv = ctypes.c_size_t()
        assert _lib.status("fdc_layer_workspace_size", lp, None, ctypes.byref(sv), None) == FDC_OK
        assert n.value == sv.value
        assert _lib.status("fdc_layer_plan_destroy", lp) == FDC_OK
    assert b.value == 2 * tmax * 8 and f.value >= b.value
    n = ctypes.c_size_t()
    assert _lib.status("fdc_cic_stack_saved_size", p, 2, ctypes.byref(n)) == FDC_EINVAL
    d = ctypes.c_void_p(0x1000)
    arr = (ctypes.c_void_p * 2)(0x1000, 0x1000)
    null_arr = (ctypes.c_void_p * 2)(0x1000, None)
    assert _lib.status("fdc_cic_stack_forward", p, d, null_arr, d, None, d, 1 << 40, None) == FDC_EINVAL
    assert _lib.status("fdc_cic_stack_forward", p, d, arr, d, None, d, 8, None) == FDC_EWORKSPACE
    assert _lib.status("fdc_cic_stack_backward", p, d, arr, arr, None, null_arr, d, 1 << 40, None) == FDC_EINVAL
    assert _lib.status("fdc_cic_stack_backward", p, d, arr, arr, None, arr, d, 8, None) == FDC_EWORKSPACE
    assert _lib.status("fdc_cic_stack_plan_destroy", p) == FDC_OK
    assert _lib.status("fdc_cic_stack_forward", p, d, arr, d, None, d, 1 << 40, None) == FDC_EINVAL


def test_hermitian_project_validation():
    d = ctypes.c_void_p(0x1000)
    assert _lib.status("fdc_hermitian_project", d, 0, 8, 8, None) == FDC_EINVAL   # no planes
    assert _lib.status("fdc_hermitian_project", d, 2, 7, 8, None) == FDC_EINVAL   # odd H
    assert _lib.status("fdc_hermitian_project", d, 2, 8, 5, None) == FDC_EINVAL   # odd W
    assert _lib.status("fdc_hermitian_project", None, 2, 8, 8, None) == FDC_EINVAL


def test_cic_fdp_validation():
    d = ctypes.c_void_p(0x1000)
    assert _lib.status("fdc_cic_fdp_forward", d, d, d, 2, 3, 4, 8, 4, None) == FDC_EINVAL  # S mod C
    assert _lib.status("fdc_cic_fdp_forward_projected", d, d, d, 2, 3, 4, 8, 4, None) == FDC_EINVAL
    assert _lib.status("fdc_cic_fdp_backward_projected", d, d, d, d, d, 2, 1, 4, 8, 3, None) == FDC_EINVAL
    assert _lib.status("fdc_cic_fdp_backward_projected", d, d, d, None, None, 2, 1, 4, 8, 4, None) == FDC_OK
    assert _lib.status("fdc_cic_fdp_forward", d, d, d, 2, 1, 4, 8, 16, None) == FDC_EINVAL  # M > N
    assert _lib.status("fdc_cic_fdp_forward", d, d, d, 2, 1, 4, 8, 3, None) == FDC_EINVAL   # odd M
    assert _lib.status("fdc_cic_fdp_forward", None, d, d, 2, 1, 4, 8, 4, None) == FDC_EINVAL
    assert _lib.status("fdc_cic_fdp_backward", d, None, d, None, d, 2, 1, 4, 8, 4, None) == FDC_EINVAL  # gK needs X
    assert _lib.status("fdc_cic_fdp_backward", d, d, None, d, None, 2, 1, 4, 8, 4, None) == FDC_EINVAL  # gX needs K
    assert _lib.status("fdc_cic_fdp_backward", d, d, d, None, None, 2, 1, 4, 8, 4, None) == FDC_OK     # nothing asked
    m = ctypes.c_void_p(0x1008)  # 8- but not 16-byte aligned output
    assert _lib.status("fdc_cic_fdp_forward", d, d, m, 2, 1, 4, 8, 4, None) == FDC_EINVAL
    assert _lib.status("fdc_cic_fdp_backward", d, d, d, m, None, 2, 1, 4, 8, 4, None) == FDC_EINVAL
    # the dK grid: 2052 blocks of a 1024 x 513 plane times S channels must stay below 2^31
    big = 1 << 20
    assert _lib.status("fdc_cic_fdp_forward", d, d, d, 1, big, big, 1024, 512, None) == FDC_EUNSUPPORTED
    assert _lib.status("fdc_cic_fdp_backward", d, d, d, None, d, 1, big, big, 1024, 512, None) == FDC_EUNSUPPORTED


def test_dk_ranges_queries():
    """The dK batch-range count is a host-side function of the plan: one range at 8
    images, several at 32 (the 512 stack); bad plans, layers and NULL outputs are
    refused."""
    r = ctypes.c_int()
    lp = ctypes.c_void_p()
    assert _lib.status("fdc_cic_layer_plan_create", ctypes.byref(lp), 8, 1, 8, 1024, 512, 0, 1) == FDC_OK
    assert _lib.status("fdc_cic_layer_dk_ranges", lp, ctypes.byref(r)) == FDC_OK and r.value == 1
    assert _lib.status("fdc_cic_layer_dk_ranges", lp, None) == FDC_EINVAL
    assert _lib.status("fdc_layer_plan_destroy", lp) == FDC_OK
    st, sp = _stack(32, (512, 256, 128, 64, 32), (1, 8, 16, 32, 64))
    assert st == FDC_OK
    got = []
    for i in range(4):
        assert _lib.status("fdc_cic_stack_dk_ranges", sp, i, ctypes.byref(r)) == FDC_OK
        got.append(r.value)
    assert all(1 < g <= 32 // 8 for g in got), got
    assert _lib.status("fdc_cic_stack_dk_ranges", sp, 4, ctypes.byref(r)) == FDC_EINVAL
    assert _lib.status("fdc_cic_stack_plan_destroy", sp) == FDC_OK
    assert _lib.status("fdc_cic_stack_dk_ranges", sp, 0, ctypes.byref(r)) == FDC_EINVAL  # destroyed


def test_head_and_adam_validation():
    """The classifier head and Adam refuse bad sizes and NULL arguments on the host,
    before any launch; the head workspace is one float per (chunk of 1024 features,
    image, class)."""
    n = ctypes.c_size_t()
    assert _lib.status("fdc_head_workspace_size", 8, 131072, 2, ctypes.byref(n)) == FDC_OK
    assert n.value == 128 * 8 * 2 * 4
    assert _lib.status("fdc_head_workspace_size", 3, 1025, 5, ctypes.byref(n)) == FDC_OK and n.value == 2 * 3 * 5 * 4
    assert _lib.status("fdc_head_workspace_size", 0, 10, 2, ctypes.byref(n)) == FDC_EINVAL
    assert _lib.status("fdc_head_workspace_size", 2, 0, 2, ctypes.byref(n)) == FDC_EINVAL
    assert _lib.status("fdc_head_workspace_size", 2, 10, 0, ctypes.byref(n)) == FDC_EUNSUPPORTED
    assert _lib.status("fdc_head_workspace_size", 2, 10, 17, ctypes.byref(n)) == FDC_EUNSUPPORTED
    assert _lib.status("fdc_head_workspace_size", 4096, 10, 16, ctypes.byref(n)) == FDC_EUNSUPPORTED  # LDS
    assert _lib.status("fdc_head_workspace_size", 2, 10, 2, None) == FDC_EINVAL
    fake = ctypes.c_void_p(0x1000)
    # NULL tensors and a short workspace
    assert _lib.status("fdc_head_forward", None, fake, fake, fake, fake, fake, 2, 10, 2, fake, 16, None) == FDC_EINVAL
    assert _lib.status("fdc_head_forward", fake, fake, fake, fake, fake, fake, 2, 10, 2, fake, 15,
                       None) == FDC_EWORKSPACE
    assert _lib.status("fdc_head_backward", fake, fake, fake, fake, None, None, fake, 2, 10, 2,
                       None) == FDC_EINVAL
    f = ctypes.c_float
    assert _lib.status("fdc_adam_step", fake, fake, fake, fake, -1, fake, f(1e-3), f(0.9), f(0.999), f(1e-8), f(0.0),
                       None) == FDC_EINVAL
    assert _lib.status("fdc_adam_step", fake, fake, fake, fake, 10, None, f(1e-3), f(0.9), f(0.999), f(1e-8), f(0.0),
                       None) == FDC_EINVAL
    assert _lib.status("fdc_adam_step", None, fake, fake, fake, 10, fake, f(1e-3), f(0.9), f(0.999), f(1e-8), f(0.0),
                       None) == FDC_EINVAL
    assert _lib.status("fdc_adam_step", fake, fake, fake, fake, 10, fake, f(1e-3), f(1.0), f(0.999), f(1e-8), f(0.0),
                       None) == FDC_EINVAL
