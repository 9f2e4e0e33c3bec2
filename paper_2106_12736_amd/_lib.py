"""ctypes binding of libfdc (include/fdc.h).

Argument marshalling only: every function hands device pointers, sizes and
the current HIP stream to the C ABI, and raises FdcError on a non-OK status.
There is no fallback of any kind: if libfdc.so is missing the first call
raises.
"""

import ctypes
import os
import re

_HERE = os.path.dirname(os.path.abspath(__file__))
# FDC_LIBRARY may name another build of the same library (same ABI), e.g. to compare builds.
LIB_PATH = os.environ.get("FDC_LIBRARY") or os.path.join(_HERE, "libfdc.so")
HEADER = os.path.join(os.path.dirname(_HERE), "include", "fdc.h")

FDC_OK, FDC_EINVAL, FDC_EUNSUPPORTED, FDC_EWORKSPACE, FDC_EHIP = range(5)
ARTIFACT_NONE, ARTIFACT_CROP, ARTIFACT_ROLL = range(3)

_P = ctypes.c_void_p
_I = ctypes.c_int
_I64 = ctypes.c_int64
_SZ = ctypes.c_size_t
_PP = ctypes.POINTER(ctypes.c_void_p)

# name -> argtypes (restype is int status unless listed in _RESTYPES)
_SIGS = {
    "fdc_status_string": [_I],
    "fdc_last_error": [],
    "fdc_version": [],
    "fdc_fft_plan_create": [_PP, _I64, _I, _I],
    "fdc_fft_plan_destroy": [_P],
    "fdc_fft_workspace_size": [_P, ctypes.POINTER(_SZ)],
    "fdc_rfft2": [_P, _P, _P, _P, _SZ, _P],
    "fdc_irfft2": [_P, _P, _P, _P, _SZ, _P],
    "fdc_rfft2_backward": [_P, _P, _P, _P, _SZ, _P],
    "fdc_irfft2_backward": [_P, _P, _P, _P, _SZ, _P],
    "fdc_rfft2_pooled": [_P, _P, _P, _I, _I, _P],
    "fdc_rfft2_pooled_ws": [_P, _P, _P, _I, _I, _P, _SZ, _P],
    "fdc_cic_forward": [_P, _P, _P, _I, _I, _I, _I, _I, _P],
    "fdc_cic_backward": [_P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _P],
    "fdc_cic_fdp_forward": [_P, _P, _P, _I, _I, _I, _I, _I, _P],
    "fdc_cic_fdp_backward": [_P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _P],
    "fdc_cic_fdp_forward_projected": [_P, _P, _P, _I, _I, _I, _I, _I, _P],
    "fdc_cic_fdp_backward_projected": [_P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _P],
    "fdc_cic_fdp_backward_kept": [_P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _P],
    "fdc_cic_fdp_backward_projected_kept": [_P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _P],
    "fdp_forward": [_P, _P, _I64, _I, _I, _I, _I, _P],
    "fdc_head_workspace_size": [_I, _I64, _I, ctypes.POINTER(_SZ)],
    "fdc_head_forward": [_P, _P, _P, _P, _P, _P, _I, _I64, _I, _P, _SZ, _P],
    "fdc_head_forward_noalloc": [_P, _P, _P, _P, _P, _P, _I, _I64, _I, _P],
    "fdc_head_backward": [_P, _P, _P, _P, _P, _P, _P, _I, _I64, _I, _P],
    "fdc_adam_step": [_P, _P, _P, _P, _I64, _P, ctypes.c_float, ctypes.c_float, ctypes.c_float, ctypes.c_float,
                      ctypes.c_float, _P],
    "fdp_backward": [_P, _P, _I64, _I, _I, _I, _I, _P],
    "fdc_cic_layer_plan_create": [_PP, _I, _I, _I, _I, _I, _I, _I],
    "fdc_full_layer_plan_create": [_PP, _I, _I, _I, _I, _I, _I],
    "fdc_layer_plan_destroy": [_P],
    "fdc_layer_workspace_size": [_P, ctypes.POINTER(_SZ), ctypes.POINTER(_SZ), ctypes.POINTER(_SZ)],
    "fdc_layer_output_size": [_P, ctypes.POINTER(_I)],
    "fdc_cic_layer_forward": [_P, _P, _P, _P, _P, _P, _SZ, _P],
    "fdc_cic_layer_backward": [_P, _P, _P, _P, _P, _P, _P, _SZ, _P],
    "fdc_cic_spatial_workspace_size": [_P, ctypes.POINTER(_SZ), ctypes.POINTER(_SZ)],
    "fdc_cic_spatial_layer_forward": [_P, _P, _P, _P, _P, _P, _SZ, _P],
    "fdc_cic_spatial_layer_backward": [_P, _P, _P, _P, _P, _P, _P, _SZ, _P],
    "fdc_full_forward": [_P, _P, _P, _P, _P, _P, _SZ, _P],
    "fdc_full_backward": [_P, _P, _P, _P, _P, _P, _P, _SZ, _P],
    "fdc_cic_stack_plan_create": [_PP, _I, _I, _P, _P],
    "fdc_cic_stack_plan_destroy": [_P],
    "fdc_cic_stack_workspace_size": [_P, ctypes.POINTER(_SZ), ctypes.POINTER(_SZ)],
    "fdc_cic_stack_saved_size": [_P, _I, ctypes.POINTER(_SZ)],
    "fdc_cic_stack_forward": [_P, _P, _P, _P, _P, _P, _SZ, _P],
    "fdc_cic_stack_backward": [_P, _P, _P, _P, _P, _P, _P, _SZ, _P],
    "fdc_cic_stack_backward_kept": [_P, _P, _P, _P, _P, _P, _P, _SZ, _P],
    "fdc_hermitian_project": [_P, _I64, _I, _I, _P],
    "fdc_cic_spatial_stack_workspace_size": [_P, _I, ctypes.POINTER(_SZ), ctypes.POINTER(_SZ)],
    "fdc_cic_spatial_stack_forward": [_P, _I, _P, _P, _P, _P, _P, _SZ, _P],
    "fdc_cic_spatial_stack_backward": [_P, _I, _P, _P, _P, _P, _P, _P, _SZ, _P],
    "fdc_kernel_timing_enable": [_I, ctypes.c_char_p],
    "fdc_kernel_timing_disable": [],
    "fdc_kernel_timing_report": [ctypes.c_char_p, _SZ],
    "fdc_kernel_timing_launches": [ctypes.c_char_p, _SZ],
    "fdc_cic_layer_dk_ranges": [_P, ctypes.POINTER(_I)],
    "fdc_cic_stack_dk_ranges": [_P, _I, ctypes.POINTER(_I)],
    "fdc_cic_stack_tail": [_P, ctypes.POINTER(_I)],
}
_RESTYPES = {"fdc_status_string": ctypes.c_char_p, "fdc_last_error": ctypes.c_char_p, "fdc_version": _I}

_lib = None


class FdcError(RuntimeError):
    def __init__(self, status, func, detail):
        self.status = status
        super().__init__(f"{func} -> status {status}: {detail}")


def header_functions():
    """Names of the functions include/fdc.h declares."""
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b((?:fdc|fdp)_[a-z0-9_]+)\s*\(", text)))


def lib():
    """Load libfdc.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2106_12736_amd.build`")
        handle = ctypes.CDLL(LIB_PATH)
        for name, args in _SIGS.items():
            fn = getattr(handle, name)
            fn.argtypes = args
            fn.restype = _RESTYPES.get(name, _I)
        _lib = handle
    return _lib


def call(name, *args):
    """Call an fdc entry point that returns a status; raise FdcError unless FDC_OK."""
    st = getattr(lib(), name)(*args)
    if st != FDC_OK:
        raise FdcError(st, name, lib().fdc_last_error().decode())
    return st


def status(name, *args):
    """Call an fdc entry point and return its raw status (for tests of error paths)."""
    return getattr(lib(), name)(*args)


def last_error():
    return lib().fdc_last_error().decode()
