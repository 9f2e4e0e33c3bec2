"""Parity criterion shared by the GPU tests.

fp32 GPU results are compared with the float64 oracle evaluated on the same
(fp32) inputs.  A tensor passes when
  * its relative L2 error ||got - ref|| / ||ref|| is at most 1e-4, and
  * its largest absolute error is at most 1e-3 * max|ref|.
For a transform of length n the fp32 rounding error grows like
eps * log2(n) (eps = 6e-8), i.e. below 1e-6 relative for n <= 1024 per
transform; a layer chains four transforms and a product, and a stack chains up
to five layers, so 1e-4 leaves a margin of more than 10x.
"""

import numpy as np

REL_L2 = 1e-4
MAX_ABS_FRAC = 1e-3


def to_np(t):
    return t.detach().cpu().numpy()


def rel_l2(got, ref):
    got = np.asarray(got, dtype=np.complex128 if np.iscomplexobj(got) else np.float64)
    ref = np.asarray(ref)
    den = np.linalg.norm(ref.ravel())
    num = np.linalg.norm((got - ref).ravel())
    return num / den if den > 0 else num


def assert_parity(got, ref, name="tensor", rel=REL_L2, max_abs_frac=MAX_ABS_FRAC):
    got = np.asarray(got)
    ref = np.asarray(ref)
    assert got.shape == ref.shape, f"{name}: shape {got.shape} vs {ref.shape}"
    assert np.all(np.isfinite(got)), f"{name}: non-finite values"
    r = rel_l2(got, ref)
    scale = np.abs(ref).max()
    m = np.abs(got - ref).max()
    assert r <= rel, f"{name}: rel-L2 {r:.3e} > {rel:.1e}"
    assert m <= max_abs_frac * scale + 1e-30, f"{name}: max|d| {m:.3e} > {max_abs_frac:.0e} * {scale:.3e}"
    return r
