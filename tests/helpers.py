"""Shared test helpers: tolerances and comparisons (no layer arithmetic)."""
import numpy as np

# relative tolerance of the GPU path against the fp64 oracle:
# max |gpu - ref| / max |ref| over each output tensor
TOL_F32 = 1e-4
TOL_BF16 = 2e-2


def rel_err(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    if got.size == 0:
        return 0.0
    assert np.all(np.isfinite(got)), "non-finite values in GPU output"
    scale = np.max(np.abs(ref))
    diff = np.max(np.abs(got - ref))
    if scale == 0.0:
        return diff
    return diff / scale


def assert_close(got, ref, tol, what=""):
    e = rel_err(got, ref)
    assert e <= tol, f"{what}: relative error {e:.3e} > {tol:.1e}"
    return e
