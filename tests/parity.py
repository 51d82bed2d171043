"""Comparison helpers shared by the GPU parity tests."""
import numpy as np

# Parameter tolerance of the parity bar: per worker (row) and per array,
# max_c |gpu - ref| <= REL_TOL * max_c |ref|.
REL_TOL = 1e-6


def rel_err_per_row(got: np.ndarray, ref: np.ndarray) -> np.ndarray:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    num = np.abs(got - ref).max(axis=1) if got.shape[1] else np.zeros(got.shape[0])
    den = np.abs(ref).max(axis=1) if ref.shape[1] else np.ones(ref.shape[0])
    den = np.where(den == 0, 1.0, den)
    return num / den


def assert_params_close(got, ref, what: str, tol: float = REL_TOL):
    got = np.asarray(got)
    ref = np.asarray(ref)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.isfinite(got).all(), f"{what}: non-finite values"
    err = rel_err_per_row(got, ref)
    worst = int(err.argmax()) if err.size else 0
    assert (err <= tol).all(), (
        f"{what}: worker {worst} max-norm relative error {err[worst]:.3e} > {tol:g}")


def bit_mismatches(got, ref) -> int:
    g = np.ascontiguousarray(got, dtype=np.float32).view(np.uint32)
    r = np.ascontiguousarray(ref, dtype=np.float32).view(np.uint32)
    return int((g != r).sum())
