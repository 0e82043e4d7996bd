"""Shared comparison helpers for the GPU parity tests (no arithmetic of the step)."""
import numpy as np


def normwise(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref.ravel())
    return float(np.linalg.norm((got - ref).ravel()) / (den if den > 0 else 1.0))


def max_rel(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.max(np.abs(got - ref) / np.abs(ref)))


def assert_normwise(got, ref, tol, what):
    e = normwise(got, ref)
    print(f"  {what}: normwise rel err {e:.3e} (tol {tol:.0e})", flush=True)
    assert e <= tol, f"{what}: normwise relative error {e:.3e} > {tol:.0e}"


def assert_condition_aware(got, ref, cond, tol, what):
    """Every entry within tol * sum|terms| of the oracle (cancelling sums)."""
    got = np.asarray(got, dtype=np.float64)
    err = np.abs(got - ref)
    worst = float(np.max(err / np.maximum(cond, 1e-300)))
    print(f"  {what}: max |err| / sum|terms| {worst:.3e} (tol {tol:.0e})", flush=True)
    assert np.all(err <= tol * cond), f"{what}: entry error beyond {tol:.0e} * sum|terms| ({worst:.3e})"


def to_np(t):
    return t.detach().cpu().numpy()


def words_np(t):
    return to_np(t).view(np.uint32)
