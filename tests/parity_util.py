"""Comparison helpers shared by the GPU parity tests."""
from __future__ import annotations

import numpy as np

FP32_TOL = 1e-5   # per-row relative L2, fp32 path
BF16_TOL = 2e-2   # per-row relative L2, bf16 path


def row_errors(gpu: np.ndarray, ref: np.ndarray):
    """(relative L2 error per row, absolute L2 error per row, reference row norms)."""
    g = np.asarray(gpu, dtype=np.float64)
    r = np.asarray(ref, dtype=np.float64)
    assert g.shape == r.shape, (g.shape, r.shape)
    diff = np.linalg.norm(g - r, axis=1) if g.size else np.zeros(g.shape[0])
    norm = np.linalg.norm(r, axis=1) if r.size else np.zeros(r.shape[0])
    return diff, norm


def assert_rows_close(gpu, ref, tol: float, what: str = "", floor=None):
    """Per-row relative L2 error <= tol.

    Rows whose reference norm is below 1e-3 of the median row norm (rows a
    ReLU has mapped to, or near, zero) are held to an absolute bound of
    tol * median row norm instead, since a relative error is meaningless
    there.  ``floor`` (per-row norms) raises each row's denominator to the
    scale of its rounding error where the result cancels: for a sum that is
    the same sum over absolute values (the classical summation error bound
    is proportional to it).  Returns the worst relative error on the regular
    rows.
    """
    diff, norm = row_errors(gpu, ref)
    if floor is not None:
        norm = np.maximum(norm, np.asarray(floor, dtype=np.float64))
    if diff.size == 0:
        return 0.0
    med = float(np.median(norm)) if np.any(norm > 0) else 0.0
    small = norm <= 1e-3 * med
    rel = np.where(small, 0.0, diff / np.where(small, 1.0, norm))
    worst = float(rel.max())
    assert worst <= tol, f"{what}: worst per-row relative error {worst:.3e} > {tol:.1e} (row {int(rel.argmax())})"
    if small.any():
        worst_abs = float(diff[small].max())
        assert worst_abs <= tol * max(med, 1e-30), f"{what}: near-zero rows off by {worst_abs:.3e}"
    return worst


def elementwise_report(gpu, ref) -> float:
    g = np.asarray(gpu, dtype=np.float64)
    r = np.asarray(ref, dtype=np.float64)
    if g.size == 0:
        return 0.0
    rms = float(np.sqrt(np.mean(r * r))) or 1.0
    return float(np.max(np.abs(g - r) / (np.abs(r) + rms)))
