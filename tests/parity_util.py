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
    there.  ``floor`` (per-row norms of the same sums over absolute values,
    the scale of the classical summation error bound) applies only to rows
    whose result cancels: a row whose reference norm is below 1e-2 of its
    floor is measured against the floor, every other row against its own
    norm.  The worst error over the regular rows, and (with a floor) the
    worst error every row would show against its own norm, are printed.
    Returns the worst relative error on the regular rows.
    """
    diff, norm = row_errors(gpu, ref)
    if diff.size == 0:
        return 0.0
    med = float(np.median(norm)) if np.any(norm > 0) else 0.0
    small = norm <= 1e-3 * med
    denom = norm
    if floor is not None:
        fl = np.asarray(floor, dtype=np.float64)
        cancels = norm < 1e-2 * fl
        denom = np.where(cancels, fl, norm)
        raw = np.where(small | (norm == 0), 0.0, diff / np.where(norm > 0, norm, 1.0))
        print(f"[rows] {what}: worst relative error {float(raw.max()):.3e} against each row's own norm; "
              f"{int(cancels.sum())} of {norm.size} rows cancel below 1e-2 of their floor", flush=True)
    rel = np.where(small, 0.0, diff / np.where(small, 1.0, denom))
    worst = float(rel.max())
    print(f"[rows] {what}: worst relative error {worst:.3e} (tolerance {tol:.1e})", flush=True)
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
