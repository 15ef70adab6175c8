"""Tolerance rule of the fp32 HIP path against the fp64 oracle.

Per tensor: max|a - b| <= tol * max|b| (normwise), and elementwise
|a - b| <= tol * |b| wherever |b| >= 1e-2 * max|b|.  tol = 1e-4 relative,
the bound stated for the deterministic mode.  Elements far below the
tensor's scale are covered by the normwise bound only: their relative error
is dominated by fp32 rounding of larger terms of the same sums.
"""
import numpy as np

TOL = 1e-4


def close_report(a, b, tol=TOL, floor=1e-2):
    a = np.asarray(a, dtype=np.float64).ravel()
    b = np.asarray(b, dtype=np.float64).ravel()
    assert a.shape == b.shape, (a.shape, b.shape)
    scale = float(np.max(np.abs(b))) if b.size else 0.0
    if scale == 0.0:
        err = float(np.max(np.abs(a))) if a.size else 0.0
        return err == 0.0, f"reference all zero, max|a|={err:g}"
    diff = np.abs(a - b)
    norm_err = float(diff.max()) / scale
    big = np.abs(b) >= floor * scale
    rel = diff[big] / np.abs(b[big])
    worst = float(rel.max()) if rel.size else 0.0
    ok = norm_err <= tol and worst <= tol and np.all(np.isfinite(a))
    return ok, f"normwise {norm_err:.3g}, elementwise(|b|>={floor:g}*max) {worst:.3g}, scale {scale:.3g}"


def assert_close(a, b, tol=TOL, what=""):
    ok, msg = close_report(a, b, tol)
    assert ok, f"{what}: {msg}"
