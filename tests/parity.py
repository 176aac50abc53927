"""Parity rule shared by the oracle pins and the GPU parity tests.

Row i passes iff every entry is finite and
    max_l |A_il - Aref_il|  <=  tol * scale_i,
    scale_i = max_l sum_p |b_p| (sum_k |C_ik||D_jk|) |E_jl|
(the computation run on absolute values, returned by the oracle).  When
scale_i == 0 the row must be exactly zero.  tol = 1e-4 for fp32 results.

For SDDMM values the same rule applies per nonzero with
    scale_p = |b_p| sum_k |C_ik||D_jk|.
"""
from __future__ import annotations

import numpy as np

TOL = 1e-4


def row_errors(A, Aref, scale):
    """Per-row (max abs error, ratio err/scale); ratio is inf for a failing zero-scale row."""
    A = np.asarray(A, dtype=np.float64)
    Aref = np.asarray(Aref, dtype=np.float64)
    scale = np.asarray(scale, dtype=np.float64)
    if A.ndim == 1:
        A = A[:, None]
        Aref = Aref[:, None]
    if A.shape[1] == 0:
        z = np.zeros(A.shape[0])
        return z, z
    err = np.abs(A - Aref).max(axis=1)
    finite = np.isfinite(A).all(axis=1)
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(scale > 0, err / np.where(scale > 0, scale, 1.0),
                         np.where(err == 0, 0.0, np.inf))
    ratio = np.where(finite, ratio, np.inf)
    return err, ratio


def assert_rows_close(A, Aref, scale, tol=TOL, what="A"):
    err, ratio = row_errors(A, Aref, scale)
    if ratio.size == 0:
        return 0.0
    worst = int(np.argmax(ratio))
    bad = np.nonzero(~(ratio <= tol))[0]
    assert bad.size == 0, (
        f"{what}: {bad.size} of {ratio.size} rows outside {tol:g}*scale; worst row {worst}: "
        f"err={err[worst]:.3e} scale={np.asarray(scale)[worst]:.3e} ratio={ratio[worst]:.3e}")
    return float(ratio.max())
