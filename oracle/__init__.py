"""CPU oracle for the fused SDDMM->SpMM computation (fp64, plain loops).

TEST INFRASTRUCTURE ONLY.  Only the tests, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  The GPU library
never uses it: the two share no code, headers or helpers.

What it computes (oracle.c holds the loops):

* ``sddmm``      -- Figure 2a of the paper: Y[p] = b_p * sum_k C[i,k] D[j,k].
* ``spmm``       -- Figure 2b: A[i,:] = sum_p Y[p] E[j,:].
* ``fused_rows`` -- the result on chosen rows, each row computed as 2a then 2b
                    into a row-local value array, plus the per-row tolerance
                    scale  max_l sum_p |b_p| (sum_k |C_ik||D_jk|) |E_jl|.
* ``sddmm_spmm_gemm_rows``, ``spmm_gemm_rows``, ``spmmh_gemm_rows`` -- the
                    <SDDMM, SpMM, GEMM>, <SpMM, GEMM> and <SpMMH, GEMM>
                    benchmarks of Section 6.2 on chosen rows (row of the sparse
                    product, then times the dense matrix), with their scales.
* ``fused_rows_dt`` -- <SDDMM, SpMM> with D stored transposed (Section 4.3.1).

Pins that tie it to the paper and to mathematics (not to itself) are in
tests/test_oracle.py and tests/test_oracle_next.py: dense brute force
A = (B .* C D^T) E (and the products of the other benchmarks), the
perfect-nest form of Figure 2c, closed-form special cases, invariants and a
hand-worked golden example.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_SRC = os.path.join(_HERE, "oracle.c")

# -O2, no fast-math: sums are taken in the order written.
CFLAGS = ["-O2", "-fopenmp", "-fPIC", "-shared", "-Wall"]


def build(force: bool = False) -> str:
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", *CFLAGS, _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        L = ctypes.CDLL(_LIB_PATH)
        i64, vp = ctypes.c_int64, ctypes.c_void_p
        L.oracle_sddmm.restype = i64
        L.oracle_sddmm.argtypes = [i64, i64, i64, vp, vp, vp, vp, vp, vp, vp]
        L.oracle_spmm.restype = i64
        L.oracle_spmm.argtypes = [i64, i64, i64, vp, vp, vp, vp, vp, vp, vp]
        L.oracle_fused_rows.restype = i64
        L.oracle_fused_rows.argtypes = [i64, i64, i64, i64, vp, vp, vp, vp, vp, vp,
                                        vp, i64, vp, vp, vp, vp]
        L.oracle_num_threads.restype = ctypes.c_int
        _lib = L
    return _lib


def num_threads() -> int:
    return int(lib().oracle_num_threads())


def _c(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a


def _p(a):
    return None if a is None else a.ctypes.data


def _csr(rowptr, colidx, vals):
    return _c(rowptr, np.int32), _c(colidx, np.int32), _c(vals, np.float32)


def sddmm(rowptr, colidx, vals, C, D, with_scale: bool = False):
    """Figure 2a.  Returns Y (fp64, nnz), and its scale if asked, and the op count."""
    rowptr, colidx, vals = _csr(rowptr, colidx, vals)
    C, D = _c(C, np.float32), _c(D, np.float32)
    N, K = C.shape
    M = D.shape[0]
    nnz = int(rowptr[-1])
    Y = np.empty(nnz, dtype=np.float64)
    Ys = np.empty(nnz, dtype=np.float64) if with_scale else None
    ops = lib().oracle_sddmm(N, M, K, _p(rowptr), _p(colidx), _p(vals), _p(C), _p(D),
                             _p(Y), _p(Ys))
    return (Y, Ys, ops) if with_scale else (Y, ops)


def spmm(rowptr, colidx, Y, E, Yabs=None):
    """Figure 2b.  Returns A (fp64, N x L), the row scale if Yabs is given, and the op count."""
    rowptr, colidx = _c(rowptr, np.int32), _c(colidx, np.int32)
    Y = _c(Y, np.float64)
    E = _c(E, np.float32)
    N = rowptr.size - 1
    M, L = E.shape
    A = np.empty((N, L), dtype=np.float64)
    Yabs = None if Yabs is None else _c(Yabs, np.float64)
    As = np.empty(N, dtype=np.float64) if Yabs is not None else None
    ops = lib().oracle_spmm(N, M, L, _p(rowptr), _p(colidx), _p(Y), _p(E), _p(A),
                            _p(Yabs), _p(As))
    return (A, As, ops) if Yabs is not None else (A, ops)


def fused_rows(rowptr, colidx, vals, C, D, E, rows=None, with_y: bool = False):
    """Rows `rows` (default: all) of A in fp64, their tolerance scales, and the op count.

    With with_y=True also returns the rows' SDDMM values and scales (rows
    concatenated in list order)."""
    rowptr, colidx, vals = _csr(rowptr, colidx, vals)
    C, D, E = _c(C, np.float32), _c(D, np.float32), _c(E, np.float32)
    N, K = C.shape
    M, L = E.shape
    if rows is None:
        rows = np.arange(N, dtype=np.int64)
    rows = _c(rows, np.int64)
    A = np.empty((rows.size, L), dtype=np.float64)
    scale = np.empty(rows.size, dtype=np.float64)
    Y = Ys = None
    if with_y:
        ny = int((rowptr[rows + 1] - rowptr[rows]).sum()) if rows.size else 0
        Y = np.empty(ny, dtype=np.float64)
        Ys = np.empty(ny, dtype=np.float64)
    ops = lib().oracle_fused_rows(N, M, K, L, _p(rowptr), _p(colidx), _p(vals), _p(C), _p(D),
                                  _p(E), _p(rows), rows.size, _p(A), _p(scale), _p(Y), _p(Ys))
    if with_y:
        return A, scale, Y, Ys, ops
    return A, scale, ops


# ---------------------------------------------------------------- next rows

def _rows(rows, N):
    if rows is None:
        rows = np.arange(N, dtype=np.int64)
    return _c(rows, np.int64)


def _setup_next():
    L = lib()
    i64, vp = ctypes.c_int64, ctypes.c_void_p
    if not hasattr(L, "_next_ready"):
        L.oracle_sddmm_spmm_gemm_rows.restype = i64
        L.oracle_sddmm_spmm_gemm_rows.argtypes = [i64, i64, i64] + [vp] * 7 + [vp, i64, vp, vp]
        L.oracle_spmm_gemm_rows.restype = i64
        L.oracle_spmm_gemm_rows.argtypes = [i64, i64] + [vp] * 5 + [vp, i64, vp, vp]
        L.oracle_spmmh_gemm_rows.restype = i64
        L.oracle_spmmh_gemm_rows.argtypes = [i64, i64] + [vp] * 6 + [vp, i64, vp, vp]
        L.oracle_fused_rows_dt.restype = i64
        L.oracle_fused_rows_dt.argtypes = [i64, i64, i64] + [vp] * 6 + [vp, i64, vp, vp]
        L._next_ready = True
    return L


def sddmm_spmm_gemm_rows(rowptr, colidx, vals, C, D, F, W, rows=None):
    """<SDDMM, SpMM, GEMM> (Section 6.2): A = ((B .* C D^T) F) W on the chosen
    rows, in the fused loop order (row of <SDDMM, SpMM>, then times W)."""
    rowptr, colidx, vals = _csr(rowptr, colidx, vals)
    C, D, F, W = (_c(x, np.float32) for x in (C, D, F, W))
    N, K = C.shape
    L, Mo = W.shape
    assert F.shape[1] == L and D.shape[1] == K
    rows = _rows(rows, N)
    out = np.empty((rows.size, Mo), np.float64)
    scale = np.empty(rows.size, np.float64)
    ops = _setup_next().oracle_sddmm_spmm_gemm_rows(K, L, Mo, _p(rowptr), _p(colidx), _p(vals),
                                                   _p(C), _p(D), _p(F), _p(W), _p(rows),
                                                   rows.size, _p(out), _p(scale))
    return out, scale, ops


def spmm_gemm_rows(rowptr, colidx, vals, C, D, rows=None):
    """<SpMM, GEMM> (Section 6.2): A = (B C) D on the chosen rows; C is M x K,
    D is K x L."""
    rowptr, colidx, vals = _csr(rowptr, colidx, vals)
    C, D = _c(C, np.float32), _c(D, np.float32)
    K, L = D.shape
    assert C.shape[1] == K
    N = rowptr.size - 1
    rows = _rows(rows, N)
    out = np.empty((rows.size, L), np.float64)
    scale = np.empty(rows.size, np.float64)
    ops = _setup_next().oracle_spmm_gemm_rows(K, L, _p(rowptr), _p(colidx), _p(vals), _p(C),
                                              _p(D), _p(rows), rows.size, _p(out), _p(scale))
    return out, scale, ops


def spmmh_gemm_rows(rowptr, colidx, vals, C, D, E, rows=None):
    """<SpMMH, GEMM> (Section 6.2): A = (B (C .* D)) E on the chosen rows;
    C, D are M x J, E is J x L."""
    rowptr, colidx, vals = _csr(rowptr, colidx, vals)
    C, D, E = (_c(x, np.float32) for x in (C, D, E))
    J, L = E.shape
    assert C.shape[1] == J and D.shape == C.shape
    N = rowptr.size - 1
    rows = _rows(rows, N)
    out = np.empty((rows.size, L), np.float64)
    scale = np.empty(rows.size, np.float64)
    ops = _setup_next().oracle_spmmh_gemm_rows(J, L, _p(rowptr), _p(colidx), _p(vals), _p(C),
                                               _p(D), _p(E), _p(rows), rows.size, _p(out),
                                               _p(scale))
    return out, scale, ops


def fused_rows_dt(rowptr, colidx, vals, C, Dt, E, rows=None):
    """<SDDMM, SpMM> with D stored transposed (Dt is K x M; Section 4.3.1)."""
    rowptr, colidx, vals = _csr(rowptr, colidx, vals)
    C, Dt, E = (_c(x, np.float32) for x in (C, Dt, E))
    N, K = C.shape
    M, L = E.shape
    assert Dt.shape == (K, M)
    rows = _rows(rows, N)
    out = np.empty((rows.size, L), np.float64)
    scale = np.empty(rows.size, np.float64)
    ops = _setup_next().oracle_fused_rows_dt(M, K, L, _p(rowptr), _p(colidx), _p(vals), _p(C),
                                             _p(Dt), _p(E), _p(rows), rows.size, _p(out),
                                             _p(scale))
    return out, scale, ops
