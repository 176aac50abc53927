"""MI355X (gfx950) fused SDDMM->SpMM: Python binding of libsparselnr.so.

The binding only marshals arguments: it checks tensor devices, dtypes and
shapes, passes raw device pointers and the stream to the C ABI declared in
include/sparselnr.h, and raises on a non-zero status.  Every step of the
computation runs in the library's HIP kernels; there is no fallback.

    A = sparselnr_fused_sddmm_spmm(rowptr, colidx, vals, C, D, E)

computes A(i,l) = sum_{j,k} B(i,j) C(i,k) D(j,k) E(j,l) for B in CSR form
(rowptr int32[N+1], colidx int32[nnz], vals float32[nnz]) and dense
row-major float32 C (N x K), D (M x K), E (M x L).
"""
from __future__ import annotations

import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libsparselnr.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_HIP, ERR_NO_MEMORY, ERR_INVALID_CSR = range(6)

__all__ = [
    "sparselnr_fused_sddmm_spmm", "sparselnr_fused_sddmm_spmm_noalloc",
    "sparselnr_unfused_sddmm_spmm", "sparselnr_sddmm",
    "sparselnr_spmm", "sparselnr_fused_sddmm_spmm_gemm", "sparselnr_spmm_gemm",
    "sparselnr_spmmh_gemm", "sparselnr_fused_sddmm_spmm_dt", "sparselnr_validate_csr", "sparselnr_release", "sparselnr_status_string",
    "sparselnr_last_hip_error", "sparselnr_abi_version", "sparselnr_set_grid_factor",
    "sparselnr_get_grid_factor", "SparseLNRError", "lib", "LIB_PATH",
]


class SparseLNRError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = lib().sparselnr_status_string(status).decode()
        if status == ERR_HIP:
            msg += " (hipError_t %d)" % lib().sparselnr_last_hip_error()
        super().__init__("%s: %s [status %d]" % (where, msg, status))


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded C library (built in place by __graft_entry__.build())."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libsparselnr.so is not built (%s); run `python -c "
                              "'import __graft_entry__ as g; g.build()'`" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        vp, i64, ci = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
        L.sparselnr_fused_sddmm_spmm.argtypes = [vp] * 7 + [i64] * 4 + [vp]
        L.sparselnr_fused_sddmm_spmm.restype = ci
        L.sparselnr_fused_sddmm_spmm_noalloc.argtypes = [vp] * 7 + [i64] * 4 + [vp]
        L.sparselnr_fused_sddmm_spmm_noalloc.restype = ci
        L.sparselnr_unfused_sddmm_spmm.argtypes = [vp] * 8 + [i64] * 4 + [vp]
        L.sparselnr_unfused_sddmm_spmm.restype = ci
        L.sparselnr_sddmm.argtypes = [vp] * 6 + [i64] * 3 + [vp]
        L.sparselnr_sddmm.restype = ci
        L.sparselnr_spmm.argtypes = [vp] * 5 + [i64] * 3 + [vp]
        L.sparselnr_spmm.restype = ci
        L.sparselnr_fused_sddmm_spmm_gemm.argtypes = [vp] * 8 + [i64] * 5 + [vp]
        L.sparselnr_fused_sddmm_spmm_gemm.restype = ci
        L.sparselnr_spmm_gemm.argtypes = [vp] * 6 + [i64] * 4 + [vp]
        L.sparselnr_spmm_gemm.restype = ci
        L.sparselnr_spmmh_gemm.argtypes = [vp] * 7 + [i64] * 4 + [vp]
        L.sparselnr_spmmh_gemm.restype = ci
        L.sparselnr_fused_sddmm_spmm_dt.argtypes = [vp] * 7 + [i64] * 4 + [vp]
        L.sparselnr_fused_sddmm_spmm_dt.restype = ci
        L.sparselnr_validate_csr.argtypes = [vp, vp, i64, i64, i64, ctypes.POINTER(i64), vp]
        L.sparselnr_validate_csr.restype = ci
        L.sparselnr_status_string.argtypes = [ci]
        L.sparselnr_status_string.restype = ctypes.c_char_p
        L.sparselnr_last_hip_error.argtypes = []
        L.sparselnr_last_hip_error.restype = ci
        L.sparselnr_release.argtypes = []
        L.sparselnr_release.restype = ci
        L.sparselnr_abi_version.argtypes = []
        L.sparselnr_abi_version.restype = ci
        L.sparselnr_set_grid_factor.argtypes = [ci]
        L.sparselnr_set_grid_factor.restype = ci
        L.sparselnr_get_grid_factor.argtypes = []
        L.sparselnr_get_grid_factor.restype = ci
        _lib = L
    return _lib


def sparselnr_abi_version() -> int:
    return int(lib().sparselnr_abi_version())


def sparselnr_status_string(status: int) -> str:
    return lib().sparselnr_status_string(status).decode()


def sparselnr_last_hip_error() -> int:
    return int(lib().sparselnr_last_hip_error())


def sparselnr_set_grid_factor(factor: int) -> None:
    """Resident grids per walk launch: 0 automatic, 1..64 fixed (process-wide)."""
    rc = lib().sparselnr_set_grid_factor(int(factor))
    if rc != OK:
        raise SparseLNRError(rc, "sparselnr_set_grid_factor")


def sparselnr_get_grid_factor() -> int:
    return int(lib().sparselnr_get_grid_factor())


def sparselnr_release() -> None:
    rc = lib().sparselnr_release()
    if rc != OK:
        raise SparseLNRError(rc, "sparselnr_release")


# ------------------------------------------------------------ marshalling

def _torch():
    import torch
    return torch


def _check(t, name, dtype, device, ndim=None):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if t.device != device:
        raise ValueError("%s is on %s, expected %s" % (name, t.device, device))
    if t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if ndim is not None and t.dim() != ndim:
        raise ValueError("%s must have %d dimensions" % (name, ndim))


_dummy = {}


def _ptr(t, device):
    """Device address of t; a 16-byte dummy allocation when t is empty, so that
    the library never sees NULL for an empty array."""
    if t.numel() > 0:
        return t.data_ptr()
    torch = _torch()
    d = _dummy.get(device)
    if d is None:
        d = _dummy[device] = torch.zeros(4, dtype=torch.float32, device=device)
    return d.data_ptr()


def _stream(stream, device):
    if stream is None:
        return _torch().cuda.current_stream(device).cuda_stream
    return getattr(stream, "cuda_stream", stream)


def _csr(rowptr, colidx, vals, vals_name="vals"):
    torch = _torch()
    device = rowptr.device
    if device.type != "cuda":
        raise ValueError("inputs must be on a GPU device")
    _check(rowptr, "rowptr", torch.int32, device, 1)
    _check(colidx, "colidx", torch.int32, device, 1)
    _check(vals, vals_name, torch.float32, device, 1)
    if rowptr.numel() < 1:
        raise ValueError("rowptr needs N+1 >= 1 entries")
    if colidx.numel() != vals.numel():
        raise ValueError("colidx and %s differ in length" % vals_name)
    return device, rowptr.numel() - 1


def _dense(t, name, rows, device):
    torch = _torch()
    _check(t, name, torch.float32, device, 2)
    if t.shape[0] != rows:
        raise ValueError("%s has %d rows, expected %d" % (name, t.shape[0], rows))
    return t.shape[1]


def sparselnr_fused_sddmm_spmm(rowptr, colidx, vals, C, D, E, A=None, stream=None):
    """Fused SDDMM->SpMM (the paper's Figure 2d schedule).  Returns A (N x L).

    A, if given, is overwritten.  Asynchronous on `stream` (default: the
    current torch stream of the inputs' device)."""
    torch = _torch()
    device, N = _csr(rowptr, colidx, vals)
    K = _dense(C, "C", N, device)
    M = D.shape[0] if isinstance(D, torch.Tensor) and D.dim() == 2 else -1
    if _dense(D, "D", M, device) != K:
        raise ValueError("C and D differ in width K")
    L = _dense(E, "E", M, device)
    if A is None:
        A = torch.empty((N, L), dtype=torch.float32, device=device)
    elif _dense(A, "A", N, device) != L:
        raise ValueError("A must be N x L")
    rc = lib().sparselnr_fused_sddmm_spmm(
        _ptr(rowptr, device), _ptr(colidx, device), _ptr(vals, device), _ptr(C, device),
        _ptr(D, device), _ptr(E, device), _ptr(A, device), N, M, K, L, _stream(stream, device))
    if rc != OK:
        raise SparseLNRError(rc, "sparselnr_fused_sddmm_spmm")
    return A


def sparselnr_fused_sddmm_spmm_noalloc(rowptr, colidx, vals, C, D, E, A, stream=None):
    """The fused call for callers that cannot allocate: A (N x L) must be
    given; the library uses a fixed device array for split rows.  Calls that
    overlap on one GPU race (see include/sparselnr.h)."""
    torch = _torch()
    device, N = _csr(rowptr, colidx, vals)
    K = _dense(C, "C", N, device)
    M = D.shape[0] if isinstance(D, torch.Tensor) and D.dim() == 2 else -1
    if _dense(D, "D", M, device) != K:
        raise ValueError("C and D differ in width K")
    L = _dense(E, "E", M, device)
    if A is None or _dense(A, "A", N, device) != L:
        raise ValueError("A must be given, N x L")
    rc = lib().sparselnr_fused_sddmm_spmm_noalloc(
        _ptr(rowptr, device), _ptr(colidx, device), _ptr(vals, device), _ptr(C, device),
        _ptr(D, device), _ptr(E, device), _ptr(A, device), N, M, K, L, _stream(stream, device))
    if rc != OK:
        raise SparseLNRError(rc, "sparselnr_fused_sddmm_spmm_noalloc")
    return A


def sparselnr_sddmm(rowptr, colidx, vals, C, D, Y=None, stream=None):
    """SDDMM (Figure 2a): Y[p] = vals[p] * dot(C[i], D[colidx[p]]).  Returns Y."""
    torch = _torch()
    device, N = _csr(rowptr, colidx, vals)
    K = _dense(C, "C", N, device)
    M = D.shape[0] if isinstance(D, torch.Tensor) and D.dim() == 2 else -1
    if _dense(D, "D", M, device) != K:
        raise ValueError("C and D differ in width K")
    if Y is None:
        Y = torch.empty(colidx.numel(), dtype=torch.float32, device=device)
    else:
        _check(Y, "Y", torch.float32, device, 1)
        if Y.numel() != colidx.numel():
            raise ValueError("Y must have nnz entries")
    rc = lib().sparselnr_sddmm(_ptr(rowptr, device), _ptr(colidx, device), _ptr(vals, device),
                               _ptr(C, device), _ptr(D, device), _ptr(Y, device), N, M, K,
                               _stream(stream, device))
    if rc != OK:
        raise SparseLNRError(rc, "sparselnr_sddmm")
    return Y


def sparselnr_spmm(rowptr, colidx, Y, E, A=None, stream=None):
    """SpMM (Figure 2b): A[i] = sum_p Y[p] * E[colidx[p]].  Returns A."""
    torch = _torch()
    device, N = _csr(rowptr, colidx, Y, "Y")
    M = E.shape[0] if isinstance(E, torch.Tensor) and E.dim() == 2 else -1
    L = _dense(E, "E", M, device)
    if A is None:
        A = torch.empty((N, L), dtype=torch.float32, device=device)
    elif _dense(A, "A", N, device) != L:
        raise ValueError("A must be N x L")
    rc = lib().sparselnr_spmm(_ptr(rowptr, device), _ptr(colidx, device), _ptr(Y, device),
                              _ptr(E, device), _ptr(A, device), N, M, L, _stream(stream, device))
    if rc != OK:
        raise SparseLNRError(rc, "sparselnr_spmm")
    return A


def sparselnr_unfused_sddmm_spmm(rowptr, colidx, vals, C, D, E, Y=None, A=None, stream=None):
    """Unfused comparison (Figure 2a then 2b) through an nnz-sized Y.  Returns (Y, A)."""
    torch = _torch()
    device, N = _csr(rowptr, colidx, vals)
    K = _dense(C, "C", N, device)
    M = D.shape[0] if isinstance(D, torch.Tensor) and D.dim() == 2 else -1
    if _dense(D, "D", M, device) != K:
        raise ValueError("C and D differ in width K")
    L = _dense(E, "E", M, device)
    if Y is None:
        Y = torch.empty(colidx.numel(), dtype=torch.float32, device=device)
    else:
        _check(Y, "Y", torch.float32, device, 1)
        if Y.numel() != colidx.numel():
            raise ValueError("Y must have nnz entries")
    if A is None:
        A = torch.empty((N, L), dtype=torch.float32, device=device)
    elif _dense(A, "A", N, device) != L:
        raise ValueError("A must be N x L")
    rc = lib().sparselnr_unfused_sddmm_spmm(
        _ptr(rowptr, device), _ptr(colidx, device), _ptr(vals, device), _ptr(C, device),
        _ptr(D, device), _ptr(E, device), _ptr(Y, device), _ptr(A, device), N, M, K, L,
        _stream(stream, device))
    if rc != OK:
        raise SparseLNRError(rc, "sparselnr_unfused_sddmm_spmm")
    return Y, A


def _out(A, rows, cols, device, name="A"):
    torch = _torch()
    if A is None:
        return torch.empty((rows, cols), dtype=torch.float32, device=device)
    if _dense(A, name, rows, device) != cols:
        raise ValueError("%s must be %d x %d" % (name, rows, cols))
    return A


def sparselnr_fused_sddmm_spmm_gemm(rowptr, colidx, vals, C, D, F, W, A=None, stream=None):
    """<SDDMM, SpMM, GEMM>: A = ((B .* C D^T) F) W, one pass (Section 6.2).
    C: N x K, D: M x K, F: M x L, W: L x Mo.  Returns A (N x Mo)."""
    torch = _torch()
    device, N = _csr(rowptr, colidx, vals)
    K = _dense(C, "C", N, device)
    M = D.shape[0] if isinstance(D, torch.Tensor) and D.dim() == 2 else -1
    if _dense(D, "D", M, device) != K:
        raise ValueError("C and D differ in width K")
    L = _dense(F, "F", M, device)
    Mo = _dense(W, "W", L, device)
    A = _out(A, N, Mo, device)
    rc = lib().sparselnr_fused_sddmm_spmm_gemm(
        _ptr(rowptr, device), _ptr(colidx, device), _ptr(vals, device), _ptr(C, device),
        _ptr(D, device), _ptr(F, device), _ptr(W, device), _ptr(A, device), N, M, K, L, Mo,
        _stream(stream, device))
    if rc != OK:
        raise SparseLNRError(rc, "sparselnr_fused_sddmm_spmm_gemm")
    return A


def sparselnr_spmm_gemm(rowptr, colidx, vals, C, D, A=None, stream=None):
    """<SpMM, GEMM>: A = (B C) D (Section 6.2).  C: M x K, D: K x L.  Returns A (N x L)."""
    torch = _torch()
    device, N = _csr(rowptr, colidx, vals)
    M = C.shape[0] if isinstance(C, torch.Tensor) and C.dim() == 2 else -1
    K = _dense(C, "C", M, device)
    L = _dense(D, "D", K, device)
    A = _out(A, N, L, device)
    rc = lib().sparselnr_spmm_gemm(_ptr(rowptr, device), _ptr(colidx, device),
                                   _ptr(vals, device), _ptr(C, device), _ptr(D, device),
                                   _ptr(A, device), N, M, K, L, _stream(stream, device))
    if rc != OK:
        raise SparseLNRError(rc, "sparselnr_spmm_gemm")
    return A


def sparselnr_spmmh_gemm(rowptr, colidx, vals, C, D, E, A=None, stream=None):
    """<SpMMH, GEMM>: A = (B (C .* D)) E (Section 6.2).  C, D: M x J, E: J x L."""
    torch = _torch()
    device, N = _csr(rowptr, colidx, vals)
    M = C.shape[0] if isinstance(C, torch.Tensor) and C.dim() == 2 else -1
    J = _dense(C, "C", M, device)
    if _dense(D, "D", M, device) != J:
        raise ValueError("C and D must have the same shape")
    L = _dense(E, "E", J, device)
    A = _out(A, N, L, device)
    rc = lib().sparselnr_spmmh_gemm(_ptr(rowptr, device), _ptr(colidx, device),
                                    _ptr(vals, device), _ptr(C, device), _ptr(D, device),
                                    _ptr(E, device), _ptr(A, device), N, M, J, L,
                                    _stream(stream, device))
    if rc != OK:
        raise SparseLNRError(rc, "sparselnr_spmmh_gemm")
    return A


def sparselnr_fused_sddmm_spmm_dt(rowptr, colidx, vals, C, Dt, E, A=None, stream=None):
    """<SDDMM, SpMM> with D stored transposed (Dt: K x M, Section 4.3.1)."""
    torch = _torch()
    device, N = _csr(rowptr, colidx, vals)
    K = _dense(C, "C", N, device)
    M = E.shape[0] if isinstance(E, torch.Tensor) and E.dim() == 2 else -1
    if _dense(Dt, "Dt", K, device) != M:
        raise ValueError("Dt must be K x M")
    L = _dense(E, "E", M, device)
    A = _out(A, N, L, device)
    rc = lib().sparselnr_fused_sddmm_spmm_dt(
        _ptr(rowptr, device), _ptr(colidx, device), _ptr(vals, device), _ptr(C, device),
        _ptr(Dt, device), _ptr(E, device), _ptr(A, device), N, M, K, L, _stream(stream, device))
    if rc != OK:
        raise SparseLNRError(rc, "sparselnr_fused_sddmm_spmm_dt")
    return A


def sparselnr_validate_csr(rowptr, colidx, M, stream=None) -> int:
    """Checks the CSR preconditions on the device (synchronous).  Returns nnz;
    raises SparseLNRError(ERR_INVALID_CSR) on a violation."""
    torch = _torch()
    device = rowptr.device
    _check(rowptr, "rowptr", torch.int32, device, 1)
    _check(colidx, "colidx", torch.int32, device, 1)
    nnz = ctypes.c_int64(-1)
    rc = lib().sparselnr_validate_csr(_ptr(rowptr, device), _ptr(colidx, device),
                                      rowptr.numel() - 1, M, colidx.numel(), ctypes.byref(nnz),
                                      _stream(stream, device))
    if rc != OK:
        raise SparseLNRError(rc, "sparselnr_validate_csr")
    return int(nnz.value)
