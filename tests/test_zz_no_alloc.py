"""The no-allocation fused entry point (sparselnr_fused_sddmm_spmm_noalloc),
called through the C ABI, against the allocating fused entry point and the
oracle: two calls in a row, the second on a smaller input, then a call whose
grid factor has to be lowered for the partial rows to fit the fixed array.
Same rule as tests/parity.py (per row, error <= 1e-4 * the abs-value scale);
where both entry points run the same grid the results must be bit-identical.
The call must leave the device's free memory unchanged."""
import ctypes

import numpy as np
import pytest

import oracle
import paper_2205_11622_amd as slnr
from tests.gpu_util import make_problem, power_law_lengths, upload
from tests.parity import assert_rows_close

pytestmark = pytest.mark.gpu


def noalloc(d, A, stream):
    """One call of the C entry point with raw device pointers."""
    lib = slnr.lib()
    N, K = d["C"].shape
    M, L = d["E"].shape
    ptr = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
    rc = lib.sparselnr_fused_sddmm_spmm_noalloc(
        ptr(d["rowptr"]), ptr(d["colidx"]), ptr(d["vals"]), ptr(d["C"]), ptr(d["D"]),
        ptr(d["E"]), ptr(A), N, M, K, L, ctypes.c_void_p(stream.cuda_stream))
    assert rc == slnr.OK, slnr.sparselnr_status_string(rc)


def check(p, d, stream, gpu, exact):
    import torch
    with torch.cuda.stream(stream):
        ref = slnr.sparselnr_fused_sddmm_spmm(d["rowptr"], d["colidx"], d["vals"], d["C"],
                                              d["D"], d["E"])
        A = torch.full((p.N, p.L), float("nan"), device=gpu)
    stream.synchronize()
    free0 = torch.cuda.mem_get_info(gpu)[0]
    noalloc(d, A, stream)
    stream.synchronize()
    assert torch.cuda.mem_get_info(gpu)[0] == free0, "the no-allocation call allocated"
    Aref, scale, _ = oracle.fused_rows(p.rowptr, p.colidx, p.vals, p.C, p.D, p.E)
    assert_rows_close(A.cpu().numpy(), Aref, scale, what="no-allocation call")
    assert_rows_close(ref.cpu().numpy(), Aref, scale, what="allocating call")
    if exact:
        assert torch.equal(A, ref), "same grid, yet the two entry points differ"
    return A


def test_noalloc_matches_the_fused_entry_point(gpu):
    import torch
    s = torch.cuda.Stream()
    # a large power-law input (several resident grids, 64-lane workers, rows
    # split over many workers), then a smaller one on the same array
    big = power_law_lengths(300_000, seed=41, cap=20_000)
    big[11] = 60_000
    p1 = make_problem(big, 200_000, 128, 128, seed=41, dense="normal")
    print("call 1: N=%d nnz=%d K=L=128" % (p1.N, p1.nnz), flush=True)
    check(p1, upload(p1), s, gpu, exact=True)
    small = power_law_lengths(20_000, seed=42, cap=3000)
    small[5] = 9000
    p2 = make_problem(small, 9_000, 64, 64, seed=42, dense="normal")
    print("call 2: N=%d nnz=%d K=L=64" % (p2.N, p2.nnz), flush=True)
    check(p2, upload(p2), s, gpu, exact=True)


def test_noalloc_lowers_the_grid_factor_to_fit(gpu):
    import torch
    s = torch.cuda.Stream()
    big = power_law_lengths(300_000, seed=43, cap=20_000)
    big[0] = 50_000
    p = make_problem(big, 150_000, 128, 128, seed=43, dense="normal")
    d = upload(p)
    print("factor 64: N=%d nnz=%d K=L=128" % (p.N, p.nnz), flush=True)
    try:
        # at 64 resident grids the partial rows would need more than the array
        slnr.sparselnr_set_grid_factor(64)
        check(p, d, s, gpu, exact=False)
    finally:
        slnr.sparselnr_set_grid_factor(0)
    # and the next call at the automatic factor reuses the array correctly
    small = power_law_lengths(5_000, seed=44, cap=2000)
    p2 = make_problem(small, 4_000, 32, 32, seed=44)
    print("then automatic: N=%d nnz=%d K=L=32" % (p2.N, p2.nnz), flush=True)
    check(p2, upload(p2), s, gpu, exact=True)
