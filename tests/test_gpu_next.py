"""GPU parity for the further computations built on the same hot path: the
<SDDMM, SpMM, GEMM>, <SpMM, GEMM> and <SpMMH, GEMM> benchmarks of the paper's
Section 6.2 (sparse row product, then a per-row dense product in the same
pass) and <SDDMM, SpMM> with D stored transposed (Section 4.3.1).  Same rule
as tests/parity.py: per row, max error <= 1e-4 * the abs-value scale."""
import numpy as np
import pytest

import oracle
import paper_2205_11622_amd as slnr
import synth
from tests.gpu_util import make_problem, oracle_reference, power_law_lengths, rows_close_dev
from tests.parity import assert_rows_close

pytestmark = pytest.mark.gpu


def dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda:0")


def csr(p):
    return dev(p.rowptr), dev(p.colidx), dev(p.vals)


def rows_of(A, rows):
    import torch
    if rows is None:
        return A.cpu().numpy()
    return A[torch.from_numpy(rows).to(A.device)].cpu().numpy()


def lengths(seed):
    n = power_law_lengths(2501, seed=seed, cap=5000)
    n[3] = 7000
    return n


@pytest.mark.parametrize("L,Mo", [(32, 32), (32, 16), (64, 64), (64, 32), (128, 128), (128, 64),
                                  (16, 48), (256, 100), (512, 64), (64, 1),
                                  # dense matrix staged in LDS with blocks above 64 KB of LDS
                                  (64, 128), (64, 256), (32, 512), (16, 1024), (64, 257)])
def test_sddmm_spmm_gemm(gpu, L, Mo):
    p = make_problem(lengths(L + Mo), 2000, L, L, seed=L, dense="normal")
    W = synth.normal(5, 9, (L, Mo))
    A = slnr.sparselnr_fused_sddmm_spmm_gemm(*csr(p), dev(p.C), dev(p.D), dev(p.E), dev(W))
    ref, scale, _ = oracle.sddmm_spmm_gemm_rows(p.rowptr, p.colidx, p.vals, p.C, p.D, p.E, W)
    assert_rows_close(rows_of(A, None), ref, scale)


@pytest.mark.parametrize("K,L", [(32, 32), (32, 16), (64, 64), (64, 32), (128, 128), (128, 64),
                                 (16, 16), (256, 512), (512, 7), (128, 200)])
def test_spmm_gemm(gpu, K, L):
    p = make_problem(lengths(K + 2 * L), 1800, K, K, seed=K + L, dense="normal")
    C = p.D                               # M x K rows gathered by the SpMM
    Dk = synth.normal(3, 9, (K, L))       # K x L dense factor
    A = slnr.sparselnr_spmm_gemm(*csr(p), dev(C), dev(Dk))
    ref, scale, _ = oracle.spmm_gemm_rows(p.rowptr, p.colidx, p.vals, C, Dk)
    assert_rows_close(rows_of(A, None), ref, scale)


@pytest.mark.parametrize("J,L", [(32, 32), (32, 16), (64, 64), (64, 32), (128, 128), (128, 64),
                                 (16, 3), (256, 256), (512, 128)])
def test_spmmh_gemm(gpu, J, L):
    p = make_problem(lengths(J + 3 * L), 1700, J, J, seed=J * L, dense="normal")
    C, D = p.D, p.E                       # M x J each
    E = synth.normal(4, 9, (J, L))
    A = slnr.sparselnr_spmmh_gemm(*csr(p), dev(C), dev(D), dev(E))
    ref, scale, _ = oracle.spmmh_gemm_rows(p.rowptr, p.colidx, p.vals, C, D, E)
    assert_rows_close(rows_of(A, None), ref, scale)


@pytest.mark.parametrize("J,L", [(16, 3), (32, 32), (64, 17), (128, 128), (256, 64),
                                 (512, 128)])
def test_spmmh_gemm_per_nonzero_schedule(gpu, J, L):
    """Fewer than 3 nonzeros per column of B (nnz < 3 M): the library forms
    C_k .* D_k per nonzero from two gathered rows instead of forming C .* D
    once."""
    n = power_law_lengths(3000, seed=J + L, scale=1.0, cap=60)
    M = max(3000, int(n.sum()) // 3 + 1)
    p = make_problem(n, M, J, J, seed=J + 5 * L, dense="normal")
    assert p.nnz < 3 * M
    C, D = p.D, p.E
    E = synth.normal(7, 9, (J, L))
    A = slnr.sparselnr_spmmh_gemm(*csr(p), dev(C), dev(D), dev(E))
    ref, scale, _ = oracle.spmmh_gemm_rows(p.rowptr, p.colidx, p.vals, C, D, E)
    assert_rows_close(rows_of(A, None), ref, scale)


@pytest.mark.parametrize("J", [16, 128, 512])
def test_spmmh_gemm_schedules_agree_bitwise(gpu, J):
    """The two schedules of <SpMMH, GEMM> (C .* D formed once when nnz >= 3 M,
    per nonzero otherwise) round the same products in the same order, so
    padding C and D with unused rows (which moves nnz below 3 M and switches
    the schedule) must not change a bit of A."""
    import torch
    p = make_problem(lengths(J), 1500, J, J, seed=3 * J, dense="normal")
    assert p.nnz >= 3 * p.M
    C, D = p.D, p.E
    E = dev(synth.normal(8, 9, (J, 96)))
    A1 = slnr.sparselnr_spmmh_gemm(*csr(p), dev(C), dev(D), E).clone()
    pad = p.nnz // 3 + 1 - p.M
    Cp = np.vstack([C, synth.normal(9, 9, (pad, J))])
    Dp = np.vstack([D, synth.normal(9, 10, (pad, J))])
    assert p.nnz < 3 * Cp.shape[0]
    A2 = slnr.sparselnr_spmmh_gemm(*csr(p), dev(Cp), dev(Dp), E)
    assert torch.equal(A1.view(torch.int32), A2.view(torch.int32))


def test_spmmh_gemm_schedule_threshold(gpu):
    """nnz exactly 3 M takes the formed-once schedule, 3 M - 1 the other;
    both match the oracle."""
    J, M = 64, 400
    for nnz in (3 * M, 3 * M - 1):
        n = np.full(nnz // 3, 3, np.int64)
        n[: nnz - n.sum()] += 1
        p = make_problem(n, M, J, J, seed=nnz, dense="normal")
        assert p.nnz == nnz
        E = synth.normal(2, 9, (J, 40))
        A = slnr.sparselnr_spmmh_gemm(*csr(p), dev(p.D), dev(p.E), dev(E))
        ref, scale, _ = oracle.spmmh_gemm_rows(p.rowptr, p.colidx, p.vals, p.D, p.E, E)
        assert_rows_close(rows_of(A, None), ref, scale)


@pytest.mark.parametrize("K,L", [(32, 32), (128, 128), (16, 256), (3, 5), (64, 64)])
def test_transposed_D(gpu, K, L):
    p = make_problem(lengths(K + L), 2200, K, L, seed=K + 7 * L, dense="normal")
    Dt = np.ascontiguousarray(p.D.T)      # K x M
    A = slnr.sparselnr_fused_sddmm_spmm_dt(*csr(p), dev(p.C), dev(Dt), dev(p.E))
    ref, scale, _ = oracle.fused_rows_dt(p.rowptr, p.colidx, p.vals, p.C, Dt, p.E)
    assert_rows_close(rows_of(A, None), ref, scale)
    # the same numbers as the plain layout (same kernel after the transpose)
    A0 = slnr.sparselnr_fused_sddmm_spmm(*csr(p), dev(p.C), dev(p.D), dev(p.E))
    import torch
    assert torch.equal(A, A0)


def test_next_empty_and_zero_rows(gpu):
    import torch
    p = make_problem(np.zeros(700, np.int64), 50, 64, 64)
    rp, ci, v = csr(p)
    A = torch.full((p.N, 32), float("nan"), device="cuda:0")
    slnr.sparselnr_spmm_gemm(rp, ci, v, dev(p.D), dev(synth.normal(1, 1, (64, 32))), A)
    assert bool((A == 0).all())
    A = torch.full((p.N, 64), float("nan"), device="cuda:0")
    slnr.sparselnr_fused_sddmm_spmm_gemm(rp, ci, v, dev(p.C), dev(p.D), dev(p.E),
                                         dev(synth.normal(1, 2, (64, 64))), A)
    assert bool((A == 0).all())


def test_next_deterministic(gpu):
    import torch
    p = make_problem(lengths(99), 1500, 128, 128, seed=99)
    W = dev(synth.normal(2, 2, (128, 128)))
    args = (*csr(p), dev(p.D), dev(p.E), W)
    A1 = slnr.sparselnr_spmmh_gemm(*args).clone()
    A2 = slnr.sparselnr_spmmh_gemm(*args)
    assert torch.equal(A1.view(torch.int32), A2.view(torch.int32))


@pytest.mark.parametrize("factor", [1, 5, 64])
def test_next_grid_factors(gpu, factor):
    # every entry point here at grid factors the benchmark may choose
    # (sparselnr_set_grid_factor), down to mostly empty slices at 64
    p = make_problem(lengths(17), 2400, 64, 64, seed=17, dense="normal")
    W = synth.normal(5, 3, (64, 32))
    Dk = synth.normal(3, 3, (64, 40))
    E3 = synth.normal(4, 3, (64, 48))
    Dt = np.ascontiguousarray(p.D.T)
    try:
        slnr.sparselnr_set_grid_factor(factor)
        A = slnr.sparselnr_fused_sddmm_spmm_gemm(*csr(p), dev(p.C), dev(p.D), dev(p.E), dev(W))
        ref, scale, _ = oracle.sddmm_spmm_gemm_rows(p.rowptr, p.colidx, p.vals, p.C, p.D, p.E, W)
        assert_rows_close(rows_of(A, None), ref, scale, what="sddmm_spmm_gemm")
        A = slnr.sparselnr_spmm_gemm(*csr(p), dev(p.D), dev(Dk))
        ref, scale, _ = oracle.spmm_gemm_rows(p.rowptr, p.colidx, p.vals, p.D, Dk)
        assert_rows_close(rows_of(A, None), ref, scale, what="spmm_gemm")
        A = slnr.sparselnr_spmmh_gemm(*csr(p), dev(p.D), dev(p.E), dev(E3))
        ref, scale, _ = oracle.spmmh_gemm_rows(p.rowptr, p.colidx, p.vals, p.D, p.E, E3)
        assert_rows_close(rows_of(A, None), ref, scale, what="spmmh_gemm")
        A = slnr.sparselnr_fused_sddmm_spmm_dt(*csr(p), dev(p.C), dev(Dt), dev(p.E))
        ref, scale, _ = oracle.fused_rows_dt(p.rowptr, p.colidx, p.vals, p.C, Dt, p.E)
        assert_rows_close(rows_of(A, None), ref, scale, what="fused, D transposed")
    finally:
        slnr.sparselnr_set_grid_factor(0)


@pytest.mark.slow
@pytest.mark.parametrize("kernel", ["sddmm_spmm_gemm", "spmm_gemm", "spmmh_gemm", "dt"])
def test_next_on_rmat1m(gpu, kernel):
    """The R-MAT 2^20 structure at the inner sizes the paper uses for each
    benchmark (K=L=M=64; K=128, L=64; J=L=128; D transposed at K=L=128):
    every row, at every grid factor the benchmark may time and at the
    automatic one.  The output is NaN-filled before each call, so a row left
    unwritten fails."""
    import torch

    import bench
    base = synth.config("rmat1m")
    rp, ci, v = csr(base)
    r3 = (base.rowptr, base.colidx, base.vals)
    if kernel == "sddmm_spmm_gemm":
        C, D, F = (synth.normal(0, s, (base.N, 64)) for s in (3, 4, 5))
        W = synth.normal(0, 6, (64, 64))
        args = (rp, ci, v, dev(C), dev(D), dev(F), dev(W))
        call = slnr.sparselnr_fused_sddmm_spmm_gemm
        fn = lambda rows: oracle.sddmm_spmm_gemm_rows(*r3, C, D, F, W, rows=rows)  # noqa: E731
        width = 64
    elif kernel == "spmm_gemm":
        C, Dk = synth.normal(0, 4, (base.N, 128)), synth.normal(0, 6, (128, 64))
        args = (rp, ci, v, dev(C), dev(Dk))
        call = slnr.sparselnr_spmm_gemm
        fn = lambda rows: oracle.spmm_gemm_rows(*r3, C, Dk, rows=rows)  # noqa: E731
        width = 64
    elif kernel == "spmmh_gemm":
        C, D = synth.normal(0, 4, (base.N, 128)), synth.normal(0, 5, (base.N, 128))
        E = synth.normal(0, 6, (128, 128))
        args = (rp, ci, v, dev(C), dev(D), dev(E))
        call = slnr.sparselnr_spmmh_gemm
        fn = lambda rows: oracle.spmmh_gemm_rows(*r3, C, D, E, rows=rows)  # noqa: E731
        width = 128
    else:
        Dt = np.ascontiguousarray(base.D.T)
        args = (rp, ci, v, dev(base.C), dev(Dt), dev(base.E))
        call = slnr.sparselnr_fused_sddmm_spmm_dt
        fn = lambda rows: oracle.fused_rows_dt(*r3, base.C, Dt, base.E, rows=rows)  # noqa: E731
        width = base.L
    print("rmat1m %s: N=%d nnz=%d" % (kernel, base.N, base.nnz), flush=True)
    ref, scale = oracle_reference(fn, base.N, width, gpu)
    A = torch.empty((base.N, width), dtype=torch.float32, device=gpu)
    try:
        for f in (0,) + tuple(bench.GRID_FACTORS):
            slnr.sparselnr_set_grid_factor(f)
            what = "%s, grid factor %s" % (kernel, f or "automatic")
            A.fill_(float("nan"))
            call(*args, A=A)
            w = rows_close_dev(A, ref, scale, what=what)
            print("  %s: worst err/scale %.2e" % (what, w), flush=True)
    finally:
        slnr.sparselnr_set_grid_factor(0)
    del A, ref, scale
    torch.cuda.empty_cache()
