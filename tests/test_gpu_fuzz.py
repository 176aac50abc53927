"""Seeded random shapes through every entry point, against the oracle.

Row counts from 1 to a few thousand (around the 64-lane window and the
merge-path slice sizes), row-length mixes with empty rows, a single heavy
row split over many workers, constant tiny rows, duplicate and unsorted
columns, every width with a fast variant plus odd widths for the generic
path, and any output width for the Section 6.2 products; the <SDDMM, SpMM>
and Section 6.2 cases run again at a seeded grid factor.  Same tolerance rule as
tests/parity.py."""
import numpy as np
import pytest

import oracle
import paper_2205_11622_amd as slnr
import synth
from tests.gpu_util import check_A_rows, check_Y, fused, make_problem, unfused, upload
from tests.parity import assert_rows_close

pytestmark = pytest.mark.gpu


def lengths_for(rng):
    N = int(rng.choice([1, 2, 7, 63, 64, 65, 500, 1999, 3001]))
    kind = int(rng.integers(0, 4))
    if kind == 0:                                  # short uniform rows
        n = rng.integers(0, 40, N)
    elif kind == 1:                                # power law, 40% empty
        n = (rng.pareto(1.1, N) * 3).astype(np.int64)
        n[rng.random(N) < 0.4] = 0
        n = np.minimum(n, 4000)
    elif kind == 2:                                # one heavy row, the rest empty
        n = np.zeros(N, np.int64)
        n[int(rng.integers(0, N))] = int(rng.integers(1000, 20000))
    else:                                          # constant 0, 1 or 2 per row
        n = np.full(N, int(rng.integers(0, 3)), np.int64)
    return n.astype(np.int64)


def problem(rng, seed, K, L):
    n = lengths_for(rng)
    M = int(rng.choice([1, 5, 300, 2048]))
    dups = bool(rng.integers(0, 2)) or int(n.max(initial=0)) > M
    unsorted = bool(rng.integers(0, 2))
    return make_problem(n, M, K, L, seed=seed, dups=dups, unsorted=unsorted, dense="normal")


def dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda:0")


FUSED_WIDTHS = [(32, 32), (64, 64), (128, 128), (256, 256), (16, 256), (16, 16), (3, 7),
                (48, 80), (128, 64), (1, 300), (32, 128), (64, 16), (16, 512), (512, 128),
                (128, 512), (256, 64)]


@pytest.mark.parametrize("seed", range(32))
def test_fuzz_fused_and_unfused(gpu, seed):
    rng = np.random.default_rng(1000 + seed)
    K, L = FUSED_WIDTHS[seed % len(FUSED_WIDTHS)]
    p = problem(rng, seed, K, L)
    d = upload(p)
    check_A_rows(p, fused(d), what="fused seed %d" % seed)
    Y, Au = unfused(d)
    check_Y(p, Y)
    check_A_rows(p, Au, what="unfused seed %d" % seed)
    # again at a fixed grid factor (sparselnr_set_grid_factor), drawn per seed
    f = int(np.random.default_rng(5000 + seed).choice([1, 2, 3, 8, 24, 64]))
    try:
        slnr.sparselnr_set_grid_factor(f)
        check_A_rows(p, fused(d), what="fused seed %d, grid factor %d" % (seed, f))
        Y, Au = unfused(d)
        check_Y(p, Y)
        check_A_rows(p, Au, what="unfused seed %d, grid factor %d" % (seed, f))
    finally:
        slnr.sparselnr_set_grid_factor(0)


EPI_WIDTHS = [16, 32, 64, 128, 256, 512]


@pytest.mark.parametrize("seed", range(12))
def test_fuzz_section62_products(gpu, seed):
    rng = np.random.default_rng(2000 + seed)
    lin = EPI_WIDTHS[seed % len(EPI_WIDTHS)]
    lout = int(rng.integers(1, 300))
    p = problem(rng, seed, lin, lin)
    rp, ci, v = dev(p.rowptr), dev(p.colidx), dev(p.vals)
    W = synth.normal(seed, 9, (lin, lout))
    refs = [oracle.sddmm_spmm_gemm_rows(p.rowptr, p.colidx, p.vals, p.C, p.D, p.E, W),
            oracle.spmm_gemm_rows(p.rowptr, p.colidx, p.vals, p.D, W),
            oracle.spmmh_gemm_rows(p.rowptr, p.colidx, p.vals, p.D, p.E, W)]
    # at the automatic grid factor, then at a seeded fixed one
    f = int(np.random.default_rng(6000 + seed).choice([1, 2, 3, 8, 24, 64]))
    try:
        for factor in (0, f):
            slnr.sparselnr_set_grid_factor(factor)
            tag = "seed %d, grid factor %d" % (seed, factor)
            # <SDDMM, SpMM, GEMM>
            A = slnr.sparselnr_fused_sddmm_spmm_gemm(rp, ci, v, dev(p.C), dev(p.D), dev(p.E),
                                                     dev(W))
            assert_rows_close(A.cpu().numpy(), refs[0][0], refs[0][1],
                              what="sddmm_spmm_gemm " + tag)
            # <SpMM, GEMM> with C = D (M x lin)
            A = slnr.sparselnr_spmm_gemm(rp, ci, v, dev(p.D), dev(W))
            assert_rows_close(A.cpu().numpy(), refs[1][0], refs[1][1], what="spmm_gemm " + tag)
            # <SpMMH, GEMM> with C, D = D, E (M x lin each)
            A = slnr.sparselnr_spmmh_gemm(rp, ci, v, dev(p.D), dev(p.E), dev(W))
            assert_rows_close(A.cpu().numpy(), refs[2][0], refs[2][1], what="spmmh_gemm " + tag)
    finally:
        slnr.sparselnr_set_grid_factor(0)


@pytest.mark.parametrize("seed", range(6))
def test_fuzz_transposed_D(gpu, seed):
    rng = np.random.default_rng(3000 + seed)
    K, L = FUSED_WIDTHS[(2 * seed + 1) % len(FUSED_WIDTHS)]
    p = problem(rng, seed, K, L)
    Dt = np.ascontiguousarray(p.D.T)
    A = slnr.sparselnr_fused_sddmm_spmm_dt(dev(p.rowptr), dev(p.colidx), dev(p.vals), dev(p.C),
                                            dev(Dt), dev(p.E))
    ref, scale, _ = oracle.fused_rows_dt(p.rowptr, p.colidx, p.vals, p.C, Dt, p.E)
    assert_rows_close(A.cpu().numpy(), ref, scale, what="dt seed %d" % seed)
