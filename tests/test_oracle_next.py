"""Pins for the oracle's further computations (the paper's Section 6.2
benchmarks built on the same skeleton, and the transposed-D layout of
Section 4.3.1), each against dense brute force built from numpy products,
exactly on small-integer inputs, plus special cases."""
import numpy as np
import pytest

import oracle
from tests.test_oracle import dense_B, ints, random_csr


def case(seed, N=23, M=19, dups=True):
    rng = np.random.default_rng(seed)
    rp, ci = random_csr(rng, N, M, 7, allow_dups=dups)
    return rng, rp, ci, ints(rng, ci.size)


@pytest.mark.parametrize("seed", range(3))
def test_sddmm_spmm_gemm_brute_force_exact(seed):
    rng, rp, ci, v = case(seed)
    N, M, K, L, Mo = rp.size - 1, 19, 3, 4, 5
    C, D, F, W = ints(rng, (N, K)), ints(rng, (M, K)), ints(rng, (M, L)), ints(rng, (L, Mo))
    A, scale, ops = oracle.sddmm_spmm_gemm_rows(rp, ci, v, C, D, F, W)
    B = dense_B(rp, ci, v, M)
    ref = ((B * (C.astype(float) @ D.astype(float).T)) @ F) @ W
    assert np.array_equal(A, ref)
    Babs = dense_B(rp, ci, np.abs(v), M)  # duplicates: |b| per nonzero, then added
    ref_abs = ((Babs * (np.abs(C.astype(float)) @ np.abs(D.astype(float)).T)) @ np.abs(F)) @ np.abs(W)
    assert np.array_equal(scale, ref_abs.max(axis=1) if Mo else np.zeros(N))
    assert ops == ci.size * (K + L) + N * L * Mo


def test_sddmm_spmm_gemm_identity_W_is_sddmm_spmm():
    rng, rp, ci, v = case(7)
    N, M, K, L = rp.size - 1, 19, 4, 6
    C, D, F = ints(rng, (N, K)), ints(rng, (M, K)), ints(rng, (M, L))
    A, _, _ = oracle.sddmm_spmm_gemm_rows(rp, ci, v, C, D, F, np.eye(L, dtype=np.float32))
    A0, _, _ = oracle.fused_rows(rp, ci, v, C, D, F)
    assert np.array_equal(A, A0)


@pytest.mark.parametrize("seed", range(3))
def test_spmm_gemm_brute_force_exact(seed):
    rng, rp, ci, v = case(seed + 10)
    N, M, K, L = rp.size - 1, 19, 5, 3
    C, D = ints(rng, (M, K)), ints(rng, (K, L))
    A, scale, ops = oracle.spmm_gemm_rows(rp, ci, v, C, D)
    B = dense_B(rp, ci, v, M)
    assert np.array_equal(A, (B @ C) @ D)
    Babs = dense_B(rp, ci, np.abs(v), M)
    assert np.array_equal(scale, ((Babs @ np.abs(C)) @ np.abs(D)).max(axis=1))
    assert ops == ci.size * K + N * K * L


def test_spmm_gemm_special_cases():
    rng, rp, ci, v = case(3)
    M, K = 19, 4
    C = ints(rng, (M, K))
    A, _, _ = oracle.spmm_gemm_rows(rp, ci, v, C, np.eye(K, dtype=np.float32))
    assert np.array_equal(A, dense_B(rp, ci, v, M) @ C)   # D = I: plain SpMM
    A0, s0, _ = oracle.spmm_gemm_rows(rp, ci, np.zeros_like(v), C, ints(rng, (K, 3)))
    assert np.all(A0 == 0) and np.all(s0 == 0)


@pytest.mark.parametrize("seed", range(3))
def test_spmmh_gemm_brute_force_exact(seed):
    rng, rp, ci, v = case(seed + 20)
    N, M, J, L = rp.size - 1, 19, 4, 6
    C, D, E = ints(rng, (M, J)), ints(rng, (M, J)), ints(rng, (J, L))
    A, scale, ops = oracle.spmmh_gemm_rows(rp, ci, v, C, D, E)
    B = dense_B(rp, ci, v, M)
    assert np.array_equal(A, (B @ (C * D)) @ E)
    Babs = dense_B(rp, ci, np.abs(v), M)
    assert np.array_equal(scale, ((Babs @ (np.abs(C) * np.abs(D))) @ np.abs(E)).max(axis=1))
    assert ops == ci.size * J + N * J * L


def test_spmmh_ones_D_is_spmm_gemm():
    rng, rp, ci, v = case(5)
    M, J, L = 19, 4, 3
    C, E = ints(rng, (M, J)), ints(rng, (J, L))
    A, _, _ = oracle.spmmh_gemm_rows(rp, ci, v, C, np.ones((M, J), np.float32), E)
    A0, _, _ = oracle.spmm_gemm_rows(rp, ci, v, C, E)
    assert np.array_equal(A, A0)


@pytest.mark.parametrize("seed", range(3))
def test_transposed_D_matches_brute_force_and_plain_layout(seed):
    rng, rp, ci, v = case(seed + 30)
    N, M, K, L = rp.size - 1, 19, 5, 4
    C, D, E = ints(rng, (N, K)), ints(rng, (M, K)), ints(rng, (M, L))
    Dt = np.ascontiguousarray(D.T)
    A, scale, ops = oracle.fused_rows_dt(rp, ci, v, C, Dt, E)
    B = dense_B(rp, ci, v, M)
    assert np.array_equal(A, (B * (C.astype(float) @ Dt.astype(float))) @ E)
    A0, s0, _ = oracle.fused_rows(rp, ci, v, C, D, E)
    assert np.array_equal(A, A0) and np.array_equal(scale, s0)
    assert ops == ci.size * (K + L)


def test_next_rows_subset_and_rectangular():
    rng, rp, ci, v = case(40, N=30, M=11)
    N, M = 30, 11
    C, D = rng.standard_normal((M, 8)).astype(np.float32), rng.standard_normal((8, 3)).astype(np.float32)
    A, s, _ = oracle.spmm_gemm_rows(rp, ci, v, C, D)
    rows = np.array([29, 3, 3, 0], np.int64)
    As, ss, _ = oracle.spmm_gemm_rows(rp, ci, v, C, D, rows=rows)
    assert np.array_equal(As, A[rows]) and np.array_equal(ss, s[rows])
