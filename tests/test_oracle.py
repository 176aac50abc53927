"""Pins for the CPU oracle against what the paper and mathematics fix.

Nothing here re-types the oracle's own loops.  The oracle (two-kernel form,
Figure 2a then 2b, fp64) is checked against:
  * a hand-worked example (tests/golden/hand_example.json);
  * dense brute force A = (B .* (C D^T)) E, the gemm/spelmm/spmm decomposition
    of Section 3.1, built from numpy matrix products;
  * the perfect four-deep nest of Figure 2c (Section 3.1.1), O(nnz K L);
  * closed forms for special operands (E = I, C = D = 1, B = I, K = 1);
  * invariants: zero B, linearity, column order, row permutation;
  * the op counts of Section 3.1.3 (nnz K + nnz L for this schedule).
Small-integer inputs make every fp64 sum exact, so several pins compare bit
for bit.
"""
import json
import os

import numpy as np
import pytest

import oracle
from tests.parity import assert_rows_close, row_errors

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_example.json")


def random_csr(rng, N, M, max_deg, allow_dups=False, shuffle=False, empty_frac=0.2):
    rows = []
    for i in range(N):
        if rng.random() < empty_frac:
            rows.append(np.zeros(0, dtype=np.int32))
            continue
        d = int(rng.integers(1, max_deg + 1))
        if allow_dups:
            cols = rng.integers(0, M, size=d)
        else:
            cols = rng.choice(M, size=min(d, M), replace=False)
            if not shuffle:
                cols = np.sort(cols)
        rows.append(cols.astype(np.int32))
    rowptr = np.zeros(N + 1, dtype=np.int32)
    rowptr[1:] = np.cumsum([r.size for r in rows])
    colidx = np.concatenate(rows) if rows else np.zeros(0, np.int32)
    return rowptr, colidx.astype(np.int32)


def dense_B(rowptr, colidx, vals, M):
    N = rowptr.size - 1
    B = np.zeros((N, M), dtype=np.float64)
    rows = np.repeat(np.arange(N), np.diff(rowptr))
    np.add.at(B, (rows, colidx), vals.astype(np.float64))
    return B


def brute_force(rowptr, colidx, vals, C, D, E):
    """Section 3.1: T = gemm(C, D), U = spelmm(B, T), A = spmm(U, E), all dense fp64."""
    M = D.shape[0]
    B = dense_B(rowptr, colidx, vals, M)
    T = C.astype(np.float64) @ D.astype(np.float64).T
    U = B * T
    return U @ E.astype(np.float64)


def perfect_nest(rowptr, colidx, vals, C, D, E):
    """Figure 2c: one perfectly nested loop over i, p, l, k (tiny inputs only)."""
    N, K = C.shape
    L = E.shape[1]
    A = np.zeros((N, L))
    for i in range(N):
        for p in range(rowptr[i], rowptr[i + 1]):
            j = colidx[p]
            for l in range(L):
                t = 0.0
                for k in range(K):
                    t += float(vals[p]) * float(C[i, k]) * float(D[j, k]) * float(E[j, l])
                A[i, l] += t
    return A


def ints(rng, shape, lo=-3, hi=3):
    return rng.integers(lo, hi + 1, size=shape).astype(np.float32)


def test_golden_hand_example():
    g = json.load(open(GOLDEN))
    rp, ci = np.array(g["rowptr"], np.int32), np.array(g["colidx"], np.int32)
    v = np.array(g["vals"], np.float32)
    C, D, E = (np.array(g[x], np.float32) for x in "CDE")
    A, scale, Y, Ys, ops = oracle.fused_rows(rp, ci, v, C, D, E, with_y=True)
    assert np.array_equal(A, np.array(g["A"]))
    assert np.array_equal(scale, np.array(g["scale"]))
    assert np.array_equal(Y, np.array(g["Y"]))
    Y2, _ = oracle.sddmm(rp, ci, v, C, D)
    assert np.array_equal(Y2, np.array(g["Y"]))
    A2, _ = oracle.spmm(rp, ci, Y2, E)
    assert np.array_equal(A2, np.array(g["A"]))
    assert ops == 3 * (g["K"] + g["L"])


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("K,L", [(1, 1), (3, 5), (16, 32), (32, 16)])
def test_matches_dense_brute_force(seed, K, L):
    rng = np.random.default_rng(seed)
    N, M = int(rng.integers(1, 200)), int(rng.integers(1, 256))
    rp, ci = random_csr(rng, N, M, 12, allow_dups=seed % 2 == 1, shuffle=seed % 3 == 0)
    v = rng.uniform(-1, 1, ci.size).astype(np.float32)
    C = rng.standard_normal((N, K)).astype(np.float32)
    D = rng.standard_normal((M, K)).astype(np.float32)
    E = rng.standard_normal((M, L)).astype(np.float32)
    A, scale, ops = oracle.fused_rows(rp, ci, v, C, D, E)
    ref = brute_force(rp, ci, v, C, D, E)
    denom = np.abs(ref).max() + 1e-300
    assert np.abs(A - ref).max() <= 1e-12 * max(denom, 1.0)
    # the two-kernel entry points agree with the row-wise path bit for bit
    Y, _ = oracle.sddmm(rp, ci, v, C, D)
    A2, _ = oracle.spmm(rp, ci, Y, E)
    assert np.array_equal(A, A2)
    assert ops == ci.size * (K + L)


def test_integer_inputs_exact_against_brute_force_and_fig2c():
    rng = np.random.default_rng(11)
    N, M, K, L = 17, 13, 3, 4
    rp, ci = random_csr(rng, N, M, 6, allow_dups=True)
    v, C, D, E = ints(rng, ci.size), ints(rng, (N, K)), ints(rng, (M, K)), ints(rng, (M, L))
    A, _, _ = oracle.fused_rows(rp, ci, v, C, D, E)
    assert np.array_equal(A, brute_force(rp, ci, v, C, D, E))
    assert np.array_equal(A, perfect_nest(rp, ci, v, C, D, E))


def test_sddmm_values_are_sampled_gemm():
    rng = np.random.default_rng(3)
    N, M, K = 40, 50, 7
    rp, ci = random_csr(rng, N, M, 9, allow_dups=True)
    v = rng.uniform(-1, 1, ci.size).astype(np.float32)
    C = rng.standard_normal((N, K)).astype(np.float32)
    D = rng.standard_normal((M, K)).astype(np.float32)
    Y, Ys, ops = oracle.sddmm(rp, ci, v, C, D, with_scale=True)
    T = C.astype(np.float64) @ D.astype(np.float64).T
    rows = np.repeat(np.arange(N), np.diff(rp))
    ref = v.astype(np.float64) * T[rows, ci]
    assert np.allclose(Y, ref, rtol=1e-13, atol=1e-13)
    Tabs = np.abs(C.astype(np.float64)) @ np.abs(D.astype(np.float64)).T
    assert np.allclose(Ys, np.abs(v) * Tabs[rows, ci], rtol=1e-13, atol=0)
    assert ops == ci.size * K


def test_identity_E_gives_densified_sddmm():
    # E = I_M (L = M): A is the SDDMM result scattered into a dense N x M matrix
    rng = np.random.default_rng(5)
    N, M, K = 30, 24, 6
    rp, ci = random_csr(rng, N, M, 8, allow_dups=True)
    v, C, D = ints(rng, ci.size), ints(rng, (N, K)), ints(rng, (M, K))
    E = np.eye(M, dtype=np.float32)
    A, _, _ = oracle.fused_rows(rp, ci, v, C, D, E)
    T = C.astype(np.float64) @ D.astype(np.float64).T
    ref = np.zeros((N, M))
    rows = np.repeat(np.arange(N), np.diff(rp))
    np.add.at(ref, (rows, ci), v * T[rows, ci])
    assert np.array_equal(A, ref)


def test_ones_C_D_gives_scaled_spmm():
    # C = 1, D = 1: every dot product is K, so A = K * (B E)
    rng = np.random.default_rng(6)
    N, M, K, L = 25, 19, 5, 7
    rp, ci = random_csr(rng, N, M, 7, allow_dups=True)
    v, E = ints(rng, ci.size), ints(rng, (M, L))
    C, D = np.ones((N, K), np.float32), np.ones((M, K), np.float32)
    A, _, _ = oracle.fused_rows(rp, ci, v, C, D, E)
    B = dense_B(rp, ci, v, M)
    assert np.array_equal(A, K * (B @ E.astype(np.float64)))


def test_identity_B():
    # B = I: A_i = dot(C_i, D_i) * E_i
    rng = np.random.default_rng(7)
    N, K, L = 33, 9, 4
    rp = np.arange(N + 1, dtype=np.int32)
    ci = np.arange(N, dtype=np.int32)
    v = np.ones(N, np.float32)
    C, D, E = ints(rng, (N, K)), ints(rng, (N, K)), ints(rng, (N, L))
    A, _, _ = oracle.fused_rows(rp, ci, v, C, D, E)
    dots = (C.astype(np.float64) * D.astype(np.float64)).sum(axis=1)
    assert np.array_equal(A, dots[:, None] * E.astype(np.float64))


def test_K1_is_diagonal_scaling():
    # K = 1: A = diag(C) B diag(D) E
    rng = np.random.default_rng(8)
    N, M, L = 21, 16, 5
    rp, ci = random_csr(rng, N, M, 6, allow_dups=True)
    v, C, D, E = ints(rng, ci.size), ints(rng, (N, 1)), ints(rng, (M, 1)), ints(rng, (M, L))
    A, _, _ = oracle.fused_rows(rp, ci, v, C, D, E)
    B = dense_B(rp, ci, v, M)
    ref = np.diag(C[:, 0].astype(np.float64)) @ B @ np.diag(D[:, 0].astype(np.float64)) @ E
    assert np.array_equal(A, ref)


def test_zero_B_gives_exact_zero():
    rng = np.random.default_rng(9)
    N, M, K, L = 50, 40, 8, 8
    rp, ci = random_csr(rng, N, M, 10)
    v = np.zeros(ci.size, np.float32)
    C, D, E = (rng.standard_normal(s).astype(np.float32) for s in [(N, K), (M, K), (M, L)])
    A, scale, _ = oracle.fused_rows(rp, ci, v, C, D, E)
    assert np.all(A == 0) and np.all(scale == 0)


def test_linear_in_E_and_vals():
    rng = np.random.default_rng(10)
    N, M, K, L = 30, 30, 4, 6
    rp, ci = random_csr(rng, N, M, 8, allow_dups=True)
    v, C, D = ints(rng, ci.size), ints(rng, (N, K)), ints(rng, (M, K))
    E1, E2 = ints(rng, (M, L)), ints(rng, (M, L))
    A1, _, _ = oracle.fused_rows(rp, ci, v, C, D, E1)
    A2, _, _ = oracle.fused_rows(rp, ci, v, C, D, E2)
    A12, _, _ = oracle.fused_rows(rp, ci, v, C, D, E1 + 2 * E2)
    assert np.array_equal(A12, A1 + 2 * A2)
    v2 = ints(rng, ci.size)
    Av2, _, _ = oracle.fused_rows(rp, ci, v2, C, D, E1)
    Avv, _, _ = oracle.fused_rows(rp, ci, v - 3 * v2, C, D, E1)
    assert np.array_equal(Avv, A1 - 3 * Av2)


def test_column_order_within_row_does_not_matter():
    rng = np.random.default_rng(12)
    N, M, K, L = 40, 60, 5, 5
    rp, ci = random_csr(rng, N, M, 12, allow_dups=True)
    v, C, D, E = ints(rng, ci.size), ints(rng, (N, K)), ints(rng, (M, K)), ints(rng, (M, L))
    A, _, _ = oracle.fused_rows(rp, ci, v, C, D, E)
    perm = np.arange(ci.size)
    for i in range(N):
        seg = perm[rp[i]:rp[i + 1]]
        rng.shuffle(seg)
    A2, _, _ = oracle.fused_rows(rp, ci[perm], v[perm], C, D, E)
    assert np.array_equal(A, A2)


def test_row_permutation_permutes_A():
    rng = np.random.default_rng(13)
    N, M, K, L = 35, 20, 4, 3
    rp, ci = random_csr(rng, N, M, 7, allow_dups=True)
    v, C, D, E = ints(rng, ci.size), ints(rng, (N, K)), ints(rng, (M, K)), ints(rng, (M, L))
    A, _, _ = oracle.fused_rows(rp, ci, v, C, D, E)
    pi = rng.permutation(N)
    lens = np.diff(rp)[pi]
    rp2 = np.zeros(N + 1, np.int32)
    rp2[1:] = np.cumsum(lens)
    idx = np.concatenate([np.arange(rp[i], rp[i + 1]) for i in pi]).astype(np.int64)
    A2, _, _ = oracle.fused_rows(rp2, ci[idx], v[idx], C[pi], D, E)
    assert np.array_equal(A2, A[pi])


def test_scale_bounds_and_nonnegative_case():
    rng = np.random.default_rng(14)
    N, M, K, L = 60, 50, 6, 9
    rp, ci = random_csr(rng, N, M, 10, allow_dups=True)
    v = rng.uniform(-1, 1, ci.size).astype(np.float32)
    C, D, E = (rng.standard_normal(s).astype(np.float32) for s in [(N, K), (M, K), (M, L)])
    A, scale, _ = oracle.fused_rows(rp, ci, v, C, D, E)
    assert np.all(np.abs(A).max(axis=1) <= scale * (1 + 1e-12))
    # with nonnegative operands the scale is the row maximum of A itself
    Ap, sp, _ = oracle.fused_rows(rp, ci, np.abs(v), np.abs(C), np.abs(D), np.abs(E))
    assert np.allclose(Ap.max(axis=1), sp, rtol=1e-13, atol=0)


def test_scale_outputs_match_dense_absolute_products():
    """Every tolerance scale the oracle returns is its definition on absolute
    values, written here as dense numpy products on small integers (exact in
    fp64): the SDDMM scale |b_p| (|C| |D|^T)[i, j]; the SpMM scale
    max_l (S |E|)[i, l] with S[i, j] the sum of the Yabs of row i's nonzeros
    in column j; and the fused scale max_l ((|B| .* (|C| |D|^T)) |E|)[i, l].
    The inputs have negative entries in every operand and rows whose column
    sums differ, so a dropped absolute value, a sum over l in place of the
    maximum, or a transposed operand changes the result."""
    rng = np.random.default_rng(21)
    N, M, K, L = 40, 30, 5, 7
    rp, ci = random_csr(rng, N, M, 9, allow_dups=True, shuffle=True)
    v = ints(rng, ci.size)
    C, D, E = ints(rng, (N, K)), ints(rng, (M, K)), ints(rng, (M, L))
    assert (v < 0).any() and (C < 0).any() and (D < 0).any() and (E < 0).any()
    Ba = dense_B(rp, ci, np.abs(v), M)
    Ta = np.abs(C).astype(np.float64) @ np.abs(D).astype(np.float64).T
    rows = np.repeat(np.arange(N), np.diff(rp))
    # SDDMM scale per nonzero
    Y, Yscale, _ = oracle.sddmm(rp, ci, v, C, D, with_scale=True)
    assert np.array_equal(Yscale, np.abs(v).astype(np.float64) * Ta[rows, ci])
    # SpMM scale per row, from an arbitrary nonnegative Yabs (integers)
    Yabs = rng.integers(0, 5, size=ci.size).astype(np.float64)
    S = np.zeros((N, M))
    np.add.at(S, (rows, ci), Yabs)
    full = S @ np.abs(E).astype(np.float64)
    A, Ascale, _ = oracle.spmm(rp, ci, Y, E, Yabs=Yabs)
    assert np.array_equal(Ascale, full.max(axis=1))
    # the planted slips give other values on these inputs
    assert not np.array_equal(Ascale, full.sum(axis=1))
    assert not np.array_equal(Ascale, (S @ E.astype(np.float64)).max(axis=1))
    # the values themselves are unchanged by asking for the scale
    A0, _ = oracle.spmm(rp, ci, Y, E)
    assert np.array_equal(A, A0)
    # fused scale per row
    Afull = (Ba * Ta) @ np.abs(E).astype(np.float64)
    _, scale, _ = oracle.fused_rows(rp, ci, v, C, D, E)
    assert np.array_equal(scale, Afull.max(axis=1))
    # and the SpMM scale carried from the SDDMM scale equals the fused one
    _, As2, _ = oracle.spmm(rp, ci, Y, E, Yabs=Yscale)
    assert np.array_equal(As2, scale)


def test_subset_rows_match_full():
    rng = np.random.default_rng(15)
    N, M, K, L = 80, 70, 8, 8
    rp, ci = random_csr(rng, N, M, 10)
    v = rng.uniform(-1, 1, ci.size).astype(np.float32)
    C, D, E = (rng.standard_normal(s).astype(np.float32) for s in [(N, K), (M, K), (M, L)])
    A, scale, _ = oracle.fused_rows(rp, ci, v, C, D, E)
    rows = np.array([79, 0, 5, 5, 40], dtype=np.int64)
    As, ss, Ys, Yss, _ = oracle.fused_rows(rp, ci, v, C, D, E, rows=rows, with_y=True)
    assert np.array_equal(As, A[rows]) and np.array_equal(ss, scale[rows])
    Yall, Ysall, _ = oracle.sddmm(rp, ci, v, C, D, with_scale=True)
    idx = np.concatenate([np.arange(rp[i], rp[i + 1]) for i in rows])
    assert np.array_equal(Ys, Yall[idx]) and np.array_equal(Yss, Ysall[idx])


def test_parity_rule_detects_planted_mistakes():
    """The 1e-4 row rule is sharp enough to catch plausible oracle-side slips
    (a dropped nonzero, a wrong sign, a transposed D): each planted mistake is
    made on the CPU in a copy of the reference result or its inputs."""
    rng = np.random.default_rng(16)
    N, M, K, L = 64, 64, 8, 8
    rp, ci = random_csr(rng, N, M, 10, empty_frac=0.0)
    v = rng.uniform(-1, 1, ci.size).astype(np.float32)
    C, D, E = (rng.uniform(-1, 1, s).astype(np.float32) for s in [(N, K), (M, K), (M, L)])
    A, scale, _ = oracle.fused_rows(rp, ci, v, C, D, E)
    assert_rows_close(A.astype(np.float32), A, scale)
    # dropped last nonzero of every row
    v_drop = v.copy()
    v_drop[rp[1:] - 1] = 0
    Ad, _, _ = oracle.fused_rows(rp, ci, v_drop, C, D, E)
    assert (row_errors(Ad, A, scale)[1] > 1e-4).mean() > 0.9
    # sign flip of B
    Af, _, _ = oracle.fused_rows(rp, ci, -v, C, D, E)
    assert (row_errors(Af, A, scale)[1] > 1e-4).mean() > 0.9
    # D^T in place of D (square K x K block read the wrong way)
    Dt = np.ascontiguousarray(D.reshape(M // K, K, K).transpose(0, 2, 1).reshape(M, K))
    At, _, _ = oracle.fused_rows(rp, ci, v, C, Dt, E)
    assert (row_errors(At, A, scale)[1] > 1e-4).mean() > 0.9
    # NaN anywhere fails its row
    Anan = A.copy()
    Anan[3, 2] = np.nan
    assert np.isinf(row_errors(Anan, A, scale)[1][3])
