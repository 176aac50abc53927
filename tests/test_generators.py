"""Synthetic input generators: determinism, structure and distributions."""
import hashlib

import numpy as np
import pytest

import synth


def digest(*arrays):
    h = hashlib.sha256()
    for a in arrays:
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def test_counter_generator_is_splitmix64_of_counter():
    # element n of a stream is mix64(key + (n+1)*golden): consecutive draws differ,
    # and the stream restarts identically
    a = [synth.draw(0, 3, n) for n in range(4)]
    assert a == [synth.draw(0, 3, n) for n in range(4)]
    assert len(set(a)) == 4
    assert synth.draw(0, 3, 0) != synth.draw(1, 3, 0) != synth.draw(0, 4, 0)


def test_splitmix64_reference_value():
    # SplitMix64's finaliser applied to golden-ratio increments from state 0
    # reproduces the first published output of splitmix64.c seeded with 0.
    def mix(z):
        m = (1 << 64) - 1
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & m
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & m
        return z ^ (z >> 31)
    assert mix(0x9E3779B97F4A7C15) == 0xE220A8397B1DCDAF


def test_uniform_and_normal_ranges():
    u = synth.uniform(0, 9, 200_000, -1.0, 1.0)
    assert u.min() >= -1.0 and u.max() < 1.0
    assert abs(u.mean()) < 0.01 and abs(u.var() - 1 / 3) < 0.01
    # 24-bit grid: all values are multiples of 2^-23
    assert np.all(np.round(u.astype(np.float64) * 2**23) == u.astype(np.float64) * 2**23)
    z = synth.normal(0, 9, 200_001)
    assert abs(z.mean()) < 0.01 and abs(z.std() - 1) < 0.01
    assert np.isfinite(z).all()


def test_fixed_degree_structure():
    p = synth.fixed_degree(500, 300, 10, 4, 4, seed=1)
    assert p.nnz == 5000 and np.array_equal(np.diff(p.rowptr), np.full(500, 10))
    for i in range(p.N):
        row = p.colidx[p.rowptr[i]:p.rowptr[i + 1]]
        assert np.all(np.diff(row) > 0) and row.min() >= 0 and row.max() < 300
    # columns cover the range roughly uniformly
    counts = np.bincount(p.colidx, minlength=300)
    assert counts.min() > 0


def test_tiny_config_deterministic():
    a = synth.config("tiny")
    b = synth.config("tiny")
    assert digest(a.rowptr, a.colidx, a.vals, a.C, a.D, a.E) == \
        digest(b.rowptr, b.colidx, b.vals, b.C, b.D, b.E)
    assert (a.N, a.M, a.K, a.L, a.nnz) == (2048, 2048, 32, 32, 20480)
    assert np.all(np.diff(a.rowptr) == 10)
    c = synth.fixed_degree(2048, 2048, 10, 32, 32, seed=1)
    assert not np.array_equal(a.colidx, c.colidx)


def test_rmat_small():
    p = synth.rmat(10, 16, 8, 8, seed=0)
    N = 1 << 10
    assert p.N == N and 0 < p.nnz <= 16 * N
    for i in range(N):
        row = p.colidx[p.rowptr[i]:p.rowptr[i + 1]]
        assert np.all(np.diff(row) > 0)
    assert p.colidx.min() >= 0 and p.colidx.max() < N
    deg = np.diff(p.rowptr)
    assert deg.argmax() == 0  # all-zero-bits row is the heaviest
    # fraction of distinct entries in the top half of rows, before dedup this is a+b = 0.76
    top = deg[: N // 2].sum() / deg.sum()
    assert 0.68 < top < 0.80
    assert 0.0 <= p.vals.min() and p.vals.max() < 1.0


def test_rmat_thread_count_independent(monkeypatch):
    a = synth.rmat(12, 8, 4, 4, seed=3)
    b = synth.rmat(12, 8, 4, 4, seed=3)
    assert digest(a.rowptr, a.colidx, a.vals) == digest(b.rowptr, b.colidx, b.vals)


@pytest.mark.parametrize("n", [1, 2, 4, 7])
def test_stencil_structure(n):
    p = synth.stencil27(n, 2, 2)
    N = n ** 3
    assert p.N == N and p.nnz == (3 * n - 2) ** 3 if n > 1 else p.nnz == 1
    deg = np.diff(p.rowptr)
    allowed = {1} if n == 1 else ({8, 12, 18, 27} if n > 2 else {8})
    assert set(deg.tolist()) <= allowed
    # symmetric pattern containing the diagonal, sorted rows
    B = np.zeros((N, N), bool)
    rows = np.repeat(np.arange(N), deg)
    B[rows, p.colidx] = True
    assert np.array_equal(B, B.T) and B.diagonal().all()
    for i in range(N):
        assert np.all(np.diff(p.colidx[p.rowptr[i]:p.rowptr[i + 1]]) > 0)


def test_model_bytes_formula():
    p = synth.fixed_degree(10, 10, 3, 4, 5)
    assert p.model_bytes() == 4 * 11 + 8 * 30 + 4 * 30 * 9 + 4 * 10 * 4 + 4 * 10 * 5
