"""Helpers shared by the GPU parity tests: upload a synth.Problem, run the
library through its binding, and compare rows with the oracle."""
from __future__ import annotations

import numpy as np

import oracle
import paper_2205_11622_amd as slnr
from tests.parity import TOL, assert_rows_close


def upload(p, device="cuda:0"):
    import torch
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device)  # noqa: E731
    return dict(rowptr=t(p.rowptr), colidx=t(p.colidx), vals=t(p.vals), C=t(p.C), D=t(p.D),
                E=t(p.E))


def fused(d):
    return slnr.sparselnr_fused_sddmm_spmm(d["rowptr"], d["colidx"], d["vals"], d["C"], d["D"],
                                           d["E"])


def unfused(d):
    return slnr.sparselnr_unfused_sddmm_spmm(d["rowptr"], d["colidx"], d["vals"], d["C"],
                                             d["D"], d["E"])


def sample_rows(p, n_random=2000, seed=0, heaviest=64):
    """Rows to check at full size: random rows, the heaviest rows (they are
    split across workers), empty rows and the first and last rows."""
    rng = np.random.default_rng(seed)
    N = p.N
    deg = np.diff(p.rowptr)
    pick = [rng.choice(N, size=min(n_random, N), replace=False)]
    pick.append(np.argsort(deg)[-heaviest:])
    empty = np.nonzero(deg == 0)[0]
    if empty.size:
        pick.append(empty[:32])
    pick.append(np.array([0, N - 1]))
    return np.unique(np.concatenate(pick)).astype(np.int64)


def check_A_rows(p, A_dev, rows=None, tol=TOL, what="A"):
    """Compares rows of the device result with the oracle; returns the worst ratio."""
    import torch
    if rows is None:
        rows = np.arange(p.N, dtype=np.int64)
        got = A_dev.cpu().numpy()
    else:
        got = A_dev[torch.from_numpy(rows).to(A_dev.device)].cpu().numpy()
    ref, scale, _ = oracle.fused_rows(p.rowptr, p.colidx, p.vals, p.C, p.D, p.E, rows=rows)
    return assert_rows_close(got, ref, scale, tol, what)


def check_Y(p, Y_dev, rows=None, tol=TOL):
    """Compares SDDMM values per nonzero with the oracle (rows' nonzeros in order)."""
    if rows is None:
        rows = np.arange(p.N, dtype=np.int64)
    _, _, Yref, Yscale, _ = oracle.fused_rows(p.rowptr, p.colidx, p.vals, p.C, p.D, p.E,
                                              rows=rows, with_y=True)
    idx = np.concatenate([np.arange(p.rowptr[i], p.rowptr[i + 1]) for i in rows]) \
        if rows.size else np.zeros(0, np.int64)
    import torch
    got = Y_dev[torch.from_numpy(idx).to(Y_dev.device)].cpu().numpy() if idx.size else np.zeros(0)
    return assert_rows_close(got, Yref, Yscale, tol, "Y")


def make_problem(lengths, M, K, L, seed=0, dups=False, unsorted=False, dense="uniform"):
    """A seeded synth.Problem with the given row lengths (test shapes)."""
    import synth
    rng = np.random.default_rng(seed)
    lengths = np.asarray(lengths, dtype=np.int64)
    N = lengths.size
    rowptr = np.zeros(N + 1, dtype=np.int32)
    rowptr[1:] = np.cumsum(lengths)
    cols = []
    for n in lengths:
        if n == 0:
            continue
        if dups or n > M:
            c = rng.integers(0, M, size=n)
        else:
            c = rng.choice(M, size=n, replace=False)
        if not unsorted:
            c = np.sort(c)
        cols.append(c)
    colidx = (np.concatenate(cols) if cols else np.zeros(0)).astype(np.int32)
    vals = synth.uniform(seed, synth.STREAM_VALS, colidx.size, -1.0, 1.0)
    if dense == "normal":
        C = synth.normal(seed, synth.STREAM_C, (N, K))
        D = synth.normal(seed, synth.STREAM_D, (M, K))
        E = synth.normal(seed, synth.STREAM_E, (M, L))
    else:
        C = synth.uniform(seed, synth.STREAM_C, (N, K))
        D = synth.uniform(seed, synth.STREAM_D, (M, K))
        E = synth.uniform(seed, synth.STREAM_E, (M, L))
    return synth.Problem("test", N, M, K, L, rowptr, colidx, vals, C, D, E)


def power_law_lengths(N, seed=0, scale=4.0, cap=None, empty_frac=0.3):
    rng = np.random.default_rng(seed)
    n = (rng.pareto(1.1, N) * scale).astype(np.int64)
    n[rng.random(N) < empty_frac] = 0
    if cap is not None:
        n = np.minimum(n, cap)
    return n
