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


# ------------------------------------------------ every row at full size
#
# The full-size workloads are compared on every row: the oracle runs once
# over all rows in chunks of CHUNK rows (bounded host memory), its fp64
# results are kept on the device, and each GPU result is checked there with
# the rule of tests/parity.py (rows_close_dev), so a sweep over launch
# configurations costs one oracle pass.

CHUNK = 65536


def oracle_reference(fn, N, width, device, nnz_of=None, chunk=CHUNK):
    """Runs fn(rows) -> (ref rows, scale[, Y, Yscale]) over all N rows in
    chunks and returns the results as fp64 device tensors: (ref N x width,
    scale N) or, when nnz_of gives the row pointer for the SDDMM values,
    (ref, scale, Y nnz, Yscale nnz)."""
    import torch
    ref = torch.empty((N, width), dtype=torch.float64, device=device)
    scale = torch.empty(N, dtype=torch.float64, device=device)
    ys = None
    if nnz_of is not None:
        nnz = int(nnz_of[N])
        ys = (torch.empty(nnz, dtype=torch.float64, device=device),
              torch.empty(nnz, dtype=torch.float64, device=device))
    for r0 in range(0, N, chunk):
        r1 = min(N, r0 + chunk)
        out = fn(np.arange(r0, r1, dtype=np.int64))
        ref[r0:r1] = torch.from_numpy(out[0]).to(device)
        scale[r0:r1] = torch.from_numpy(out[1]).to(device)
        if ys is not None:
            p0, p1 = int(nnz_of[r0]), int(nnz_of[r1])
            ys[0][p0:p1] = torch.from_numpy(out[2]).to(device)
            ys[1][p0:p1] = torch.from_numpy(out[3]).to(device)
    return (ref, scale) if ys is None else (ref, scale) + ys


def fused_reference(p, device):
    """Every row of the <SDDMM, SpMM> result and every SDDMM value of p, with scales."""
    return oracle_reference(
        lambda rows: oracle.fused_rows(p.rowptr, p.colidx, p.vals, p.C, p.D, p.E, rows=rows,
                                       with_y=True)[:4], p.N, p.L, device, nnz_of=p.rowptr)


def row_ratios_dev(got, ref, scale):
    """The per-row ratio err / scale of tests/parity.py for torch tensors
    (any device): inf for a non-finite row or a nonzero row of zero scale."""
    import torch
    g = got.double()
    r = ref
    if g.dim() == 1:
        g, r = g[:, None], r[:, None]
    if g.shape[1] == 0:
        return torch.zeros(g.shape[0], dtype=torch.float64, device=g.device)
    err = (g - r).abs().amax(dim=1)
    finite = torch.isfinite(g).all(dim=1)
    inf = torch.full_like(err, float("inf"))
    pos = scale > 0
    ratio = torch.where(pos, err / torch.where(pos, scale, torch.ones_like(scale)),
                        torch.where(err == 0, torch.zeros_like(err), inf))
    ratio = torch.where(finite, ratio, inf)
    return torch.where(torch.isnan(ratio), inf, ratio), err


def rows_close_dev(got, ref, scale, tol=TOL, what="A", chunk=CHUNK):
    """Asserts the parity rule on every row (chunked); returns the worst ratio."""
    worst = 0.0
    n = got.shape[0]
    for r0 in range(0, n, chunk):
        r1 = min(n, r0 + chunk)
        ratio, err = row_ratios_dev(got[r0:r1], ref[r0:r1], scale[r0:r1])
        bad = int((~(ratio <= tol)).sum())
        k = int(ratio.argmax())
        if bad:
            raise AssertionError(
                "%s: %d rows in [%d, %d) outside %g*scale; worst row %d: err=%.3e scale=%.3e "
                "ratio=%.3e" % (what, bad, r0, r1, tol, r0 + k, float(err[k]),
                                float(scale[r0 + k]), float(ratio[k])))
        worst = max(worst, float(ratio[k]))
    return worst
