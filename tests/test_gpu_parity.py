"""GPU parity: the HIP library (through its C ABI) against the fp64 oracle.

Tolerance (tests/parity.py): per row, max_l |A - Aref| <= 1e-4 * scale_i with
scale_i = max_l sum_p |b_p| (sum_k |C_ik||D_jk|) |E_jl|; zero-scale rows must
be exactly zero; NaN/Inf fail.  Structure (Y's order, which rows are written)
must match exactly; invariants marked "bit" are compared bit for bit.
"""
import numpy as np
import pytest

import oracle
import paper_2205_11622_amd as slnr
import synth
from tests.gpu_util import (check_A_rows, check_Y, fused, fused_reference, make_problem,
                            power_law_lengths, rows_close_dev, sample_rows, unfused, upload)
from tests.parity import assert_rows_close

pytestmark = pytest.mark.gpu


# ---------------------------------------------------------------- variants

# (K, L): the first five have hand-tuned fast variants, the rest go through
# the generic kernel (odd widths, K != L, tiny widths, wide L needing tiles);
# the unfused SpMM also has fast variants at L = 16 and 512.
WIDTHS = [(32, 32), (64, 64), (128, 128), (256, 256), (16, 256),
          (1, 1), (3, 5), (16, 16), (20, 36), (17, 300), (64, 520), (128, 64), (64, 512)]


@pytest.mark.parametrize("K,L", WIDTHS)
def test_fused_and_unfused_power_law(gpu, K, L):
    # 3001 rows (ragged), ~30% empty, heavy rows spanning many workers
    lengths = power_law_lengths(3001, seed=K * 1000 + L, cap=6000)
    lengths[7] = 9000
    p = make_problem(lengths, 2500, K, L, seed=K + L, dense="normal")
    d = upload(p)
    A = fused(d)
    check_A_rows(p, A, what="fused A")
    Y, Au = unfused(d)
    check_Y(p, Y)
    check_A_rows(p, Au, what="unfused A")


@pytest.mark.parametrize("K,L", [(32, 32), (128, 128), (16, 256), (5, 7)])
def test_unsorted_and_duplicate_columns(gpu, K, L):
    lengths = np.random.default_rng(3).integers(0, 60, size=777)
    p = make_problem(lengths, 50, K, L, seed=5, dups=True, unsorted=True)
    d = upload(p)
    check_A_rows(p, fused(d))
    Y, Au = unfused(d)
    check_Y(p, Y)
    check_A_rows(p, Au)


# ------------------------------------------------------------ edge cases

def test_empty_matrix(gpu):
    import torch
    dev = gpu
    rp = torch.zeros(1, dtype=torch.int32, device=dev)
    ci = torch.zeros(0, dtype=torch.int32, device=dev)
    v = torch.zeros(0, device=dev)
    C = torch.zeros(0, 32, device=dev)
    D = torch.zeros(5, 32, device=dev)
    E = torch.zeros(5, 32, device=dev)
    A = slnr.sparselnr_fused_sddmm_spmm(rp, ci, v, C, D, E)
    assert A.shape == (0, 32)
    Y, A = slnr.sparselnr_unfused_sddmm_spmm(rp, ci, v, C, D, E)
    assert Y.shape == (0,) and A.shape == (0, 32)


@pytest.mark.parametrize("K,L", [(32, 32), (128, 128), (16, 256), (3, 5)])
def test_no_nonzeros_gives_zero_rows(gpu, K, L):
    import torch
    p = make_problem(np.zeros(1234, np.int64), 10, K, L)
    d = upload(p)
    A = torch.full((p.N, L), float("nan"), device=gpu)
    slnr.sparselnr_fused_sddmm_spmm(d["rowptr"], d["colidx"], d["vals"], d["C"], d["D"], d["E"], A)
    assert bool((A == 0).all())


@pytest.mark.parametrize("K,L", [(128, 128), (16, 256), (64, 64), (32, 32), (9, 9)])
def test_one_dense_row(gpu, K, L):
    # a single row holding every column: the row is split over all workers
    p = make_problem([100_000], 100_000, K, L, seed=2, dense="normal")
    d = upload(p)
    check_A_rows(p, fused(d))
    Y, Au = unfused(d)
    check_Y(p, Y)
    check_A_rows(p, Au)


WIDTHS = [16, 32, 64, 128, 256, 512]


@pytest.mark.parametrize("K", WIDTHS)
@pytest.mark.parametrize("L", WIDTHS)
def test_fused_every_width_pair(gpu, K, L):
    # every K, L pair of the fast variants (and the few that fall back to the
    # generic kernel): power-law rows, one 9000-nonzero row split over many
    # workers, 30% empty rows
    n = power_law_lengths(2300, seed=K * 7 + L, cap=2000)
    n[11] = 9000
    p = make_problem(n, 2500, K, L, seed=K + 3 * L, dense="normal")
    d = upload(p)
    check_A_rows(p, fused(d))
    Y, Au = unfused(d)
    check_Y(p, Y)
    check_A_rows(p, Au)


def _large_problem(N, K, L, seed):
    """Enough rows for several resident grids (the wide-worker kernels): Pareto
    row lengths with 30% empty rows and one 20000-nonzero row, built without a
    per-row loop; columns sorted within rows, repeats allowed."""
    rng = np.random.default_rng(seed)
    lengths = power_law_lengths(N, seed=seed, scale=2.0, cap=3000)
    lengths[N // 3] = 20_000
    rowptr = np.zeros(N + 1, np.int64)
    rowptr[1:] = np.cumsum(lengths)
    nnz = int(rowptr[-1])
    rows = np.repeat(np.arange(N), lengths)
    cols = rng.integers(0, N, size=nnz)
    order = np.lexsort((cols, rows))
    colidx = cols[order].astype(np.int32)
    vals = synth.uniform(seed, synth.STREAM_VALS, nnz, -1.0, 1.0)
    C = synth.normal(seed, synth.STREAM_C, (N, K))
    D = synth.normal(seed, synth.STREAM_D, (N, K))
    E = synth.normal(seed, synth.STREAM_E, (N, L))
    return synth.Problem("large", N, N, K, L, rowptr.astype(np.int32), colidx, vals, C, D, E)


@pytest.mark.parametrize("K,L", [(64, 64), (128, 128)])
def test_large_input_wide_workers(gpu, K, L):
    # 300000 rows need several resident grids at these widths, so the fused
    # kernel and both unfused passes run with one 64-lane worker per wave;
    # every row and every SDDMM value is checked, and a second call must give
    # the same bits
    p = _large_problem(300_000, K, L, seed=K)
    d = upload(p)
    A = fused(d)
    check_A_rows(p, A, what="fused A")
    assert bool((fused(d) == A).all()), "fused result not deterministic"
    Y, Au = unfused(d)
    check_Y(p, Y)
    check_A_rows(p, Au, what="unfused A")


@pytest.mark.parametrize("K,L", [(64, 64), (128, 128)])
def test_large_input_wide_workers_unsorted(gpu, K, L):
    # the wide kernels on columns that are neither sorted nor distinct within
    # rows (duplicates add), and the SpMM entry point on its own; all rows
    # of a 320000-row input (above the large-input size at every kernel's
    # occupancy) are checked
    rng = np.random.default_rng(K + 1)
    p = _large_problem(320_000, K, L, seed=K + 7)
    for i in rng.choice(p.N, size=3000, replace=False):  # shuffle some rows' columns
        a, b = int(p.rowptr[i]), int(p.rowptr[i + 1])
        if b - a > 1:
            p.colidx[a:b] = rng.permutation(p.colidx[a:b])
    d = upload(p)
    check_A_rows(p, fused(d), what="fused A")
    Y, Au = unfused(d)
    check_Y(p, Y)
    check_A_rows(p, Au, what="unfused A")
    A2 = slnr.sparselnr_spmm(d["rowptr"], d["colidx"], Y, d["E"])
    assert bool((A2 == Au).all()), "sparselnr_spmm differs from the SpMM pass of the unfused call"


@pytest.mark.parametrize("K,L", [(128, 128), (16, 256)])
def test_grid_factors(gpu, K, L):
    # every grid factor the benchmark may choose (sparselnr_set_grid_factor):
    # each gives a correct, deterministic result; the SDDMM values do not
    # depend on it among the factors that launch the same kernel; 0 restores
    # the automatic choice
    p = _large_problem(120_000, K, L, seed=7 + K)
    d = upload(p)
    rows = sample_rows(p, n_random=3000)
    Y_wide = None
    try:
        for f in (1, 2, 3, 12, 48, 64):
            slnr.sparselnr_set_grid_factor(f)
            assert slnr.sparselnr_get_grid_factor() == f
            A = fused(d)
            check_A_rows(p, A, rows=rows, what="fused A, grid factor %d" % f)
            assert bool((fused(d) == A).all()), "fused not deterministic at factor %d" % f
            Y, Au = unfused(d)
            check_Y(p, Y, rows=rows)
            check_A_rows(p, Au, rows=rows, what="unfused A, grid factor %d" % f)
            if f >= 2:
                if Y_wide is None:
                    Y_wide = Y
                assert bool((Y == Y_wide).all()), "SDDMM values depend on the grid factor"
    finally:
        slnr.sparselnr_set_grid_factor(0)
    assert slnr.sparselnr_get_grid_factor() == 0
    check_A_rows(p, fused(d), rows=rows, what="fused A, automatic grid factor")


@pytest.mark.slow
def test_gathered_array_above_4gib(gpu):
    # E holds M x 256 floats with M * 256 * 4 > 2^32 bytes: the gathers need
    # 64-bit offsets, so every entry point takes the generic kernel.  Columns
    # reach the last rows of E, and one row is split over many workers.
    K, L = 16, 256
    M = (1 << 32) // (4 * L) + 4096
    lengths = power_law_lengths(3000, seed=11, scale=3.0, cap=2000)
    lengths[1500] = 30_000
    p = make_problem(lengths, M, K, L, seed=11, dups=True)
    col = p.colidx.copy()
    col[::7] = M - 1 - (np.arange(col[::7].size) % 4096)   # the rows past 4 GiB
    p = synth.Problem("above 4 GiB", p.N, M, K, L, p.rowptr, col.astype(np.int32), p.vals,
                      p.C, p.D, p.E)
    assert M * L * 4 >= 1 << 32 and int(col.max()) == M - 1
    d = upload(p)
    check_A_rows(p, fused(d), what="fused A, E above 4 GiB")
    Y, Au = unfused(d)
    check_Y(p, Y)
    check_A_rows(p, Au, what="unfused A, E above 4 GiB")


@pytest.mark.parametrize("L", [16, 32, 512, 12])
def test_one_dense_row_spmm_widths(gpu, L):
    # the SpMM alone on one row split over every worker, at the narrowest and
    # widest fast widths and at a width with no fast variant
    import torch
    p = make_problem([0, 60_000, 3], 60_000, 4, L, seed=L, dense="normal")
    d = upload(p)
    Y = torch.from_numpy(np.ascontiguousarray(p.vals)).to(gpu)
    A = slnr.sparselnr_spmm(d["rowptr"], d["colidx"], Y, d["E"])
    ref, scale, _ = oracle.spmm(p.rowptr, p.colidx, p.vals, p.E, Yabs=np.abs(p.vals))
    assert_rows_close(A.cpu().numpy(), ref, scale)


@pytest.mark.parametrize("K,L", [(32, 32), (128, 128)])
def test_one_nonzero_rows_and_rectangular(gpu, K, L):
    p = make_problem(np.ones(5000, np.int64), 77, K, L, seed=4)   # N != M
    d = upload(p)
    check_A_rows(p, fused(d))


def test_K1_L1_and_K0(gpu):
    lengths = power_law_lengths(500, seed=9, cap=300)
    for K, L in [(1, 1), (1, 64), (64, 1)]:
        p = make_problem(lengths, 400, K, L, seed=K + 2 * L)
        check_A_rows(p, fused(upload(p)))
    p = make_problem(lengths, 400, 0, 32)
    A = fused(upload(p))
    assert bool((A == 0).all())


def test_misaligned_operands_take_the_generic_path(gpu):
    import torch
    lengths = power_law_lengths(700, seed=10, cap=500)
    p = make_problem(lengths, 300, 32, 32, seed=11)
    d = upload(p)
    # views starting one float into a buffer: 4-byte aligned, not 16-byte aligned
    def shifted(a):
        buf = torch.empty(a.numel() + 1, dtype=a.dtype, device=a.device)
        v = buf[1:].view(a.shape)
        v.copy_(a)
        return v
    C, D, E = shifted(d["C"]), shifted(d["D"]), shifted(d["E"])
    A = shifted(torch.zeros(p.N, 32, device=gpu))
    slnr.sparselnr_fused_sddmm_spmm(d["rowptr"], d["colidx"], d["vals"], C, D, E, A)
    check_A_rows(p, A)


# ------------------------------------------------------------ invariants

def test_deterministic_bit_exact(gpu):
    p = make_problem(power_law_lengths(4000, seed=12, cap=8000), 3000, 128, 128, seed=12)
    d = upload(p)
    A1 = fused(d).clone()
    A2 = fused(d)
    assert bool(torch_equal(A1, A2))
    Y1, Au1 = unfused(d)
    Y1, Au1 = Y1.clone(), Au1.clone()
    Y2, Au2 = unfused(d)
    assert bool(torch_equal(Y1, Y2)) and bool(torch_equal(Au1, Au2))


@pytest.mark.parametrize("K,L,factors", [(32, 32, (1, 2, 7, 64)), (64, 64, (2, 7, 64))])
def test_short_rows_of_small_inputs_are_never_split(gpu, K, L, factors):
    """An input with fewer than 16 merge-path items per worker takes 16-item
    slices, and no slice boundary splits a row of at most 16 nonzeros: every
    row is summed by one worker in nonzero order whatever the grid factor, so
    the factors that launch the same lane mapping give bit-identical A (and
    every factor matches the oracle).  At K = L = 32 every factor keeps the
    8-lane mapping (the burst walk at one resident grid, the paced one
    above); at K = L = 64 one resident grid takes 16-lane workers and more
    take 64-lane ones."""
    rng = np.random.default_rng(41 + K)
    lengths = rng.integers(0, 17, size=3000)
    p = make_problem(lengths, 2500, K, L, seed=43 + K)
    d = upload(p)
    ref = None
    try:
        for f in (1,) + tuple(factors):
            slnr.sparselnr_set_grid_factor(f)
            A = fused(d).clone()
            check_A_rows(p, A, what="fused A, grid factor %d" % f)
            Y, Au = unfused(d)
            check_A_rows(p, Au, what="unfused A, grid factor %d" % f)
            if f in factors:
                if ref is None:
                    ref = (A, Au.clone())
                assert bool(torch_equal(A, ref[0])), "fused A differs at grid factor %d" % f
                assert bool(torch_equal(Au, ref[1])), "unfused A differs at grid factor %d" % f
    finally:
        slnr.sparselnr_set_grid_factor(0)


def torch_equal(a, b):
    import torch
    return torch.equal(a.view(torch.int32), b.view(torch.int32))


def test_zero_B_and_power_of_two_scaling_bit_exact(gpu):
    p = make_problem(power_law_lengths(3000, seed=13, cap=4000), 2000, 16, 256, seed=13)
    d = upload(p)
    A = fused(d).clone()
    d2 = dict(d)
    d2["vals"] = d["vals"] * 0
    assert bool((fused(d2) == 0).all())
    for key in ["vals", "C", "D", "E"]:
        d2 = dict(d)
        d2[key] = d[key] * 2
        assert bool(torch_equal(fused(d2), A * 2)), key


def test_column_order_within_rows(gpu):
    p = make_problem(power_law_lengths(2000, seed=14, cap=3000), 1500, 64, 64, seed=14)
    d = upload(p)
    A = fused(d).cpu().numpy()
    rng = np.random.default_rng(1)
    perm = np.arange(p.nnz)
    for i in range(p.N):
        rng.shuffle(perm[p.rowptr[i]:p.rowptr[i + 1]])
    q = synth.Problem("perm", p.N, p.M, p.K, p.L, p.rowptr, p.colidx[perm], p.vals[perm],
                      p.C, p.D, p.E)
    A2 = fused(upload(q)).cpu().numpy()
    ref, scale, _ = oracle.fused_rows(p.rowptr, p.colidx, p.vals, p.C, p.D, p.E)
    assert_rows_close(A2, A, 2 * scale)


def test_validate_csr(gpu):
    import torch
    p = make_problem(power_law_lengths(300, seed=15, cap=100), 200, 8, 8)
    d = upload(p)
    assert slnr.sparselnr_validate_csr(d["rowptr"], d["colidx"], 200) == p.nnz
    bad = d["colidx"].clone()
    bad[p.nnz // 2] = 200
    with pytest.raises(slnr.SparseLNRError) as e:
        slnr.sparselnr_validate_csr(d["rowptr"], bad, 200)
    assert e.value.status == slnr.ERR_INVALID_CSR
    rp = d["rowptr"].clone()
    a, b = int(rp[5]), int(rp[6])
    rp[5] = b + 1          # rowptr[5] > rowptr[6]: decreasing
    rp[6] = a
    with pytest.raises(slnr.SparseLNRError):
        slnr.sparselnr_validate_csr(rp, d["colidx"], 200)
    short = d["colidx"][: p.nnz // 2].clone()
    with pytest.raises(slnr.SparseLNRError):
        slnr.sparselnr_validate_csr(d["rowptr"], short, 200)


def test_stream_argument_and_workspace_release(gpu):
    import torch
    p = make_problem(power_law_lengths(1000, seed=16, cap=2000), 900, 32, 32, seed=16)
    d = upload(p)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        A = slnr.sparselnr_fused_sddmm_spmm(d["rowptr"], d["colidx"], d["vals"], d["C"], d["D"],
                                            d["E"], stream=s)
    s.synchronize()
    check_A_rows(p, A)
    slnr.sparselnr_release()
    check_A_rows(p, fused(d))


def test_two_streams_in_flight(gpu):
    # each (device, stream) has its own carry workspace: calls in flight on two
    # streams at once, both with rows split over many workers, must not share
    # partial rows; every result is bit-equal to the same call run alone
    import torch
    la = power_law_lengths(3000, seed=21, cap=4000)
    la[100] = 20_000
    lb = power_law_lengths(2500, seed=22, cap=4000)
    lb[7] = 15_000
    pa = make_problem(la, 2000, 64, 64, seed=21, dups=True)
    pb = make_problem(lb, 1800, 128, 128, seed=22, dups=True)
    da, db = upload(pa), upload(pb)
    Aa_ref, Ab_ref = fused(da).clone(), fused(db).clone()
    check_A_rows(pa, Aa_ref, what="stream test A alone")
    check_A_rows(pb, Ab_ref, what="stream test B alone")
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    Aa = [torch.full_like(Aa_ref, float("nan")) for _ in range(6)]
    Ab = [torch.full_like(Ab_ref, float("nan")) for _ in range(6)]
    torch.cuda.synchronize()
    for t in range(6):
        slnr.sparselnr_fused_sddmm_spmm(da["rowptr"], da["colidx"], da["vals"], da["C"], da["D"],
                                        da["E"], A=Aa[t], stream=s1)
        slnr.sparselnr_fused_sddmm_spmm(db["rowptr"], db["colidx"], db["vals"], db["C"], db["D"],
                                        db["E"], A=Ab[t], stream=s2)
    torch.cuda.synchronize()
    for t in range(6):
        assert torch.equal(Aa[t], Aa_ref), "stream 1, call %d differs from the call alone" % t
        assert torch.equal(Ab[t], Ab_ref), "stream 2, call %d differs from the call alone" % t


def test_hip_graph_capture_and_replay(gpu):
    # once a call on a stream has sized that stream's workspace, the fused and
    # unfused calls launch kernels only, so a HIP graph can capture them; each
    # replay, with eager calls in between, must give the eager result exactly
    import torch
    lengths = power_law_lengths(3000, seed=31, cap=3000)
    lengths[5] = 12_000
    p = make_problem(lengths, 2000, 32, 32, seed=31, dups=True)
    d = upload(p)
    args = (d["rowptr"], d["colidx"], d["vals"], d["C"], d["D"], d["E"])
    s = torch.cuda.Stream()
    A = torch.empty((p.N, p.L), dtype=torch.float32, device=gpu)
    A2 = torch.empty_like(A)
    Y = torch.empty(p.nnz, dtype=torch.float32, device=gpu)
    with torch.cuda.stream(s):  # warm-up: sizes the workspace of s
        slnr.sparselnr_fused_sddmm_spmm(*args, A=A, stream=s)
        slnr.sparselnr_unfused_sddmm_spmm(*args, Y=Y, A=A2, stream=s)
    s.synchronize()
    ref, ref2, Yref = A.clone(), A2.clone(), Y.clone()
    check_A_rows(p, ref, what="eager fused")
    check_A_rows(p, ref2, what="eager unfused")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        slnr.sparselnr_fused_sddmm_spmm(*args, A=A, stream=s)
        slnr.sparselnr_unfused_sddmm_spmm(*args, Y=Y, A=A2, stream=s)
    for t in range(4):
        A.fill_(float("nan"))
        A2.fill_(float("nan"))
        Y.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(A, ref), "replay %d: fused result differs from eager" % t
        assert torch.equal(A2, ref2), "replay %d: unfused result differs from eager" % t
        assert torch.equal(Y, Yref), "replay %d: SDDMM values differ from eager" % t
        assert torch.equal(fused(d), ref), "eager call after replay %d differs" % t
        torch.cuda.synchronize()


# ------------------------------------------------- the five named workloads

@pytest.mark.parametrize("name", ["tiny", "uniform"])
def test_config_full(gpu, name):
    p = synth.config(name)
    d = upload(p)
    check_A_rows(p, fused(d), what=name + " fused")
    Y, Au = unfused(d)
    check_Y(p, Y)
    check_A_rows(p, Au, what=name + " unfused")


@pytest.mark.slow
@pytest.mark.parametrize("name", ["rmat1m", "rmat4m", "banded"])
def test_config_every_row(gpu, name):
    # Full size, every row of A and every SDDMM value (the fused and the
    # separate forms compute the same result: Section 3.1, Figure 2), at the
    # automatic grid factor and at every factor the benchmark may time (it
    # picks one per call from bench.GRID_FACTORS).  Outputs are NaN-filled
    # before each call, so a row left unwritten fails.
    import torch

    import bench
    p = synth.config(name)
    print("%s: N=%d nnz=%d K=%d L=%d" % (name, p.N, p.nnz, p.K, p.L), flush=True)
    ref, scale, Yref, Yscale = fused_reference(p, gpu)
    d = upload(p)
    A = torch.empty((p.N, p.L), dtype=torch.float32, device=gpu)
    Au = torch.empty_like(A)
    Y = torch.empty(p.nnz, dtype=torch.float32, device=gpu)
    args = (d["rowptr"], d["colidx"], d["vals"], d["C"], d["D"], d["E"])
    try:
        for f in (0,) + tuple(bench.GRID_FACTORS):
            slnr.sparselnr_set_grid_factor(f)
            what = "%s, grid factor %s" % (name, f or "automatic")
            for t in (A, Au, Y):
                t.fill_(float("nan"))
            slnr.sparselnr_fused_sddmm_spmm(*args, A=A)
            slnr.sparselnr_unfused_sddmm_spmm(*args, Y=Y, A=Au)
            w = rows_close_dev(A, ref, scale, what=what + ", fused")
            wy = rows_close_dev(Y, Yref, Yscale, what=what + ", Y")
            wu = rows_close_dev(Au, ref, scale, what=what + ", unfused")
            print("  %s: worst err/scale fused %.2e, Y %.2e, unfused %.2e" % (what, w, wy, wu),
                  flush=True)
    finally:
        slnr.sparselnr_set_grid_factor(0)
    del A, Au, Y, d, ref, scale, Yref, Yscale
    torch.cuda.empty_cache()
