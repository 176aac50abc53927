"""Host model of the library's merge-path work split and carry fixup.

The GPU kernels split the merged sequence (N row ends + nnz nonzeros) into
equal slices, one per worker; rows straddling slices leave head / tail
partials that a fixup kernel adds in slice order.  This test re-enacts those
rules in Python on many CSR shapes (empty rows, one huge row, rows ending
exactly on a slice boundary, more workers than items) and checks that every
nonzero is consumed exactly once, every row of A is written exactly once,
and every index stays inside its buffer, before any kernel runs on a GPU.
"""
import numpy as np
import pytest


def mp_search(rowptr, N, nnz, d):
    lo, hi = max(0, d - nnz), min(d, N)
    while lo < hi:
        mid = (lo + hi + 1) >> 1
        if rowptr[mid] + mid <= d:
            lo = mid
        else:
            hi = mid - 1
    return lo


def slice_bounds(rowptr, N, nnz, S, d, snap):
    """Merge-path coordinate of diagonal d, moved back to the row start when it
    falls inside a row of at most `snap` nonzeros."""
    i = mp_search(rowptr, N, nnz, d)
    p = d - i
    if i < N and p > rowptr[i] and rowptr[i + 1] - rowptr[i] <= snap:
        p = int(rowptr[i])
    return i, p


SHORT_SLICE = 16  # kShortSlice of the kernels
SNAP_ROW = 16     # kSnapRow of the kernels


def slice_len(items, workers, min_chunk, short=SHORT_SLICE, N=None, nnz=None):
    """The kernels' slice length: ceil(items / workers), raised to `short`
    below it when the rows average at most SNAP_ROW nonzeros (N, nnz; None:
    they do), else to min_chunk."""
    S = -(-items // workers)
    short_rows = N is None or nnz <= SNAP_ROW * N
    if S < short and short_rows:
        return short
    return max(S, min_chunk)


def snap_len(S, snap_row=SNAP_ROW):
    """Longest row a slice boundary never splits: S/4, or min(S, snap_row)
    when that is larger (short slices)."""
    return max(S // 4, min(S, snap_row))


def simulate(rowptr, workers, min_chunk, L=3, rng=None, use_snap=True, short=SHORT_SLICE):
    """Returns (A, writes) computed through the slice / carry / fixup rules."""
    N = rowptr.size - 1
    nnz = int(rowptr[N])
    items = N + nnz
    S = slice_len(items, workers, min_chunk, short, N, nnz)
    snap = snap_len(S) if use_snap else -1
    rng = rng or np.random.default_rng(0)
    contrib = rng.integers(-5, 6, size=(nnz, L)).astype(np.float64)  # y_p * E_j, exact ints
    A = np.full((N, L), np.nan)
    writes = np.zeros(N, dtype=int)
    consumed = np.zeros(nnz, dtype=int)
    carry = np.full((workers, 2, L), np.nan)
    meta = np.full((workers, 2), -7, dtype=np.int64)
    for w in range(workers):
        d0 = w * S
        if d0 >= items:
            meta[w] = (-1, -1)
            continue
        d1 = min(d0 + S, items)
        i0, p0 = slice_bounds(rowptr, N, nnz, S, d0, snap)
        i1, p1 = slice_bounds(rowptr, N, nnz, S, d1, snap)
        assert 0 <= i0 <= i1 <= N and 0 <= p0 <= p1 <= nnz
        assert rowptr[i0] <= p0 <= (rowptr[i0 + 1] if i0 < N else nnz)
        head = i0 < i1 and p0 > rowptr[i0]
        i, p = i0, p0
        while True:
            has_end = i < i1
            if not has_end and i >= N:
                break
            r_end = rowptr[i + 1] if has_end else p1
            acc = np.zeros(L)
            while p < r_end:
                assert 0 <= p < p1 <= nnz
                consumed[p] += 1
                acc += contrib[p]
                p += 1
            if not has_end:
                carry[w, 1] = acc
            elif i == i0 and head:
                carry[w, 0] = acc
            else:
                assert 0 <= i < N
                A[i] = acc
                writes[i] += 1
            if not has_end:
                break
            i += 1
        meta[w] = (i1 if i1 < N else -1, i0 if head else -1)
    # fixup
    for c in range(workers):
        r = meta[c, 1]
        if r < 0:
            continue
        first = c
        while first - 1 >= 0 and meta[first - 1, 0] == r:
            first -= 1
        s = np.zeros(L)
        for cc in range(first, c):
            assert not np.isnan(carry[cc, 1]).any(), "tail slot read before written"
            s += carry[cc, 1]
        assert not np.isnan(carry[c, 0]).any()
        s += carry[c, 0]
        A[r] = s
        writes[r] += 1
    ref = np.zeros((N, L))
    for i in range(N):
        ref[i] = contrib[rowptr[i]:rowptr[i + 1]].sum(axis=0)
    return A, writes, consumed, ref


def csr_from_lengths(lengths):
    rowptr = np.zeros(len(lengths) + 1, dtype=np.int64)
    rowptr[1:] = np.cumsum(lengths)
    return rowptr


CASES = {
    "uniform": [10] * 50,
    "empty": [0] * 17,
    "one_huge": [0, 3, 1000, 0, 2],
    "power_law": [int(x) for x in (np.random.default_rng(1).pareto(1.2, 300) * 3)],
    "mixed_empty": [0, 0, 5, 0, 0, 0, 64, 1, 0, 33, 0],
    "single_row": [257],
    "single_empty": [0],
}


@pytest.mark.parametrize("short", [1, SHORT_SLICE])
@pytest.mark.parametrize("use_snap", [True, False])
@pytest.mark.parametrize("name", sorted(CASES))
@pytest.mark.parametrize("workers,min_chunk", [(1, 1), (3, 1), (7, 2), (64, 1), (64, 32),
                                                (1000, 1), (5, 1000), (40, 8), (1000, 64)])
def test_every_row_once(name, workers, min_chunk, use_snap, short):
    rowptr = csr_from_lengths(CASES[name])
    A, writes, consumed, ref = simulate(rowptr, workers, min_chunk, use_snap=use_snap,
                                        short=short)
    assert np.all(consumed == 1)
    assert np.all(writes == 1)
    assert np.array_equal(A, ref)


def test_slice_length_rule():
    # fewer than 16 items per worker: 16-item slices; 16 to 64: 64; above: the quotient
    assert slice_len(22528, 32768, 64) == 16      # 2048 rows of 10 nonzeros
    assert slice_len(1114112, 32768, 64) == 64    # 65536 rows of 16 nonzeros, 34 per worker
    assert slice_len(1114112, 16384, 64) == 68
    assert slice_len(15 * 100, 100, 64) == 16
    assert slice_len(16 * 100, 100, 64) == 64
    # rows averaging more than 16 nonzeros (a hub row) keep 64-item slices
    assert slice_len(22528, 32768, 64, N=2048, nnz=20480) == 16
    assert slice_len(2048 + 32768, 32768, 64, N=2048, nnz=32768) == 16
    assert slice_len(2048 + 32769, 32768, 64, N=2048, nnz=32769) == 64
    assert slice_len(1000 + 108000, 32768, 64, N=1000, nnz=108000) == 64
    assert [snap_len(S) for S in (1, 7, 16, 63, 64, 68, 1000)] == [1, 7, 16, 16, 16, 17, 250]


@pytest.mark.parametrize("workers", [300, 3000, 30000])
def test_snapping_splits_only_long_rows(workers):
    lengths = [int(x) for x in (np.random.default_rng(2).pareto(1.2, 2000) * 3)]
    rowptr = csr_from_lengths(lengths)
    N, nnz = len(lengths), int(rowptr[-1])
    S = slice_len(N + nnz, workers, 64, N=N, nnz=nnz)
    snap = snap_len(S)
    assert snap <= S
    for w in range(1, -(-(N + nnz) // S)):
        i, p = slice_bounds(rowptr, N, nnz, S, w * S, snap)
        if i < N and p > rowptr[i]:
            assert rowptr[i + 1] - rowptr[i] > snap


def test_short_slices_keep_short_rows_whole():
    # 2048 rows of 10 nonzeros on 32768 workers: 16-item slices, no partial rows
    rowptr = csr_from_lengths([10] * 2048)
    N, nnz = 2048, int(rowptr[-1])
    S = slice_len(N + nnz, 32768, 64, N=N, nnz=nnz)
    assert S == 16
    ns = -(-(N + nnz) // S)
    prev = (0, 0)
    for w in range(1, ns + 1):
        i, p = slice_bounds(rowptr, N, nnz, S, min(w * S, N + nnz), snap_len(S))
        assert p == rowptr[i]  # every boundary at a row start
        assert (i, p) > prev or (i, p) == (N, nnz)  # no empty slice
        prev = (i, p)


def test_rows_ending_on_slice_boundaries():
    # every slice boundary lands exactly on a row end, on a row start, or mid-row
    for S in range(1, 12):
        lengths = [S - 1, S, 2 * S, 0, 0, S + 1, 1]
        rowptr = csr_from_lengths(lengths)
        items = len(lengths) + rowptr[-1]
        workers = -(-items // S)
        for use_snap in (True, False):
            A, writes, consumed, ref = simulate(rowptr, workers, 1, use_snap=use_snap, short=1)
            assert np.all(consumed == 1) and np.all(writes == 1) and np.array_equal(A, ref)


def mp_search2_wide(rowptr, N, nnz, da, db, G):
    """Host model of the kernels' paired search: both diagonals advance in
    the same steps, each by the rule of mp_search_wide."""
    ra, sa = mp_search_wide(rowptr, N, nnz, da, G)
    rb, sb = mp_search_wide(rowptr, N, nnz, db, G)
    return ra, rb, max(sa, sb)


def mp_search_wide(rowptr, N, nnz, d, G):
    """Host model of the kernel's G-lane search: G probes per step, keep the
    sub-interval the ballot points to."""
    lo, hi = max(0, d - nnz), min(d, N)
    steps = 0
    while lo < hi:
        step = -(-(hi - lo) // G)
        xs = [min(hi, lo + (t + 1) * step) for t in range(G)]
        ok = [rowptr[x] + x <= d for x in xs]
        m = 0
        while m < G and ok[m]:
            m += 1
        assert all(ok[:m]) and not any(ok[m:]), "probe results must be monotone"
        xm1, xm = lo + m * step, lo + (m + 1) * step
        new_lo = min(xm1, hi) if m > 0 else lo
        new_hi = min(xm, hi) - 1 if m < G else hi
        lo, hi = new_lo, new_hi
        steps += 1
        assert steps < 64
    return lo, steps


@pytest.mark.parametrize("G", [4, 8, 16, 32, 64])
@pytest.mark.parametrize("name", sorted(CASES))
def test_wide_search_matches_bisection(G, name):
    rowptr = csr_from_lengths(CASES[name])
    N, nnz = rowptr.size - 1, int(rowptr[-1])
    for d in range(N + nnz + 1):
        got, steps = mp_search_wide(rowptr, N, nnz, d, G)
        assert got == mp_search(rowptr, N, nnz, d), (d, G)
        assert rowptr[got] <= d - got <= (rowptr[got + 1] if got < N else nnz)


@pytest.mark.parametrize("G", [4, 8, 64])
def test_paired_search_matches_two_searches(G):
    rowptr = csr_from_lengths(CASES["power_law"])
    N, nnz = rowptr.size - 1, int(rowptr[-1])
    for S in (1, 7, 16, 64):
        for d0 in range(0, N + nnz + 1, S):
            d1 = min(d0 + S, N + nnz)
            a, b, steps = mp_search2_wide(rowptr, N, nnz, d0, d1, G)
            assert (a, b) == (mp_search(rowptr, N, nnz, d0), mp_search(rowptr, N, nnz, d1))
            assert a <= b


def test_wide_search_step_count():
    rowptr = csr_from_lengths([16] * (1 << 20))
    N, nnz = rowptr.size - 1, int(rowptr[-1])
    for d in [0, 1, 12345, N + nnz // 2, N + nnz]:
        _, steps = mp_search_wide(rowptr, N, nnz, d, 32)
        assert steps <= 5


@pytest.mark.parametrize("blocks,wpb,ns", [(8, 8, 1), (8, 8, 64), (16, 2, 31), (24, 16, 383),
                                           (64, 4, 256), (8, 1, 8), (40, 16, 7)])
def test_xcd_slice_assignment_is_a_bijection(blocks, wpb, ns):
    """XCD x (blocks dealt round-robin over 8 XCDs) takes slices
    [x * ceil(ns/8), (x+1) * ceil(ns/8)); every slice < ns has one worker."""
    xcds = 8
    workers = blocks * wpb
    assert ns <= workers
    per_xcd = -(-ns // xcds)
    seen = []
    for b in range(blocks):
        for local in range(wpb):
            xcd, in_xcd = b % xcds, (b // xcds) * wpb + local
            sid = xcd * per_xcd + in_xcd
            if in_xcd < per_xcd and sid < ns:
                seen.append(sid)
    assert sorted(seen) == list(range(ns))


def fixup_shape(cus, workers):
    """Host model of the library's fixup_shape()."""
    max_waves = cus * 32
    G = 8
    while G < 64 and -(-workers // G) > max_waves:
        G *= 2
    waves = -(-workers // G)
    blocks = min(-(-waves // 4), max_waves // 4)
    return max(blocks, 1), G


@pytest.mark.parametrize("ns,workers,cus", [(1, 64, 256), (63, 64, 1), (64, 64, 1), (65, 128, 1),
                                            (352, 65536, 256), (65536, 65536, 256),
                                            (1000, 262144, 256), (131072, 131072, 4),
                                            (129, 200, 1), (5000, 5000, 2)])
def test_fixup_groups_visit_each_head_once(ns, workers, cus):
    """Host model of carry_fixup's iteration: with G slices per group, wave w
    takes the groups starting at w*G, (w + waves)*G, ...; within a group it
    visits the slices whose head entry is set, in ascending order.  Every
    head slice below ns is visited exactly once and no slice >= ns is read."""
    blocks, G = fixup_shape(cus, workers)
    assert G in (8, 16, 32, 64) and blocks * 4 <= max(cus * 32, 4)
    waves = blocks * 4
    rng = np.random.default_rng(ns * 7 + workers)
    head = np.full(workers + 64, -1)
    head[:ns] = np.where(rng.random(ns) < 0.3, rng.integers(0, 1000, ns), -1)
    head[ns:] = 5  # stale entries of earlier calls: must never be used
    visits = np.zeros(workers + 64, dtype=int)
    for w in range(waves):
        g0 = w * G
        while g0 < ns:
            flags = [lane < G and (g0 + lane < ns) and head[g0 + lane] >= 0 for lane in range(64)]
            for b in range(64):
                if flags[b]:
                    visits[g0 + b] += 1
            g0 += waves * G
    assert np.array_equal(visits[:ns], (head[:ns] >= 0).astype(int))
    assert not visits[ns:].any()
