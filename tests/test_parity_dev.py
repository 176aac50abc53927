"""The device form of the parity rule (tests/gpu_util.py: row_ratios_dev,
rows_close_dev), used by the full-size GPU tests, agrees with the host form
(tests/parity.py) row for row.  Runs on CPU tensors."""
import numpy as np
import pytest

from tests.gpu_util import oracle_reference, row_ratios_dev, rows_close_dev
from tests.parity import row_errors


def _case(seed, n=300, L=9):
    rng = np.random.default_rng(seed)
    ref = rng.standard_normal((n, L))
    scale = np.abs(ref).max(axis=1) * rng.uniform(0.5, 2.0, n)
    got = (ref + rng.standard_normal((n, L)) * 1e-5 * scale[:, None]).astype(np.float32)
    scale[:7] = 0.0                          # zero-scale rows
    ref[:7] = 0.0
    got[:3] = 0.0                            # ... exact zeros pass
    got[3, 1] = 1e-30                        # ... anything else fails
    got[10, 4] = np.nan                      # non-finite rows fail
    got[11, 0] = np.inf
    got[20] += 1e-3 * scale[20]              # outside the tolerance
    return got, ref, scale


@pytest.mark.parametrize("seed", [0, 1])
def test_device_rule_matches_host_rule(seed):
    import torch
    got, ref, scale = _case(seed)
    _, host = row_errors(got, ref, scale)
    dev, _ = row_ratios_dev(torch.from_numpy(got), torch.from_numpy(ref), torch.from_numpy(scale))
    dev = dev.numpy()
    assert np.array_equal(np.isinf(host), np.isinf(dev))
    fin = np.isfinite(host)
    assert np.allclose(host[fin], dev[fin], rtol=1e-12, atol=0)
    assert np.array_equal(host <= 1e-4, dev <= 1e-4)


def test_rows_close_dev_names_the_bad_rows():
    import torch
    got, ref, scale = _case(2)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))  # noqa: E731
    with pytest.raises(AssertionError, match="outside"):
        rows_close_dev(t(got), t(ref), t(scale), chunk=64)
    ok = slice(30, 300)
    w = rows_close_dev(t(got[ok]), t(ref[ok]), t(scale[ok]), chunk=64)
    assert 0 < w <= 1e-4


def test_vector_form_for_sddmm_values():
    import torch
    ref = np.array([1.0, -2.0, 0.0, 3.0])
    scale = np.array([1.0, 2.0, 0.0, 3.0])
    got = np.array([1.0, -2.0, 0.0, 3.0 + 1e-3], dtype=np.float32)
    r, _ = row_ratios_dev(torch.from_numpy(got), torch.from_numpy(ref), torch.from_numpy(scale))
    assert np.array_equal(r.numpy() <= 1e-4, [True, True, True, False])


def test_chunked_reference_matches_one_pass():
    """oracle_reference stitches chunks into the same arrays as one oracle pass."""
    import torch

    import oracle
    from tests.gpu_util import make_problem, power_law_lengths
    p = make_problem(power_law_lengths(1000, seed=3, cap=300), 700, 8, 12, seed=3)
    A, s, Y, Ys, _ = oracle.fused_rows(p.rowptr, p.colidx, p.vals, p.C, p.D, p.E, with_y=True)
    got = oracle_reference(
        lambda rows: oracle.fused_rows(p.rowptr, p.colidx, p.vals, p.C, p.D, p.E, rows=rows,
                                       with_y=True)[:4], p.N, p.L, torch.device("cpu"),
        nnz_of=p.rowptr, chunk=97)
    for a, b in zip(got, (A, s, Y, Ys)):
        assert np.array_equal(a.numpy(), b)
