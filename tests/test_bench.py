"""bench.py's contract on the host (no GPU needed): one GPU only, a loud
failure without a GPU, and the byte model it prices."""
import os
import subprocess
import sys

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


def run(args, env=None):
    e = dict(os.environ)
    e.update(env or {})
    return subprocess.run([sys.executable, BENCH] + args, capture_output=True, text=True,
                          timeout=600, cwd=ROOT, env=e)


def test_more_than_one_gpu_is_refused():
    r = run(["--gpus", "2"])
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    r = run([], env={"WORLD_SIZE": "2"})
    assert r.returncode == 2


def test_no_gpu_fails_loudly():
    import torch
    if torch.cuda.is_available():
        return
    r = run(["--steps", "1", "--warmup", "0", "--no-cpu-baseline"])
    assert r.returncode != 0
    assert "needs a GPU" in r.stderr
    assert r.stdout.strip() == ""  # no JSON line without a measurement


def test_help_lists_the_launch_and_cache_options():
    r = run(["--help"])
    assert r.returncode == 0
    for opt in ("--grid-factor", "--compare-grid-factor", "--cold", "--kernel", "--config"):
        assert opt in r.stdout


def test_byte_model_matches_its_formula():
    # 4(N+1) + 8 nnz + 4 nnz (K+L) + 4 N K + 4 N L on the tiny workload
    p = synth.config("tiny")
    N, K, L, nnz = p.N, p.K, p.L, p.nnz
    assert nnz == 20480
    assert p.model_bytes() == 4 * (N + 1) + 8 * nnz + 4 * nnz * (K + L) + 4 * N * K + 4 * N * L


def test_row_parity_rule_of_the_bench_line():
    """bench.row_parity applies the tests' per-row rule (tests/parity.py)."""
    import numpy as np

    import bench
    from tests.parity import row_errors
    rng = np.random.default_rng(4)
    ref = rng.standard_normal((500, 6))
    scale = np.abs(ref).max(axis=1) * 1.5
    got = (ref * (1 + 1e-6 * rng.standard_normal(ref.shape))).astype(np.float32)
    scale[:4] = 0.0
    ref[:4] = 0.0
    got[:3] = 0.0
    got[3, 0] = 1e-20          # nonzero in a zero-scale row
    got[9, 2] = np.nan
    got[17] += 1e-3 * scale[17]
    worst, bad = bench.row_parity(got, ref, scale, chunk=64)
    _, ratio = row_errors(got, ref, scale)
    assert bad == int((~(ratio <= 1e-4)).sum()) == 3
    assert worst == np.inf
    worst_ok, bad_ok = bench.row_parity(got[20:], ref[20:], scale[20:], chunk=64)
    assert bad_ok == 0 and worst_ok == ratio[20:].max()
