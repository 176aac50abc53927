"""bench.py end to end on the GPU: one JSON line with the fields the
benchmark contract names (tiny workload, a few steps)."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_json_line(gpu):
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--config", "tiny",
                        "--steps", "5", "--warmup", "1"],
                       capture_output=True, text=True, timeout=480, cwd=ROOT)
    print(r.stderr[-2000:], flush=True)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1, r.stdout
    d = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
                "roofline", "cpu_baseline", "unfused", "launch"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 5 and d["warmup"] == 1
    assert d["value"] > 0 and d["ms_per_step"] > 0 and d["unit"] == "Gnnz/s"
    assert d["config"]["workload"].startswith("tiny")
    roof = d["roofline"]
    assert roof["bound"] == "hbm" and roof["peak"] == 8000.0 and roof["unit"] == "GB/s"
    assert abs(roof["frac"] - roof["achieved"] / roof["peak"]) < 1e-3
    # traffic is reported exactly when the stored counters belong to these sources
    sys.path.insert(0, ROOT)
    import bench
    stored = bench.stored_traffic(bench.workload_key("tiny", "sddmm_spmm"))
    if stored is not None:
        assert roof["traffic"] == stored["bytes_per_call"] > 0
    else:
        assert roof["traffic"] is None
    cpu = d["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["value"] > 0 and cpu["cores"] >= 1
    assert d["unfused"]["ms_per_call"] > 0
    assert 1 <= d["launch"]["grid_factor"] <= 64
    assert d["device"]["cus"] > 0 and "gfx950" in d["device"]["arch"]
