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
    assert roof["peak"] == 8000.0 and roof["unit"] == "GB/s"
    assert abs(roof["frac"] - roof["achieved"] / roof["peak"]) < 1e-3
    # a model fraction above 1 is not a fraction of the HBM roofline
    assert roof["bound"] == ("hbm" if roof["frac"] <= 1.0 else "l2")
    assert "traffic_frac" in roof and "traffic_GBps" in roof
    # traffic is reported exactly when the stored counters belong to these sources
    sys.path.insert(0, ROOT)
    import bench
    stored = bench.stored_traffic(bench.workload_key("tiny", "sddmm_spmm"))
    if stored is not None:
        assert roof["traffic"] == stored["bytes_per_call"] > 0
        ms = d["ms_per_step"]
        assert abs(roof["traffic_frac"] - roof["traffic"] / (ms * 1e-3) / 8e12) < 1e-3
        ctr = d["counters"]
        assert ctr["kernel"] == stored["dominant"]
        assert ctr["l2_hit_rate"] == stored.get("l2_hit_rate")
        assert ctr["valu_busy_pct"] == stored.get("valu_busy_pct")
    else:
        assert roof["traffic"] is None and roof["traffic_frac"] is None
        assert d["counters"] is None
    cpu = d["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["value"] > 0 and cpu["cores"] >= 1
    host = cpu["host"]
    for key in ("cpu_model", "physical_cores", "logical_cpus", "cpus_available"):
        assert key in host, key
    assert host["logical_cpus"] >= 1 and host["cpus_available"] >= 1
    # the timed call's output agrees with the oracle on every row
    par = d["parity"]
    assert par["rows"] == d["config"]["N"] and par["rows_outside_tol"] == 0
    assert par["max_err_over_scale"] <= 1e-4
    ctx = d["paper_context"]
    assert ctx["fused_vs_taco_separate_64_threads"] == "0.90-1.23x"
    assert "Threadripper 3990X" in ctx["hardware"]
    assert d["unfused"]["ms_per_call"] > 0
    assert 1 <= d["launch"]["grid_factor"] <= 64
    assert d["device"]["cus"] > 0 and "gfx950" in d["device"]["arch"]
