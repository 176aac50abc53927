#!/usr/bin/env python3
"""Benchmark of the fused SDDMM->SpMM hot path on one MI355X.

    python bench.py [--steps K] [--warmup W] [--config rmat1m]

One step is one call of sparselnr_fused_sddmm_spmm over the whole matrix
(merge-path walk kernel + carry fixup kernel), inputs resident in HBM.  The
default workload is the R-MAT graph with 2^20 vertices, 16 edges per vertex
drawn (duplicates merged, 16,085,851 nonzeros), K = L = 128, seed 0.

Prints ONE JSON line with throughput (Gnnz/s), the roofline of the fused
call against MI355X HBM peak (algorithmic bytes of the fused schedule:
CSR arrays + one gathered D row and E row per nonzero + C and A streams),
the in-library unfused comparison, and the CPU oracle timed on the host.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, published
METRIC = "fused SDDMM→SpMM Gnnz/s + achieved HBM GB/s vs peak, R-MAT 1M rows K=L=128"
KERNEL_SOURCES = ["paper_2205_11622_amd/csrc/walker.hpp", "paper_2205_11622_amd/csrc/sparselnr.hip"]


def source_digest() -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def stored_traffic(config: str):
    """HBM traffic per fused call from committed rocprofv3 counter runs, only
    if they were taken on the kernel sources as they are now."""
    path = os.path.join(ROOT, "profiles", "traffic_%s.json" % config)
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        t = json.load(fh)
    if t.get("source_digest") != source_digest():
        return None
    return t


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="rmat1m")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-unfused", action="store_true")
    ap.add_argument("--copy-probe", action="store_true",
                    help="after timing, run three plain 1 GiB device copies (torch copy_), the "
                         "reference for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE readings")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on exactly one GPU: the fused kernel shards by rows with no "
              "communication, and this build measures one GPU's share only (--gpus 1).",
              file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import paper_2205_11622_amd as slnr
    import synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    dev = torch.device("cuda:0")
    t0 = time.time()
    p = synth.config(args.config)
    gen_s = time.time() - t0
    print("# %s: N=%d nnz=%d K=%d L=%d (generated in %.1fs)" % (args.config, p.N, p.nnz, p.K, p.L,
                                                                gen_s), file=sys.stderr, flush=True)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    rowptr, colidx, vals, C, D, E = (t(x) for x in (p.rowptr, p.colidx, p.vals, p.C, p.D, p.E))
    A = torch.empty((p.N, p.L), dtype=torch.float32, device=dev)
    Y = torch.empty(p.nnz, dtype=torch.float32, device=dev)
    A2 = torch.empty_like(A)
    stream = torch.cuda.current_stream(dev)

    def fused():
        slnr.sparselnr_fused_sddmm_spmm(rowptr, colidx, vals, C, D, E, A, stream=stream)

    def unfused():
        slnr.sparselnr_unfused_sddmm_spmm(rowptr, colidx, vals, C, D, E, Y, A2, stream=stream)

    def timed(fn, steps, warmup):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        t_start = time.perf_counter()
        ev[0].record(stream)
        for s in range(steps):
            fn()
            ev[s + 1].record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t_start
        per = np.array([ev[s].elapsed_time(ev[s + 1]) for s in range(steps)])
        return per, ev[0].elapsed_time(ev[steps]), wall

    per, total_ms, wall = timed(fused, args.steps, args.warmup)
    ms = total_ms / args.steps
    print("# fused: %.4f ms/call (median %.4f, min %.4f, max %.4f)"
          % (ms, np.median(per), per.min(), per.max()), file=sys.stderr, flush=True)
    unf = None
    if not args.no_unfused:
        uper, utotal, _ = timed(unfused, args.steps, args.warmup)
        # interleave a second fused round so both see the same machine state
        per2, total2, _ = timed(fused, args.steps, 1)
        unf = {"ms_per_call": utotal / args.steps, "median_ms": float(np.median(uper)),
               "fused_ms_rerun": total2 / args.steps,
               "fused_speedup": (utotal / args.steps) / ms}
        print("# unfused: %.4f ms/call; fused rerun %.4f ms" % (unf["ms_per_call"],
                                                               unf["fused_ms_rerun"]),
              file=sys.stderr, flush=True)

    if args.copy_probe:
        src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    nnz = p.nnz
    model_bytes = p.model_bytes()
    gnnz = nnz / (ms * 1e-3) / 1e9
    achieved = model_bytes / (ms * 1e-3) / 1e9
    traffic = stored_traffic(args.config)
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                "traffic": traffic["bytes_per_call"] if traffic else None,
                "kernel": "walk_fast fused + carry_fixup (one call)",
                "bytes_per_call": model_bytes,
                "bytes_model": "4(N+1) + 8 nnz + 4 nnz (K+L) + 4 N K + 4 N L"}

    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        rows = np.arange(p.N, dtype=np.int64)
        t1 = time.perf_counter()
        oracle.fused_rows(p.rowptr, p.colidx, p.vals, p.C, p.D, p.E, rows=rows)
        cs = time.perf_counter() - t1
        cpu = {"value": round(nnz / cs / 1e9, 6), "unit": "Gnnz/s", "cores": oracle.num_threads(),
               "kind": "oracle", "seconds": round(cs, 3),
               "sample": "the whole %s workload (%d rows, %d nonzeros), one pass, fp64 "
                         "accumulation, OpenMP over rows" % (args.config, p.N, nnz)}

    out = {
        "metric": METRIC, "value": round(gnnz, 4), "unit": "Gnnz/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "%s: %s" % (args.config, synth.CONFIGS[args.config]["desc"]),
                   "N": p.N, "M": p.M, "nnz": nnz, "K": p.K, "L": p.L, "seed": 0},
        "roofline": roofline, "cpu_baseline": cpu,
        "achieved_GBps": round(achieved, 1),
        "median_ms": round(float(np.median(per)), 5), "wall_s": round(wall, 3),
        "unfused": unf, "source_digest": source_digest(),
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
