#!/usr/bin/env python3
"""Benchmark of the fused SDDMM->SpMM hot path on one MI355X.

    python bench.py [--steps K] [--warmup W] [--config rmat1m] [--kernel sddmm_spmm]

One step is one library call over the whole matrix (merge-path walk kernel +
carry fixup kernel), inputs resident in HBM.  Before the timed region the
library's grid factor (resident grids per walk launch) is chosen per call:
the timed call and each pass of the comparison run at the fastest of a fixed
candidate list (--grid-factor / --compare-grid-factor fix them instead).  The default is
sparselnr_fused_sddmm_spmm on the R-MAT graph with 2^20 vertices, 16 edges
per vertex drawn (duplicates merged, 16,085,851 nonzeros), K = L = 128,
seed 0.

Prints ONE JSON line with throughput (Gnnz/s), the roofline of the call
against MI355X HBM peak (algorithmic bytes of the fused schedule: CSR arrays
+ the gathered dense rows per nonzero + the dense row streams), an in-run
comparison with the same result computed in separate passes, and the CPU
oracle timed on the host.

--kernel picks one of the further computations of the paper's Section 6.2
instead, each on the --config sparsity structure at the inner sizes the
paper uses for it:

  sddmm_spmm_gemm  A = ((B .* C D^T) F) W,  K = L = Mo = 64
  spmm_gemm        A = (B C) D,             C is M x 128, D is 128 x 64
  spmmh_gemm       A = (B (C .* D)) E,      C, D are M x 128, E is 128 x 128
  dt               <SDDMM, SpMM> with D stored transposed (K x M), K = L = 128

--sweep instead prints one JSON line per (K, L) in {16, 32, 64, 128, 256,
512}^2 on the --config sparsity structure, the fused call against the
separate passes: with --kernel spmm_gemm, SpMM into an N x K temporary then
torch.mm (the inner-size study of the paper's Section 6.3, Figure 8); with
--kernel sddmm_spmm, the library's unfused SDDMM then SpMM.
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
KERNEL_SOURCES = ["paper_2205_11622_amd/csrc/walker.hpp", "paper_2205_11622_amd/csrc/epilogue.hpp",
                  "paper_2205_11622_amd/csrc/sparselnr.hip"]
KERNELS = ("sddmm_spmm", "sddmm_spmm_gemm", "spmm_gemm", "spmmh_gemm", "dt")
CPU_SECONDS = 10.0  # oracle passes are repeated until about this much wall time
# Grid factors (resident grids per walk launch) tried for each library call
# before the timed region; the timed call and each pass of the comparison run
# at their own fastest one.
GRID_FACTORS = (1, 2, 4, 8, 12, 16, 24, 32, 48, 64)
TUNE_CALLS = 5
# Untimed, waited-for calls before each timed region, in seconds of wall time.
SETTLE_S = 0.05
SMALL_CONFIGS = ("tiny", "uniform")  # calls of tens of microseconds: more timed calls by default
SMALL_STEPS = 200


def source_digest() -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def workload_key(config: str, kernel: str) -> str:
    return config if kernel == "sddmm_spmm" else "%s_%s" % (config, kernel)


def stored_traffic(key: str):
    """HBM traffic per call from committed rocprofv3 counter runs, only if they
    were taken on the kernel sources as they are now."""
    path = os.path.join(ROOT, "profiles", "traffic_%s.json" % key)
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        t = json.load(fh)
    if t.get("source_digest") != source_digest():
        return None
    return t


def device_info(dev) -> dict:
    """The GPU the line was measured on (boxes of one model differ by up to 15%)."""
    import torch
    p = torch.cuda.get_device_properties(dev)
    return {"name": p.name, "arch": getattr(p, "gcnArchName", ""), "cus": p.multi_processor_count,
            "memory_GiB": round(p.total_memory / 2 ** 30, 1)}


def host_info() -> dict:
    """The host the CPU baseline ran on: lscpu's model and socket / core /
    thread counts, and the CPUs this process may use."""
    import subprocess
    info = {"cpu_model": None, "sockets": None, "physical_cores": None, "threads_per_core": None,
            "logical_cpus": os.cpu_count(), "cpus_available": len(os.sched_getaffinity(0))}
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        kv = dict(l.split(":", 1) for l in out.splitlines() if ":" in l)
        kv = {k.strip(): v.strip() for k, v in kv.items()}
        info["cpu_model"] = kv.get("Model name")
        sockets = int(kv["Socket(s)"]) if kv.get("Socket(s)", "").isdigit() else None
        cps = int(kv["Core(s) per socket"]) if kv.get("Core(s) per socket", "").isdigit() else None
        tpc = int(kv["Thread(s) per core"]) if kv.get("Thread(s) per core", "").isdigit() else None
        info.update(sockets=sockets, threads_per_core=tpc,
                    physical_cores=sockets * cps if sockets and cps else None)
    except (OSError, ValueError, KeyError, subprocess.SubprocessError):
        pass
    if info["cpu_model"] is None:
        try:
            with open("/proc/cpuinfo") as fh:
                for line in fh:
                    if line.startswith("model name"):
                        info["cpu_model"] = line.split(":", 1)[1].strip()
                        break
        except OSError:
            pass
    return info


# The paper's own results for each computation (Section 6.1 setup, Section
# 6.2 results), quoted as context: other hardware, the paper's matrices, TACO
# baselines.  Not a target and not comparable to the GPU figures.
PAPER_HARDWARE = ("1x AMD Ryzen Threadripper 3990X (64 cores, 2.2 GHz, 16 MB L3); GCC 7.5 -O3 "
                  "-ffast-math; OpenMP 4.5, 64 threads for multi-thread runs; double precision; "
                  "TACO-generated C (Section 6.1)")
PAPER_CONTEXT = {
    "sddmm_spmm": {"computation": "<SDDMM,SpMM>, K = L = 64 (Section 6.2)",
                   "fused_vs_taco_separate_64_threads": "0.90-1.23x",
                   "fused_vs_taco_separate_1_thread": "0.91-1.50x",
                   "fused_vs_taco_original_64_threads": "3.31-16.05x",
                   "fused_vs_taco_original_1_thread": "10.75-33.39x",
                   "wins_over_separate_on": "the matrices with the most nonzeros (circuit5M, "
                                            "shipsec1, consph, pdb1HYS, cant)"},
    "sddmm_spmm_gemm": {"computation": "<SDDMM,SpMM,GEMM>, K = L = M = 64 (Section 6.2)",
                        "fused_vs_taco_separate_64_threads": "1.06-2.09x",
                        "fused_vs_taco_separate_1_thread": "1.20-2.26x"},
    "spmm_gemm": {"computation": "<SpMM,GEMM>, inner sizes 128 and 64 (Section 6.2)",
                  "note": "the text's assignment of its two speedup ranges to the two baselines "
                          "is garbled; see the paper's abstract and Section 6.2"},
    "spmmh_gemm": {"computation": "<SpMMH,GEMM>, J = L = 128 (Section 6.2)",
                   "fused_vs_taco_separate_64_threads": "1.28-2.40x",
                   "fused_vs_taco_separate_1_thread": "1.60-1.99x"},
    "dt": {"computation": "<SDDMM,SpMM> with D transposed (Section 4.3.1)",
           "note": "the paper prints no separate figure for this layout"},
}


def row_parity(got, ref, scale, tol=1e-4, chunk=65536):
    """Worst per-row ratio max_l |A_il - Aref_il| / scale_i over every row (a
    row of zero scale must be exactly zero; a non-finite value fails), and
    the number of rows outside tol."""
    import numpy as np
    worst, bad = 0.0, 0
    for r0 in range(0, got.shape[0], chunk):
        g = got[r0:r0 + chunk].astype(np.float64)
        r = ref[r0:r0 + chunk]
        s = scale[r0:r0 + chunk]
        err = np.abs(g - r).max(axis=1) if g.shape[1] else np.zeros(g.shape[0])
        with np.errstate(divide="ignore", invalid="ignore"):
            ratio = np.where(s > 0, err / np.where(s > 0, s, 1.0),
                             np.where(err == 0, 0.0, np.inf))
        ratio = np.where(np.isfinite(g).all(axis=1), ratio, np.inf)
        bad += int((~(ratio <= tol)).sum())
        worst = max(worst, float(np.where(np.isnan(ratio), np.inf, ratio).max(initial=0.0)))
    return worst, bad


def make_workload(kernel, config, dev):
    """Inputs on the device, the timed call, the comparison call, the byte model
    and the oracle leg for one kernel."""
    import numpy as np
    import torch

    import paper_2205_11622_amd as slnr
    import synth

    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    stream = torch.cuda.current_stream(dev)
    base = synth.config(config)
    N, M, nnz = base.N, base.M, base.nnz
    rp, ci, v = t(base.rowptr), t(base.colidx), t(base.vals)
    w = {"N": N, "M": M, "nnz": nnz, "seed": 0}
    desc = "%s: %s" % (config, synth.CONFIGS[config]["desc"])
    csr_bytes = 4 * (N + 1) + 8 * nnz

    if kernel == "sddmm_spmm":
        p = base
        C, D, E = t(p.C), t(p.D), t(p.E)
        A = torch.empty((N, p.L), dtype=torch.float32, device=dev)
        Y = torch.empty(nnz, dtype=torch.float32, device=dev)
        A2 = torch.empty_like(A)
        w.update(K=p.K, L=p.L)
        return dict(
            metric=METRIC if config == "rmat1m" else
            "fused SDDMM→SpMM Gnnz/s + achieved HBM GB/s vs peak, %s K=%d L=%d" % (config, p.K, p.L),
            desc=desc, sizes=w,
            call=lambda: slnr.sparselnr_fused_sddmm_spmm(rp, ci, v, C, D, E, A, stream=stream),
            compare_parts=[
                ("sparselnr_sddmm", lambda: slnr.sparselnr_sddmm(rp, ci, v, C, D, Y,
                                                                 stream=stream)),
                ("sparselnr_spmm", lambda: slnr.sparselnr_spmm(rp, ci, Y, E, A2,
                                                               stream=stream))],
            compare_desc="library unfused path: sparselnr_sddmm into an nnz-sized Y, then "
                         "sparselnr_spmm, each pass at its own grid factor",
            bytes=p.model_bytes(), bytes_model="4(N+1) + 8 nnz + 4 nnz (K+L) + 4 N K + 4 N L",
            footprint=csr_bytes + 4 * (N * p.K + M * p.K + M * p.L + N * p.L),
            dominant="walk_fast fused + carry_fixup (one call)", out=A,
            oracle=lambda: __import__("oracle").fused_rows(p.rowptr, p.colidx, p.vals, p.C, p.D,
                                                           p.E))

    if kernel == "sddmm_spmm_gemm":
        K = L = Mo = 64
        Ch, Dh, Fh = (synth.normal(0, s, (n, K)) for s, n in ((3, N), (4, M), (5, M)))
        Wh = synth.normal(0, 6, (L, Mo))
        C, D, F, W = t(Ch), t(Dh), t(Fh), t(Wh)
        A = torch.empty((N, Mo), dtype=torch.float32, device=dev)
        T = torch.empty((N, L), dtype=torch.float32, device=dev)
        A2 = torch.empty_like(A)

        def two_pass():
            slnr.sparselnr_fused_sddmm_spmm(rp, ci, v, C, D, F, T, stream=stream)
            torch.mm(T, W, out=A2)
        w.update(K=K, L=L, Mo=Mo)
        return dict(
            metric="fused <SDDMM,SpMM,GEMM> Gnnz/s + achieved HBM GB/s vs peak, "
                   "%s K=L=M=64" % config, desc=desc, sizes=w,
            call=lambda: slnr.sparselnr_fused_sddmm_spmm_gemm(rp, ci, v, C, D, F, W, A,
                                                              stream=stream),
            compare_parts=[("comparison", two_pass)],
            compare_desc="sparselnr_fused_sddmm_spmm into an N x L temporary, then torch.mm "
                         "by W",
            bytes=csr_bytes + 4 * nnz * (K + L) + 4 * N * K + 4 * N * Mo + 4 * L * Mo,
            bytes_model="4(N+1) + 8 nnz + 4 nnz (K+L) + 4 N K + 4 N Mo + 4 L Mo",
            footprint=csr_bytes + 4 * (N * K + M * K + M * L + L * Mo + N * Mo),
            dominant="walk_epi fused with matrix-core epilogue + carry_fixup (one call)", out=A,
            oracle=lambda: __import__("oracle").sddmm_spmm_gemm_rows(
                base.rowptr, base.colidx, base.vals, Ch, Dh, Fh, Wh))

    if kernel == "spmm_gemm":
        K, L = 128, 64
        Ch = synth.normal(0, 4, (M, K))
        Dh = synth.normal(0, 6, (K, L))
        C, D = t(Ch), t(Dh)
        A = torch.empty((N, L), dtype=torch.float32, device=dev)
        T = torch.empty((N, K), dtype=torch.float32, device=dev)
        A2 = torch.empty_like(A)

        def two_pass():
            slnr.sparselnr_spmm(rp, ci, v, C, T, stream=stream)
            torch.mm(T, D, out=A2)
        w.update(K=K, L=L)
        return dict(
            metric="fused <SpMM,GEMM> Gnnz/s + achieved HBM GB/s vs peak, %s K=128 L=64"
                   % config, desc=desc, sizes=w,
            call=lambda: slnr.sparselnr_spmm_gemm(rp, ci, v, C, D, A, stream=stream),
            compare_parts=[("comparison", two_pass)],
            compare_desc="sparselnr_spmm (B C) into an N x K temporary, then torch.mm by D",
            bytes=csr_bytes + 4 * nnz * K + 4 * K * L + 4 * N * L,
            bytes_model="4(N+1) + 8 nnz + 4 nnz K + 4 K L + 4 N L",
            footprint=csr_bytes + 4 * (M * K + K * L + N * L),
            dominant="walk_epi SpMM with matrix-core epilogue + carry_fixup (one call)", out=A,
            oracle=lambda: __import__("oracle").spmm_gemm_rows(base.rowptr, base.colidx,
                                                               base.vals, Ch, Dh))

    if kernel == "spmmh_gemm":
        J, L = 128, 128
        Ch, Dh = synth.normal(0, 4, (M, J)), synth.normal(0, 5, (M, J))
        Eh = synth.normal(0, 6, (J, L))
        C, D, E = t(Ch), t(Dh), t(Eh)
        A = torch.empty((N, L), dtype=torch.float32, device=dev)
        H = torch.empty((M, J), dtype=torch.float32, device=dev)
        T = torch.empty((N, J), dtype=torch.float32, device=dev)
        A2 = torch.empty_like(A)

        def two_pass():
            torch.mul(C, D, out=H)
            slnr.sparselnr_spmm(rp, ci, v, H, T, stream=stream)
            torch.mm(T, E, out=A2)
        w.update(J=J, L=L)
        # the library forms C .* D once when nnz >= 3 M (12 M J bytes, then
        # one gathered row per nonzero), else per nonzero from two rows
        hoisted = nnz >= 3 * M
        return dict(
            metric="fused <SpMMH,GEMM> Gnnz/s + achieved HBM GB/s vs peak, %s J=L=128" % config,
            desc=desc, sizes=w,
            call=lambda: slnr.sparselnr_spmmh_gemm(rp, ci, v, C, D, E, A, stream=stream),
            compare_parts=[("comparison", two_pass)],
            compare_desc="torch.mul C .* D into an M x J temporary, sparselnr_spmm into an "
                         "N x J temporary, then torch.mm by E",
            bytes=(12 * M * J + csr_bytes + 4 * nnz * J + 4 * J * L + 4 * N * L) if hoisted
            else (csr_bytes + 8 * nnz * J + 4 * J * L + 4 * N * L),
            bytes_model="12 M J + 4(N+1) + 8 nnz + 4 nnz J + 4 J L + 4 N L (C .* D formed once)"
            if hoisted else "4(N+1) + 8 nnz + 8 nnz J + 4 J L + 4 N L (C .* D per nonzero)",
            footprint=csr_bytes + 4 * ((3 if hoisted else 2) * M * J + J * L + N * L),
            dominant="hadamard4_kernel + walk_epi SpMM with matrix-core epilogue + carry_fixup "
                     "(one call)" if hoisted else
                     "walk_epi Hadamard SpMM with matrix-core epilogue + carry_fixup (one call)",
            out=A,
            oracle=lambda: __import__("oracle").spmmh_gemm_rows(base.rowptr, base.colidx,
                                                                base.vals, Ch, Dh, Eh))

    if kernel == "dt":
        p = base
        Dth = np.ascontiguousarray(p.D.T)
        C, D, Dt, E = t(p.C), t(p.D), t(Dth), t(p.E)
        A = torch.empty((N, p.L), dtype=torch.float32, device=dev)
        A2 = torch.empty_like(A)
        w.update(K=p.K, L=p.L)
        return dict(
            metric="fused SDDMM→SpMM with D stored K x M, Gnnz/s + achieved HBM GB/s vs peak, "
                   "%s K=L=%d" % (config, p.K), desc=desc, sizes=w,
            call=lambda: slnr.sparselnr_fused_sddmm_spmm_dt(rp, ci, v, C, Dt, E, A,
                                                            stream=stream),
            compare_parts=[("sparselnr_fused_sddmm_spmm",
                            lambda: slnr.sparselnr_fused_sddmm_spmm(rp, ci, v, C, D, E, A2,
                                                                    stream=stream))],
            compare_desc="sparselnr_fused_sddmm_spmm on D stored M x K (the cost of the layout)",
            bytes=p.model_bytes() + 8 * M * p.K,
            bytes_model="8 M K (transpose pass) + 4(N+1) + 8 nnz + 4 nnz (K+L) + 4 N K + 4 N L",
            footprint=csr_bytes + 4 * (N * p.K + 2 * M * p.K + M * p.L + N * p.L),
            dominant="transpose_kernel + walk_fast fused + carry_fixup (one call)", out=A,
            oracle=lambda: __import__("oracle").fused_rows_dt(p.rowptr, p.colidx, p.vals, p.C,
                                                              Dth, p.E))
    raise ValueError(kernel)


SWEEP_SIZES = (16, 32, 64, 128, 256, 512)


def sweep_spmm_gemm(args, dev, timed) -> None:
    import numpy as np
    import torch

    import paper_2205_11622_amd as slnr
    import synth

    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    stream = torch.cuda.current_stream(dev)
    base = synth.config(args.config)
    N, M, nnz = base.N, base.M, base.nnz
    rp, ci, v = t(base.rowptr), t(base.colidx), t(base.vals)
    cmax = synth.normal(0, 4, (M, max(SWEEP_SIZES)))
    for K in SWEEP_SIZES:
        C = t(cmax[:, :K])
        T = torch.empty((N, K), dtype=torch.float32, device=dev)
        for L in SWEEP_SIZES:
            D = t(synth.normal(0, 6, (K, L)))
            A = torch.empty((N, L), dtype=torch.float32, device=dev)
            A2 = torch.empty_like(A)

            def fused():
                slnr.sparselnr_spmm_gemm(rp, ci, v, C, D, A, stream=stream)

            def separate():
                slnr.sparselnr_spmm(rp, ci, v, C, T, stream=stream)
                torch.mm(T, D, out=A2)
            _, f_ms, _ = timed(fused, args.steps, args.warmup)
            _, s_ms, _ = timed(separate, args.steps, args.warmup)
            f_ms /= args.steps
            s_ms /= args.steps
            model = 4 * (N + 1) + 8 * nnz + 4 * nnz * K + 4 * K * L + 4 * N * L
            gbs = model / (f_ms * 1e-3) / 1e9
            print(json.dumps({"sweep": "spmm_gemm", "config": args.config, "K": K, "L": L,
                              "fused_ms": round(f_ms, 5), "separate_ms": round(s_ms, 5),
                              "speedup": round(s_ms / f_ms, 4), "fused_GBps": round(gbs, 1),
                              "frac": round(gbs / HBM_PEAK_GBPS, 4),
                              "bytes_model": "4(N+1) + 8 nnz + 4 nnz K + 4 K L + 4 N L"}),
                  flush=True)
            del A, A2, D
        del C, T
        torch.cuda.empty_cache()


def sweep_sddmm_spmm(args, dev, timed) -> None:
    """Fused <SDDMM, SpMM> against the library's unfused passes over K, L in
    {16..512} on the --config sparsity structure: where fusion pays on this GPU."""
    import numpy as np
    import torch

    import paper_2205_11622_amd as slnr
    import synth

    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    stream = torch.cuda.current_stream(dev)
    base = synth.config(args.config)
    N, M, nnz = base.N, base.M, base.nnz
    rp, ci, v = t(base.rowptr), t(base.colidx), t(base.vals)
    Y = torch.empty(nnz, dtype=torch.float32, device=dev)
    top = max(SWEEP_SIZES)
    cmax, dmax, emax = (t(synth.normal(0, s, (n, top))) for s, n in ((3, N), (4, M), (5, M)))
    for K in SWEEP_SIZES:
        C, D = cmax[:, :K].contiguous(), dmax[:, :K].contiguous()
        for L in SWEEP_SIZES:
            E = emax[:, :L].contiguous()
            A = torch.empty((N, L), dtype=torch.float32, device=dev)
            A2 = torch.empty_like(A)
            _, f_ms, _ = timed(lambda: slnr.sparselnr_fused_sddmm_spmm(
                rp, ci, v, C, D, E, A, stream=stream), args.steps, args.warmup)
            _, u_ms, _ = timed(lambda: slnr.sparselnr_unfused_sddmm_spmm(
                rp, ci, v, C, D, E, Y, A2, stream=stream), args.steps, args.warmup)
            f_ms /= args.steps
            u_ms /= args.steps
            model = 4 * (N + 1) + 8 * nnz + 4 * nnz * (K + L) + 4 * N * K + 4 * N * L
            gbs = model / (f_ms * 1e-3) / 1e9
            print(json.dumps({"sweep": "sddmm_spmm", "config": args.config, "K": K, "L": L,
                              "fused_ms": round(f_ms, 5), "unfused_ms": round(u_ms, 5),
                              "speedup": round(u_ms / f_ms, 4), "fused_GBps": round(gbs, 1),
                              "frac": round(gbs / HBM_PEAK_GBPS, 4),
                              "bytes_model": "4(N+1) + 8 nnz + 4 nnz (K+L) + 4 N K + 4 N L"}),
                  flush=True)
            del A, A2, E
        del C, D
        torch.cuda.empty_cache()


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed calls (default: 200 for the tiny and uniform workloads, whose calls "
                         "take tens of microseconds, else 20)")
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="rmat1m")
    ap.add_argument("--kernel", default="sddmm_spmm", choices=KERNELS)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-unfused", action="store_true",
                    help="skip the in-run comparison with the separate-pass computation")
    ap.add_argument("--sweep", action="store_true",
                    help="with --kernel sddmm_spmm or spmm_gemm: the fused call against the "
                         "separate passes over K, L in {16..512} (one JSON line per point)")
    ap.add_argument("--grid-factor", default="auto",
                    help="resident grids per walk launch for the timed call: 'auto' (fastest "
                         "of %s, chosen before the timed region) or a fixed value in 1..64"
                         % ",".join(map(str, GRID_FACTORS)))
    ap.add_argument("--compare-grid-factor", default="auto",
                    help="the same for the comparison: 'auto', one value for every pass, or "
                         "one comma-separated value per pass")
    ap.add_argument("--cold", action="store_true",
                    help="also time each call after writing and reading a 1 GiB buffer (which evicts "
                         "the 256 MB MALL and the L2s); reported as `cold`, never as `value`")
    ap.add_argument("--copy-probe", action="store_true",
                    help="after timing, run three plain 1 GiB device copies (torch copy_), the "
                         "reference for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE readings")
    args = ap.parse_args()
    if args.steps is None:
        args.steps = SMALL_STEPS if args.config in SMALL_CONFIGS and not args.sweep else 20
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on exactly one GPU: the fused kernel shards by rows with no "
              "communication, and this build measures one GPU's share only (--gpus 1).",
              file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    if args.config not in synth.CONFIGS:
        print("unknown config %r" % args.config, file=sys.stderr)
        return 2
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)

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

    if args.sweep:
        if args.kernel == "spmm_gemm":
            sweep_spmm_gemm(args, dev, timed)
        elif args.kernel == "sddmm_spmm":
            sweep_sddmm_spmm(args, dev, timed)
        else:
            print("--sweep is defined for --kernel sddmm_spmm and spmm_gemm", file=sys.stderr)
            return 2
        return 0

    t0 = time.time()
    wl = make_workload(args.kernel, args.config, dev)
    print("# %s / %s: %s (inputs made in %.1fs)" % (args.config, args.kernel, wl["sizes"],
                                                    time.time() - t0),
          file=sys.stderr, flush=True)

    import paper_2205_11622_amd as slnr
    set_factor = slnr.lib().sparselnr_set_grid_factor

    def tune(name, fn):
        """Fastest grid factor for one library call: per candidate, one untimed
        call, then the median of TUNE_CALLS timed ones."""
        res = {}
        for f in GRID_FACTORS:
            slnr.sparselnr_set_grid_factor(f)
            res[f] = round(float(np.median(timed(fn, TUNE_CALLS, 1)[0])), 5)
        best = min(res, key=res.get)
        print("# grid factor for %s: %d (%s)" % (name, best, " ".join(
            "%d:%.4f" % kv for kv in res.items())), file=sys.stderr, flush=True)
        return best, res

    def factors_for(parts, spec, what):
        if spec == "auto":
            chosen = [tune(name, fn) for name, fn in parts]
            return [c[0] for c in chosen], {name: c[1] for (name, _), c in zip(parts, chosen)}
        vals = [int(x) for x in spec.split(",")]
        if len(vals) == 1:
            vals = vals * len(parts)
        if len(vals) != len(parts) or not all(1 <= f <= 64 for f in vals):
            raise SystemExit("%s: need 'auto' or %d value(s) in 1..64" % (what, len(parts)))
        return vals, None

    def bound(parts, factors):
        calls = list(zip(factors, [fn for _, fn in parts]))

        def run():
            for f, fn in calls:
                set_factor(f)
                fn()
        return run

    def settle(fn, seconds=SETTLE_S):
        """Untimed calls, each waited for, until `seconds` of wall time have
        passed: a call of a few microseconds otherwise meets the GPU still at
        the clocks of the host-side set-up before it."""
        t_end = time.perf_counter() + seconds
        while True:
            fn()
            torch.cuda.synchronize()
            if time.perf_counter() >= t_end:
                break

    call_parts = [("timed call", wl["call"])]
    call_factors, call_tuning = factors_for(call_parts, args.grid_factor, "--grid-factor")
    call = bound(call_parts, call_factors)
    settle(call)
    per, total_ms, wall = timed(call, args.steps, args.warmup)
    ms = total_ms / args.steps
    print("# fused: %.4f ms/call (median %.4f, min %.4f, max %.4f)"
          % (ms, np.median(per), per.min(), per.max()), file=sys.stderr, flush=True)
    unf = None
    cmp_tuning = None
    if not args.no_unfused:
        parts = wl["compare_parts"]
        cmp_factors, cmp_tuning = factors_for(parts, args.compare_grid_factor,
                                              "--compare-grid-factor")
        settle(bound(parts, cmp_factors))
        uper, utotal, _ = timed(bound(parts, cmp_factors), args.steps, args.warmup)
        # interleave a second fused round so both see the same machine state
        per2, total2, _ = timed(call, args.steps, 1)
        unf = {"what": wl["compare_desc"], "ms_per_call": utotal / args.steps,
               "median_ms": float(np.median(uper)), "fused_ms_rerun": total2 / args.steps,
               "fused_speedup": (utotal / args.steps) / ms,
               "grid_factors": {name: f for (name, _), f in zip(parts, cmp_factors)}}
        print("# comparison: %.4f ms/call; fused rerun %.4f ms" % (unf["ms_per_call"],
                                                                  unf["fused_ms_rerun"]),
              file=sys.stderr, flush=True)
    cold = None
    if args.cold:
        flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)
        flush.fill_(0.0)
        cper = []
        ce = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        for _ in range(args.steps):
            flush.add_(1.0)  # reads and writes 1 GiB on the same stream, just before the call
            ce[0].record(stream)
            call()
            ce[1].record(stream)
            torch.cuda.synchronize()
            cper.append(ce[0].elapsed_time(ce[1]))
        del flush
        torch.cuda.empty_cache()
        cold = {"ms_per_call_median": round(float(np.median(cper)), 5),
                "ms_per_call_min": round(float(np.min(cper)), 5), "calls": len(cper),
                "flush": "1 GiB read and written on the stream before each call"}
        print("# cold: %.4f ms/call (median)" % cold["ms_per_call_median"], file=sys.stderr,
              flush=True)
    slnr.sparselnr_set_grid_factor(0)

    # context for comparing runs across machines: the rate of torch's own
    # 1 GiB device-to-device copy (read + write = 2 GiB moved)
    src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    _, copy_ms, _ = timed(lambda: dst.copy_(src), 5, 2)
    copy_gbps = 2 * (1 << 30) / (copy_ms / 5 * 1e-3) / 1e9
    del src, dst
    torch.cuda.empty_cache()

    if args.copy_probe:
        src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    nnz = wl["sizes"]["nnz"]
    model_bytes = wl["bytes"]
    gnnz = nnz / (ms * 1e-3) / 1e9
    achieved = model_bytes / (ms * 1e-3) / 1e9
    key = workload_key(args.config, args.kernel)
    traffic = stored_traffic(key)
    frac = achieved / HBM_PEAK_GBPS
    tbytes = traffic["bytes_per_call"] if traffic else None
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                "unit": "GB/s", "frac": round(frac, 4), "traffic": tbytes,
                "traffic_GBps": round(tbytes / (ms * 1e-3) / 1e9, 1) if tbytes else None,
                "traffic_frac": round(tbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4)
                if tbytes else None,
                "kernel": wl["dominant"], "bytes_per_call": model_bytes,
                "bytes_model": wl["bytes_model"],
                "torch_copy_GBps": round(copy_gbps, 1)}
    if frac > 1.0:
        # the algorithmic bytes count every gathered row, and here more of
        # them come from L2 and the MALL than the HBM peak could deliver:
        # the figure is not a fraction of the HBM roofline
        roofline["bound"] = "l2"
        roofline["note"] = ("algorithmic bytes exceed what HBM could deliver in this time: "
                            "gathered rows are served by L2 and the MALL; traffic_frac (measured "
                            "FETCH_SIZE + WRITE_SIZE per second / HBM peak) is the HBM-side "
                            "figure")

    cpu = None
    parity = None
    if not args.no_cpu_baseline:
        import oracle
        times = []
        t1 = time.perf_counter()
        res = None
        while not times or (time.perf_counter() - t1 < CPU_SECONDS and len(times) < 50):
            del res
            s0 = time.perf_counter()
            res = wl["oracle"]()
            times.append(time.perf_counter() - s0)
        cs = float(np.median(times))
        cpu = {"value": round(nnz / cs / 1e9, 6), "unit": "Gnnz/s", "cores": oracle.num_threads(),
               "cores_meaning": "OpenMP threads the oracle ran with", "kind": "oracle",
               "seconds": float("%.4g" % cs), "passes": len(times),
               "host": host_info(),
               "sample": "the whole %s workload (%d rows, %d nonzeros) per pass, median of %d "
                         "passes; each pass is the oracle as the tests use it: fp64 "
                         "accumulation, OpenMP over rows, plus the tolerance scale (the same "
                         "loops on absolute values, twice the arithmetic) and an fp64 N x %d "
                         "result" % (key, wl["sizes"]["N"], nnz, len(times),
                                     wl["out"].shape[1])}
        # the timed call's output (its last run) against this oracle pass, every row
        worst, bad = row_parity(wl["out"].cpu().numpy(), res[0], res[1])
        parity = {"rows": int(wl["out"].shape[0]),
                  "max_err_over_scale": float("%.4g" % worst) if np.isfinite(worst) else "inf",
                  "rows_outside_tol": bad, "tol": 1e-4,
                  "rule": "per row: max_l |A - Aref| <= tol * max_l of the same computation on "
                          "absolute values"}
        del res

    out = {
        "metric": wl["metric"], "value": round(gnnz, 4), "unit": "Gnnz/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": dict({"workload": wl["desc"], "kernel": args.kernel}, **wl["sizes"]),
        "roofline": roofline, "cpu_baseline": cpu, "parity": parity,
        "counters": ({"kernel": traffic["dominant"],
                      "l2_hit_rate": traffic.get("l2_hit_rate"),
                      "valu_busy_pct": traffic.get("valu_busy_pct"),
                      "source": "rocprofv3 --pmc passes committed under profiles/ (counters_%s.md)"
                                % key} if traffic else None),
        "paper_context": dict(PAPER_CONTEXT[args.kernel], hardware=PAPER_HARDWARE,
                              use="context only: the paper's CPU speedups over TACO, not a "
                                  "target for this GPU path"),
        "achieved_GBps": round(achieved, 1),
        "footprint_bytes": wl["footprint"],
        "median_ms": round(float(np.median(per)), 5), "min_ms": round(float(per.min()), 5),
        "p90_ms": round(float(np.percentile(per, 90)), 5), "wall_s": round(wall, 3),
        "unfused": unf, "cold": cold, "source_digest": source_digest(),
        "device": device_info(dev),
        "launch": {"grid_factor": call_factors[0],
                   "chosen_by": "'auto': fastest of %s, median of %d calls each, before the "
                                "timed region; else fixed on the command line (timed call %s, "
                                "comparison %s)" % (list(GRID_FACTORS), TUNE_CALLS,
                                                    args.grid_factor, args.compare_grid_factor),
                   "tuning_ms": {"timed call": call_tuning and call_tuning["timed call"],
                                 "comparison": cmp_tuning}},
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
