"""Seeded synthetic inputs for the fused SDDMM->SpMM workloads.

This package only *draws* inputs (CSR structures and dense fp32 arrays); it
holds none of the method's arithmetic.  The CPU oracle and the GPU library are
both fed from what it returns, and neither of them imports it.

The paper's evaluation uses SuiteSparse / Network Repository matrices with
randomly drawn dense operands (Section 6.1, Table 1); none of those files are
used here.  The five named workloads below stand in for them by shape and
structure class: a cora-sized uniform matrix, a mid-size uniform matrix at the
paper's inner sizes K=L=64 (Section 6.2, <SDDMM, SpMM> paragraph), two R-MAT
power-law graphs (webbase-1M / circuit5M scale) and a 27-point-stencil FEM-like
matrix (cant / consph / shipsec1 class).

All randomness comes from one counter-based SplitMix64 stream per array (see
gen.c), so every array is a pure function of (seed, stream id, index).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_SRC = os.path.join(_HERE, "gen.c")

# stream ids: one independent stream per array of a problem
STREAM_STRUCTURE, STREAM_VALS, STREAM_C, STREAM_D, STREAM_E = 1, 2, 3, 4, 5

RMAT_ABC = (0.57, 0.19, 0.19)


def build(force: bool = False) -> str:
    """Compile gen.c into libsynth.so (gcc, OpenMP)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall",
                               _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        L = ctypes.CDLL(_LIB_PATH)
        i64, u64, f64, vp = ctypes.c_int64, ctypes.c_uint64, ctypes.c_double, ctypes.c_void_p
        L.synth_draw.restype = u64
        L.synth_draw.argtypes = [u64, u64, u64]
        L.synth_uniform_f32.restype = None
        L.synth_uniform_f32.argtypes = [u64, u64, f64, f64, i64, vp]
        L.synth_normal_f32.restype = None
        L.synth_normal_f32.argtypes = [u64, u64, i64, vp]
        L.synth_csr_fixed_degree.restype = ctypes.c_int
        L.synth_csr_fixed_degree.argtypes = [u64, u64, i64, i64, i64, vp, vp]
        L.synth_rmat.restype = i64
        L.synth_rmat.argtypes = [u64, u64, ctypes.c_int, i64, f64, f64, f64, vp, vp]
        L.synth_stencil27.restype = i64
        L.synth_stencil27.argtypes = [i64, vp, vp]
        L.synth_num_threads.restype = ctypes.c_int
        _lib = L
    return _lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def draw(seed: int, stream: int, n: int) -> int:
    """Raw 64-bit output number n of stream (seed, stream)."""
    return int(lib().synth_draw(seed, stream, n))


def uniform(seed: int, stream: int, shape, lo: float = -1.0, hi: float = 1.0) -> np.ndarray:
    out = np.empty(shape, dtype=np.float32)
    lib().synth_uniform_f32(seed, stream, lo, hi, out.size, _ptr(out))
    return out


def normal(seed: int, stream: int, shape) -> np.ndarray:
    out = np.empty(shape, dtype=np.float32)
    lib().synth_normal_f32(seed, stream, out.size, _ptr(out))
    return out


@dataclass
class Problem:
    """One instance of A(i,l) = sum_{j,k} B(i,j) C(i,k) D(j,k) E(j,l) with B in CSR."""
    name: str
    N: int
    M: int
    K: int
    L: int
    rowptr: np.ndarray  # int32[N+1]
    colidx: np.ndarray  # int32[nnz]
    vals: np.ndarray    # float32[nnz]
    C: np.ndarray       # float32[N, K]
    D: np.ndarray       # float32[M, K]
    E: np.ndarray       # float32[M, L]
    info: dict = field(default_factory=dict)

    @property
    def nnz(self) -> int:
        return int(self.rowptr[-1]) if self.rowptr.size else 0

    def model_bytes(self) -> int:
        """Algorithmic bytes of one fused pass: CSR arrays, one gathered D row and
        E row per nonzero, and the C / A streams."""
        N, K, L, nnz = self.N, self.K, self.L, self.nnz
        return 4 * (N + 1) + 8 * nnz + 4 * nnz * (K + L) + 4 * N * K + 4 * N * L


def _dense(seed, N, M, K, L, dist):
    if dist == "normal":
        return (normal(seed, STREAM_C, (N, K)), normal(seed, STREAM_D, (M, K)),
                normal(seed, STREAM_E, (M, L)))
    return (uniform(seed, STREAM_C, (N, K)), uniform(seed, STREAM_D, (M, K)),
            uniform(seed, STREAM_E, (M, L)))


def fixed_degree(N: int, M: int, deg: int, K: int, L: int, seed: int = 0,
                 vals_range=(-1.0, 1.0), dense: str = "uniform", name: str = "fixed") -> Problem:
    """Every row has exactly `deg` distinct uniformly drawn columns (sorted)."""
    rowptr = np.empty(N + 1, dtype=np.int32)
    colidx = np.empty(N * deg, dtype=np.int32)
    rc = lib().synth_csr_fixed_degree(seed, STREAM_STRUCTURE, N, M, deg, _ptr(rowptr), _ptr(colidx))
    if rc != 0:
        raise ValueError("bad fixed-degree arguments")
    vals = uniform(seed, STREAM_VALS, colidx.size, *vals_range)
    C, D, E = _dense(seed, N, M, K, L, dense)
    return Problem(name, N, M, K, L, rowptr, colidx, vals, C, D, E,
                   {"kind": "fixed_degree", "deg": deg, "seed": seed})


def rmat(levels: int, avg_degree: int, K: int, L: int, seed: int = 0, abc=RMAT_ABC,
         vals_range=(0.0, 1.0), dense: str = "normal", name: str = "rmat") -> Problem:
    """R-MAT graph with 2**levels vertices and avg_degree * 2**levels drawn edges,
    duplicates merged (so nnz is a little lower)."""
    N = 1 << levels
    samples = avg_degree * N
    rowptr = np.empty(N + 1, dtype=np.int32)
    colidx = np.empty(max(samples, 1), dtype=np.int32)
    nnz = lib().synth_rmat(seed, STREAM_STRUCTURE, levels, samples, abc[0], abc[1], abc[2],
                           _ptr(rowptr), _ptr(colidx))
    if nnz < 0:
        raise MemoryError("R-MAT generation failed")
    colidx = colidx[:nnz].copy()
    vals = uniform(seed, STREAM_VALS, nnz, *vals_range)
    C, D, E = _dense(seed, N, N, K, L, dense)
    return Problem(name, N, N, K, L, rowptr, colidx, vals, C, D, E,
                   {"kind": "rmat", "levels": levels, "samples": samples, "abc": list(abc),
                    "seed": seed})


def stencil27(n: int, K: int, L: int, seed: int = 0, vals_range=(-1.0, 1.0),
              dense: str = "uniform", name: str = "stencil") -> Problem:
    """27-point stencil on an n^3 grid, boundary rows truncated."""
    N = n ** 3
    side = max(3 * n - 2, 0) if n > 1 else n
    rowptr = np.empty(N + 1, dtype=np.int32)
    colidx = np.empty(side ** 3, dtype=np.int32)
    nnz = lib().synth_stencil27(n, _ptr(rowptr), _ptr(colidx))
    assert nnz == colidx.size, (nnz, colidx.size)
    vals = uniform(seed, STREAM_VALS, nnz, *vals_range)
    C, D, E = _dense(seed, N, N, K, L, dense)
    return Problem(name, N, N, K, L, rowptr, colidx, vals, C, D, E,
                   {"kind": "stencil27", "n": n, "seed": seed})


# The five named workloads (sizes as stated; seed 0 for all).
CONFIGS = {
    "tiny": dict(desc="2048x2048 CSR, 10 distinct uniform columns per row, vals U[-1,1); "
                      "C,D,E U[-1,1), K=L=32"),
    "uniform": dict(desc="65536x65536 CSR, 16 distinct uniform columns per row, vals U[-1,1); "
                         "C,D,E U[-1,1), K=L=64"),
    "rmat1m": dict(desc="R-MAT 2^20 vertices, (a,b,c,d)=(.57,.19,.19,.05), 16 edges/vertex drawn, "
                        "duplicates merged, vals U[0,1); C,D,E N(0,1), K=L=128"),
    "rmat4m": dict(desc="R-MAT 2^22 vertices, (a,b,c,d)=(.57,.19,.19,.05), 32 edges/vertex drawn, "
                        "duplicates merged, vals U[0,1); C,D,E N(0,1), K=L=64"),
    "banded": dict(desc="27-point stencil on a 128^3 grid (2,097,152 rows), vals U[-1,1); "
                        "C,D U[-1,1) K=16, E U[-1,1) L=256"),
}


def config(name: str, seed: int = 0) -> Problem:
    if name == "tiny":
        return fixed_degree(2048, 2048, 10, 32, 32, seed, name=name)
    if name == "uniform":
        return fixed_degree(65536, 65536, 16, 64, 64, seed, name=name)
    if name == "rmat1m":
        return rmat(20, 16, 128, 128, seed, name=name)
    if name == "rmat4m":
        return rmat(22, 32, 64, 64, seed, name=name)
    if name == "banded":
        return stencil27(128, 16, 256, seed, name=name)
    raise KeyError(name)
