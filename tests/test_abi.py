"""The C ABI: the library loads, exports every declared symbol, and rejects
bad arguments before touching HIP (runs without a GPU)."""
import ctypes
import os
import re

import pytest

import paper_2205_11622_amd as slnr

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sparselnr.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sparselnr_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ["sparselnr_fused_sddmm_spmm", "sparselnr_unfused_sddmm_spmm",
                     "sparselnr_sddmm", "sparselnr_spmm", "sparselnr_validate_csr",
                     "sparselnr_status_string", "sparselnr_last_hip_error",
                     "sparselnr_release", "sparselnr_abi_version"]:
        assert required in names


def test_library_exports_every_declared_symbol():
    lib = slnr.lib()
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_binding_names_match_the_abi():
    for name in declared_functions():
        assert hasattr(slnr, name), name


def test_version_and_status_strings():
    assert slnr.sparselnr_abi_version() == 1
    for code in range(6):
        s = slnr.sparselnr_status_string(code)
        assert isinstance(s, str) and s
    assert slnr.sparselnr_status_string(99) == "unknown status"
    assert slnr.sparselnr_status_string(0) == "ok"


def test_grid_factor_setter():
    lib = slnr.lib()
    before = slnr.sparselnr_get_grid_factor()
    try:
        for f in (1, 8, 48, 64):
            slnr.sparselnr_set_grid_factor(f)
            assert slnr.sparselnr_get_grid_factor() == f
        slnr.sparselnr_set_grid_factor(0)
        assert slnr.sparselnr_get_grid_factor() == 0
        for bad in (-1, 65, 1 << 20):
            assert lib.sparselnr_set_grid_factor(bad) == slnr.ERR_INVALID_ARG
            assert slnr.sparselnr_get_grid_factor() == 0
        with pytest.raises(slnr.SparseLNRError):
            slnr.sparselnr_set_grid_factor(-3)
    finally:
        slnr.sparselnr_set_grid_factor(before)


def test_grid_factor_environment():
    # SPARSELNR_GRID_FACTOR gives the first value (1..64, anything else means
    # automatic); sparselnr_set_grid_factor overrides it
    import subprocess
    import sys
    code = ("import paper_2205_11622_amd as s; a = s.sparselnr_get_grid_factor(); "
            "s.sparselnr_set_grid_factor(3); b = s.sparselnr_get_grid_factor(); "
            "s.sparselnr_set_grid_factor(0); print(a, b, s.sparselnr_get_grid_factor())")
    for env, want in (("12", "12 3 0"), ("64", "64 3 0"), ("65", "0 3 0"), ("0", "0 3 0"),
                      ("x", "0 3 0"), (None, "0 3 0")):
        e = dict(os.environ)
        e.pop("SPARSELNR_GRID_FACTOR", None)
        if env is not None:
            e["SPARSELNR_GRID_FACTOR"] = env
        r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                           timeout=120, cwd=ROOT, env=e)
        assert r.returncode == 0, r.stderr
        assert r.stdout.split() == want.split(), (env, r.stdout)


NULL = None
FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: every case fails validation first


@pytest.mark.parametrize("args,code", [
    # negative sizes
    ((FAKE,) * 7 + (-1, 4, 4, 4, NULL), slnr.ERR_INVALID_ARG),
    ((FAKE,) * 7 + (4, -1, 4, 4, NULL), slnr.ERR_INVALID_ARG),
    ((FAKE,) * 7 + (4, 4, -1, 4, NULL), slnr.ERR_INVALID_ARG),
    ((FAKE,) * 7 + (4, 4, 4, -1, NULL), slnr.ERR_INVALID_ARG),
    # NULL arrays
    ((NULL,) + (FAKE,) * 6 + (4, 4, 4, 4, NULL), slnr.ERR_INVALID_ARG),
    ((FAKE, NULL) + (FAKE,) * 5 + (4, 4, 4, 4, NULL), slnr.ERR_INVALID_ARG),
    ((FAKE, FAKE, NULL) + (FAKE,) * 4 + (4, 4, 4, 4, NULL), slnr.ERR_INVALID_ARG),
    ((FAKE,) * 3 + (NULL,) + (FAKE,) * 3 + (4, 4, 4, 4, NULL), slnr.ERR_INVALID_ARG),
    ((FAKE,) * 4 + (NULL,) + (FAKE,) * 2 + (4, 4, 4, 4, NULL), slnr.ERR_INVALID_ARG),
    ((FAKE,) * 5 + (NULL, FAKE) + (4, 4, 4, 4, NULL), slnr.ERR_INVALID_ARG),
    ((FAKE,) * 6 + (NULL,) + (4, 4, 4, 4, NULL), slnr.ERR_INVALID_ARG),
    # too wide / too many rows
    ((FAKE,) * 7 + (4, 4, 65537, 4, NULL), slnr.ERR_UNSUPPORTED),
    ((FAKE,) * 7 + (4, 4, 4, 65537, NULL), slnr.ERR_UNSUPPORTED),
    ((FAKE,) * 7 + (2**31, 4, 4, 4, NULL), slnr.ERR_UNSUPPORTED),
    # empty problems need no HIP call at all
    ((NULL,) * 7 + (0, 0, 0, 0, NULL), slnr.OK),
    ((FAKE,) * 3 + (FAKE, FAKE, NULL, NULL) + (5, 5, 4, 0, NULL), slnr.OK),
])
def test_fused_argument_errors(args, code):
    assert slnr.lib().sparselnr_fused_sddmm_spmm(*args) == code


def test_other_entry_points_argument_errors():
    L = slnr.lib()
    assert L.sparselnr_sddmm(*(FAKE,) * 6, -1, 4, 4, NULL) == slnr.ERR_INVALID_ARG
    assert L.sparselnr_sddmm(FAKE, FAKE, FAKE, FAKE, FAKE, NULL, 4, 4, 4, NULL) == slnr.ERR_INVALID_ARG
    assert L.sparselnr_sddmm(*(NULL,) * 6, 0, 0, 0, NULL) == slnr.OK
    assert L.sparselnr_spmm(*(FAKE,) * 5, 4, 4, -2, NULL) == slnr.ERR_INVALID_ARG
    assert L.sparselnr_spmm(FAKE, FAKE, NULL, FAKE, FAKE, 4, 4, 4, NULL) == slnr.ERR_INVALID_ARG
    assert L.sparselnr_spmm(*(FAKE,) * 5, 4, 4, 70000, NULL) == slnr.ERR_UNSUPPORTED
    assert L.sparselnr_unfused_sddmm_spmm(*(FAKE,) * 6, NULL, FAKE, 4, 4, 4, 4, NULL) == \
        slnr.ERR_INVALID_ARG
    assert L.sparselnr_unfused_sddmm_spmm(*(FAKE,) * 8, 4, 4, 4, -4, NULL) == slnr.ERR_INVALID_ARG
    nnz = ctypes.c_int64(0)
    assert L.sparselnr_validate_csr(NULL, FAKE, 4, 4, 4, ctypes.byref(nnz), NULL) == \
        slnr.ERR_INVALID_ARG
    assert L.sparselnr_validate_csr(FAKE, FAKE, -1, 4, 4, ctypes.byref(nnz), NULL) == \
        slnr.ERR_INVALID_ARG
    assert L.sparselnr_validate_csr(FAKE, NULL, 4, 4, 4, ctypes.byref(nnz), NULL) == \
        slnr.ERR_INVALID_ARG


def test_no_hip_error_recorded_by_validation_failures():
    slnr.lib().sparselnr_fused_sddmm_spmm(*(FAKE,) * 7, -1, 4, 4, 4, NULL)
    assert slnr.sparselnr_last_hip_error() == 0


def test_binding_refuses_cpu_tensors():
    torch = pytest.importorskip("torch")
    rp = torch.zeros(3, dtype=torch.int32)
    ci = torch.zeros(0, dtype=torch.int32)
    v = torch.zeros(0)
    C = torch.zeros(2, 4)
    with pytest.raises(ValueError):
        slnr.sparselnr_fused_sddmm_spmm(rp, ci, v, C, C, C)


def test_product_package_does_not_touch_the_oracle():
    """The product path neither imports nor links the oracle or the input generators."""
    pkg = os.path.join(ROOT, "paper_2205_11622_amd")
    pat = re.compile(r"^\s*(import|from)\s+(oracle|synth)\b|liboracle|libsynth|oracle\.c", re.M)
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".hpp", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert not pat.search(text), f


def test_next_entry_points_argument_errors():
    L = slnr.lib()
    # <SDDMM, SpMM, GEMM>: negative size, NULL W, unsupported shapes (K != L, K = L = 48)
    assert L.sparselnr_fused_sddmm_spmm_gemm(*(FAKE,) * 8, 4, 4, 4, 4, -1, NULL) == \
        slnr.ERR_INVALID_ARG
    assert L.sparselnr_fused_sddmm_spmm_gemm(*(FAKE,) * 6, NULL, FAKE, 4, 4, 4, 4, 4, NULL) == \
        slnr.ERR_INVALID_ARG
    assert L.sparselnr_fused_sddmm_spmm_gemm(*(FAKE,) * 8, 4, 4, 64, 32, 32, NULL) == \
        slnr.ERR_UNSUPPORTED
    assert L.sparselnr_fused_sddmm_spmm_gemm(*(FAKE,) * 8, 4, 4, 48, 48, 48, NULL) == \
        slnr.ERR_UNSUPPORTED
    assert L.sparselnr_fused_sddmm_spmm_gemm(*(NULL,) * 8, 0, 0, 0, 0, 0, NULL) == slnr.OK
    # <SpMM, GEMM>
    assert L.sparselnr_spmm_gemm(*(FAKE,) * 6, 4, 4, -1, 4, NULL) == slnr.ERR_INVALID_ARG
    assert L.sparselnr_spmm_gemm(FAKE, FAKE, FAKE, FAKE, NULL, FAKE, 4, 4, 4, 4, NULL) == \
        slnr.ERR_INVALID_ARG
    assert L.sparselnr_spmm_gemm(*(FAKE,) * 6, 4, 4, 100, 4, NULL) == slnr.ERR_UNSUPPORTED
    # <SpMMH, GEMM>
    assert L.sparselnr_spmmh_gemm(FAKE, FAKE, FAKE, FAKE, NULL, FAKE, FAKE, 4, 4, 4, 4, NULL) == \
        slnr.ERR_INVALID_ARG
    assert L.sparselnr_spmmh_gemm(*(FAKE,) * 7, 4, 4, 100, 64, NULL) == slnr.ERR_UNSUPPORTED
    # transposed D
    assert L.sparselnr_fused_sddmm_spmm_dt(*(FAKE,) * 4, NULL, FAKE, FAKE, 4, 4, 4, 4, NULL) == \
        slnr.ERR_INVALID_ARG
    assert L.sparselnr_fused_sddmm_spmm_dt(*(FAKE,) * 7, -4, 4, 4, 4, NULL) == slnr.ERR_INVALID_ARG


@pytest.mark.parametrize("entry", ["sparselnr_fused_sddmm_spmm", "sparselnr_fused_sddmm_spmm_dt",
                                   "sparselnr_fused_sddmm_spmm_noalloc"])
@pytest.mark.parametrize("which", ["rowptr", "colidx", "vals", "C", "D", "E", "A"])
def test_fused_null_pointer_rejected_before_any_hip_call(entry, which):
    """Both fused entry points (plain and transposed D) reject every NULL array
    with ERR_INVALID_ARG.  On this GPU-less host any HIP call would fail with
    ERR_HIP instead, so the status shows that the check precedes all device
    work (the transposed-D call allocates and transposes only afterwards)."""
    names = ["rowptr", "colidx", "vals", "C", "D", "E", "A"]
    args = [NULL if n == which else FAKE for n in names]
    fn = getattr(slnr.lib(), entry)
    assert fn(*args, 64, 48, 16, 32, NULL) == slnr.ERR_INVALID_ARG
    # the same call with every pointer set gets past the checks to the HIP
    # runtime, which fails without a GPU: the checks alone made the difference
    if not _gpu_visible():
        assert fn(*(FAKE,) * 7, 64, 48, 16, 32, NULL) == slnr.ERR_HIP


def _gpu_visible():
    """True where a GPU may be present (then the fake pointers must never
    reach a launch).  Counting devices does not initialise HIP."""
    if os.path.exists("/dev/kfd"):
        return True
    try:
        import torch
        return torch.cuda.device_count() > 0
    except Exception:
        return True


def test_header_is_plain_c(tmp_path):
    """The header and the C caller compile as C11 (no C++ in the interface)."""
    import subprocess
    src = os.path.join(ROOT, "tests", "c_abi", "abi_check.c")
    r = subprocess.run(["gcc", "-std=c11", "-Wall", "-Werror", "-fsyntax-only",
                        "-I/opt/rocm/include", "-I" + os.path.join(ROOT, "include"), src],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
