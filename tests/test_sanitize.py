"""Sanitizer builds of the host code that the tests rely on (runs without a
GPU): the CPU oracle and the input generators, compiled together with a
driver that calls every exported function (tests/sanitize/sanitize_check.c),
and the plain C caller of the library's ABI in its host-only mode
(tests/c_abi/abi_check.c: inputs, oracle, comparison routine and the
argument-error calls, which return before any HIP call), each under
AddressSanitizer and UndefinedBehaviorSanitizer with leak detection.  Any
report makes the program exit non-zero."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-O1", "-g", "-std=c11", "-Wall", "-fsanitize=address,undefined",
       "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-fopenmp"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
           UBSAN_OPTIONS="print_stacktrace=1", OMP_NUM_THREADS="4")


def _gcc_or_skip():
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")


def _run(exe, *args):
    r = subprocess.run([exe, *args], capture_output=True, text=True, timeout=300, env=ENV)
    return r.returncode, r.stdout + r.stderr


def test_oracle_and_generators_under_sanitizers(tmp_path):
    _gcc_or_skip()
    exe = str(tmp_path / "sanitize_check")
    subprocess.check_call(["gcc", *SAN, os.path.join(ROOT, "tests", "sanitize", "sanitize_check.c"),
                           os.path.join(ROOT, "oracle", "oracle.c"),
                           os.path.join(ROOT, "synth", "gen.c"), "-o", exe, "-lm"])
    rc, out = _run(exe)
    assert rc == 0, out
    assert "sanitize_check: ok" in out


def test_c_abi_caller_host_phases_under_sanitizers(tmp_path):
    _gcc_or_skip()
    lib = os.path.join(ROOT, "paper_2205_11622_amd", "libsparselnr.so")
    if not os.path.exists(lib):
        pytest.fail("libsparselnr.so is not built: run __graft_entry__.build()")
    exe = str(tmp_path / "abi_check_san")
    subprocess.check_call([
        "gcc", *SAN, "-I/opt/rocm/include", "-I" + os.path.join(ROOT, "include"),
        os.path.join(ROOT, "tests", "c_abi", "abi_check.c"), os.path.join(ROOT, "oracle", "oracle.c"),
        "-o", exe, "-L" + os.path.dirname(lib), "-lsparselnr", "-L/opt/rocm/lib", "-lamdhip64",
        "-lm", "-Wl,-rpath," + os.path.dirname(lib) + ":/opt/rocm/lib"])
    rc, out = _run(exe, "--host-only")
    assert rc == 0, out
    assert "abi_check: host phases ok" in out
    # the exit-handler marker shows the program reached its own teardown
    assert "exit handlers reached (last phase: done (host only))" in out
