"""Address- and undefined-behaviour-sanitised CPU builds of the oracle and of
the library's host code (validation, planning, workspace layout, dispatch),
each driven in a child process by the CPU tests that exercise it.

The oracle is built with gcc's sanitizers and runs every oracle pin; the
library is built with the host half of each HIP source sanitised (device code
is compiled as usual and never runs here) and runs the C-ABI tests, which
cover every validation path, the size queries and the mapping of a refused
HIP launch to LSA_ERR_HIP.  A sanitizer report or a non-zero exit fails the
test.
"""
import glob
import importlib.util
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_09079_amd", "csrc")
_spec = importlib.util.spec_from_file_location("_lsa_build", os.path.join(ROOT, "paper_2606_09079_amd", "_build.py"))
_build = importlib.util.module_from_spec(_spec)
_spec.loader.exec_module(_build)
SOURCES = _build.SOURCES
REPORTS = ("ERROR: AddressSanitizer", "runtime error:", "ERROR: LeakSanitizer")


def _no_device():
    import torch
    return torch.cuda.device_count() == 0


def _run_tests(env_extra, test_file):
    env = dict(os.environ)
    env.update(env_extra)
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    res = subprocess.run([sys.executable, "-m", "pytest", test_file, "-q", "-x", "-m", "not gpu",
                          "-p", "no:cacheprovider"], cwd=ROOT, env=env, capture_output=True, text=True,
                         timeout=900)
    out = res.stdout + res.stderr
    for r in REPORTS:
        assert r not in out, out[-4000:]
    assert res.returncode == 0, out[-4000:]
    assert " passed" in res.stdout, out[-4000:]


def test_oracle_under_sanitizers(tmp_path):
    so = str(tmp_path / "liblsa_oracle_san.so")
    subprocess.check_call(["gcc", "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-fno-fast-math",
                           "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                           "-fno-sanitize-recover=undefined", os.path.join(ROOT, "oracle", "lsa_oracle.c"),
                           "-o", so, "-lm"])
    asan = subprocess.check_output(["gcc", "-print-file-name=libasan.so"], text=True).strip()
    _run_tests({"LD_PRELOAD": asan, "LSA_ORACLE_SO": so}, "tests/test_oracle.py")


@pytest.mark.skipif(not _no_device(), reason="the C-ABI tests force LSA_ERR_HIP only where no device exists")
def test_host_code_under_sanitizers(tmp_path):
    rts = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    if not rts:
        pytest.skip("no clang address-sanitizer runtime under /opt/rocm/llvm")
    so = str(tmp_path / "liblsa_san.so")
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    cmd = [hipcc, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-shared", "-fno-omit-frame-pointer",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-shared-libsan",
           *[os.path.join(CSRC, s) for s in SOURCES], "-o", so]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-4000:]
    nm = subprocess.run(["nm", "-D", so], capture_output=True, text=True).stdout
    assert "__asan_report" in nm and "__ubsan_handle" in nm, "host code was not instrumented"
    _run_tests({"LD_PRELOAD": rts[0], "LSA_LIB": so}, "tests/test_abi.py")
