"""The C ABI's validation layer (rola_api.cpp) built for the host with AddressSanitizer and
UndefinedBehaviorSanitizer (g++, no device code) and linked against the library's kernels, then
exercised by a driver whose every call is invalid (tests/asan/abi_checks.cpp): all must be rejected
with the expected status, and the sanitizers must report nothing. CPU only."""

import os
import shutil
import subprocess

import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2609_06712_amd")
LIB = os.path.join(PKG, "librola.so")


@pytest.mark.skipif(torch.cuda.device_count() > 0, reason="host-validation test: CPU only")
@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_abi_validation_under_asan(tmp_path):
    if not os.path.exists(LIB):
        pytest.skip("librola.so is not built")
    exe = str(tmp_path / "abi_checks")
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    sanitize = "-fsanitize=" + ",".join(("address", "undefined"))
    cmd = ["g++", "-std=c++17", "-g", "-O1", sanitize, "-fno-omit-frame-pointer",
           "-fno-sanitize-recover=undefined", "-D__HIP_PLATFORM_AMD__",
           f"-I{rocm}/include", f"-I{ROOT}/include", f"-I{PKG}/csrc",
           os.path.join(PKG, "csrc", "rola_api.cpp"), os.path.join(ROOT, "tests", "asan", "abi_checks.cpp"),
           f"-L{PKG}", "-lrola", f"-Wl,-rpath,{PKG}", f"-L{rocm}/lib", "-lamdhip64",
           f"-Wl,-rpath,{rocm}/lib", "-o", exe]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert run.returncode == 0, run.stdout[-2000:] + run.stderr[-4000:]
    assert "0 failed" in run.stdout, run.stdout
    assert "ERROR: AddressSanitizer" not in run.stderr and "runtime error" not in run.stderr, run.stderr
