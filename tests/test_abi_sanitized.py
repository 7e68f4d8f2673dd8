"""The library's host code (argument validation, planning, workspace layout,
status strings) under AddressSanitizer and UndefinedBehaviorSanitizer: the
library is built with both on the host side only (the device code is
compiled as usual and never runs here) and the CPU tests of the C ABI run
against it in a child process with the ASan runtime preloaded.  Any
out-of-bounds access, use after free or undefined operation aborts the run."""
import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2609_04910_amd", "csrc", "gauss_sum.hip")
RUNNER = os.path.join(ROOT, "tests", "abi_runner.py")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _asan_runtime():
    found = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return found[-1] if found else None


@pytest.mark.skipif(_asan_runtime() is None or shutil.which(HIPCC) is None and not os.path.exists(HIPCC)
                    or bool(os.environ.get("LD_PRELOAD")),
                    reason="needs hipcc, clang's AddressSanitizer runtime and no other preloaded library")
def test_abi_cpu_tests_clean_under_host_sanitizers(tmp_path):
    lib = str(tmp_path / "libgauss_sum_san.so")
    cmd = [HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-shared",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "include"), "-Wno-unused-result", "-o", lib, SRC]
    subprocess.run(cmd, check=True, capture_output=True, timeout=900)
    env = dict(os.environ, LD_PRELOAD=_asan_runtime(),
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    res = subprocess.run([sys.executable, RUNNER, lib], capture_output=True, text=True, env=env,
                         timeout=600)
    out = res.stdout + res.stderr
    assert res.returncode == 0, out[-6000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-6000:]
