"""The C ABI from C: tests/c/abi_consumer.c includes include/gauss_sum.h in a
C11 translation unit (gcc, -Werror), links the in-tree library and checks the
host-side contract (version, workspace sizes, status strings, argument
validation) without a GPU."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIBDIR = os.path.join(ROOT, "paper_2609_04910_amd")


@pytest.mark.skipif(shutil.which("gcc") is None or not os.path.exists(os.path.join(LIBDIR, "libgauss_sum.so")),
                    reason="needs gcc and the built library")
def test_c_consumer(tmp_path):
    exe = str(tmp_path / "abi_consumer")
    subprocess.run(["gcc", "-std=c11", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
                    "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include",
                    "-o", exe, os.path.join(ROOT, "tests", "c", "abi_consumer.c"),
                    "-L", LIBDIR, "-lgauss_sum", "-Wl,-rpath," + LIBDIR, "-lm"], check=True)
    res = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stdout + res.stderr
    assert res.stdout.strip().endswith("0 failed")
