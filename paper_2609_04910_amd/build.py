"""Build the gfx950 HIP libraries in-tree (hipcc, no JIT cache): libgauss_sum.so
(the Gauss-sum kernels and their C ABI) and libgs_peaks.so (the rate
calibration kernels the benchmark measures the device's own rates with).

Flags: -O3 for gfx950 only; packed fp32 instructions are disabled in the
device code (-Xclang -target-feature -Xclang -packed-fp32-ops).
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(HERE, "csrc", "gauss_sum.hip")
LIB = os.path.join(HERE, "libgauss_sum.so")
PEAKS_SRC = os.path.join(HERE, "peaks", "gs_peaks.hip")
PEAKS_LIB = os.path.join(HERE, "libgs_peaks.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # matrix-core results in ordinary VGPRs: the exponent and conversion
    # instructions then read them without accumulator-register copies
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    "-Wall", "-Wno-unused-result",
    "-I", os.path.join(ROOT, "include"),
]


def build(verbose: bool = False) -> str:
    """Compile csrc/gauss_sum.hip into libgauss_sum.so and peaks/gs_peaks.hip
    into libgs_peaks.so; returns the path of libgauss_sum.so."""
    compile_one(PEAKS_SRC, PEAKS_LIB, verbose)
    return compile_one(SRC, LIB, verbose)


def compile_one(src: str, lib: str, verbose: bool) -> str:
    tmp = lib + ".tmp%d" % os.getpid()
    cmd = [HIPCC] + FLAGS + ["-o", tmp, src]
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "not a recognized feature for this target"
    msgs = "\n".join(ln for ln in (res.stdout + res.stderr).splitlines() if noise not in ln)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed (%d):\n%s" % (res.returncode, msgs))
    if verbose and msgs.strip():
        print(msgs)
    os.replace(tmp, lib)
    return lib


def sources():
    d = os.path.join(HERE, "csrc")
    return [os.path.join(d, f) for f in sorted(os.listdir(d))] + [
        os.path.join(ROOT, "include", "gauss_sum.h")]


if __name__ == "__main__":
    print(build(verbose=True))
