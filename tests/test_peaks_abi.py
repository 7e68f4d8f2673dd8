"""The rate-calibration library on the CPU: it loads, exports every function
include/gs_peaks.h declares, and rejects invalid arguments before any launch
(fake device addresses, never dereferenced)."""
import os
import re
import subprocess

from paper_2609_04910_amd import peaks

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gs_peaks.h")
FAKE = 0x100000


def test_exports_every_declared_symbol():
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    names = set(re.findall(r"\b(gs_peaks_\w+)\s*\(", text))
    assert names == set(peaks.EXPORTED)
    out = subprocess.run(["nm", "-D", "--defined-only", peaks.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (\w+)", out))
    assert names <= exported
    # the header's constants are the binding's
    for macro, val in (("GS_PEAKS_THREADS", peaks.THREADS), ("GS_PEAKS_MFMA_CHAINS", peaks.MFMA_CHAINS),
                       ("GS_PEAKS_CHAINS", peaks.CHAINS), ("GS_PEAKS_LDS_READS", peaks.LDS_READS)):
        assert re.search(r"#define %s (\d+)" % macro, text).group(1) == str(val)


def test_invalid_arguments_rejected_before_launch():
    lib = peaks.load()
    assert lib.gs_peaks_mfma(None, 4, 1, 0, None) == 1
    assert lib.gs_peaks_mfma(FAKE, 0, 1, 0, None) == 1
    assert lib.gs_peaks_mfma(FAKE, 4, 0, 0, None) == 1
    assert lib.gs_peaks_mfma(FAKE, 4, 1, 2, None) == 1
    assert lib.gs_peaks_mfma(FAKE, 1 << 31, 1, 0, None) == 1
    assert lib.gs_peaks_exp(None, 4, 1, None) == 1
    assert lib.gs_peaks_exp(FAKE, -1, 1, None) == 1
    assert lib.gs_peaks_fma(FAKE, 4, -3, None) == 1
    assert lib.gs_peaks_read(None, 16, FAKE, 4, None) == 1
    assert lib.gs_peaks_read(FAKE, 24, FAKE, 4, None) == 1        # not a multiple of 16
    assert lib.gs_peaks_read(FAKE + 8, 16, FAKE, 4, None) == 1    # misaligned
    assert lib.gs_peaks_read(FAKE, 0, FAKE, 4, None) == 1
    assert lib.gs_peaks_read(FAKE, 16, None, 4, None) == 1
    assert lib.gs_peaks_lds(None, 4, 1, None) == 1
    assert lib.gs_peaks_lds(FAKE, 0, 1, None) == 1
    assert lib.gs_peaks_lds(FAKE, 4, 0, None) == 1
