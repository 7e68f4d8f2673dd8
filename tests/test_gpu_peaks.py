"""The rate-calibration kernels on the GPU: the streaming read touches every
16-byte word exactly once (the xor of its per-lane results equals the xor of
the buffer, for grids that leave ragged tails), and the measured rates are
positive and below the published peaks (the work accounting is not off by a
factor)."""
import numpy as np
import pytest
import torch

from paper_2609_04910_amd import peaks

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("words16,workgroups", [(1, 1), (1000, 3), (257 * 1024 + 5, 7), (1 << 20, 1024)])
def test_read_covers_every_word_once(words16, workgroups):
    lib = peaks.load()
    rng = np.random.default_rng(words16)
    host = rng.integers(0, 2**32, size=words16 * 4, dtype=np.uint64).astype(np.uint32)
    dev = torch.from_numpy(host.view(np.int32)).cuda()
    out = torch.full((workgroups * peaks.THREADS,), -1, dtype=torch.int32, device="cuda")
    rc = lib.gs_peaks_read(dev.data_ptr(), words16 * 16, out.data_ptr(), workgroups,
                           torch.cuda.current_stream().cuda_stream)
    assert rc == 0
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(out.cpu().numpy().view(np.uint32))
    assert got == np.bitwise_xor.reduce(host)


def test_measured_rates_are_plausible():
    r = peaks.measure(read_bytes=256 << 20, reps=2, settle_s=0.02)
    for key, nominal in (("mfma_f16_16x16x32_flop_per_s", 2.5e15), ("mfma_f16_32x32x16_flop_per_s", 2.5e15),
                         ("exp2_per_s", 256 * 4 * 8 * 2.4e9), ("fma_f32_flop_per_s", 157.3e12)):
        assert 0.05 * nominal < r[key] < 1.05 * nominal, (key, r[key])
    # LDS: between 128 and 256 bytes per CU and clock at 2.4 GHz
    assert 0.05 * 256 * 128 * 2.4e9 < r["lds_read_bytes_per_s"] < 1.05 * 256 * 256 * 2.4e9
    assert 1e11 < r["read_bytes_per_s"] < 2e13   # a 256 MiB buffer may be served from the 256 MB cache
