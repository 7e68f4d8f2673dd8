"""ctypes binding of libgs_peaks.so: the device's own matrix-core, exp2, FMA,
streaming-read and LDS-read rates, timed with HIP events on the caller's stream.

`measure()` returns the rates as a dict; the work per launch follows the
formulas stated in include/gs_peaks.h.  Raises if the library is missing or
no GPU is present (there is no CPU stand-in for a rate measurement)."""
import ctypes
import os
import time

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(os.path.dirname(HERE), "libgs_peaks.so")
THREADS = 256
MFMA_CHAINS = 4
CHAINS = 8
LDS_READS = 4
EXPORTED = ("gs_peaks_mfma", "gs_peaks_exp", "gs_peaks_fma", "gs_peaks_read", "gs_peaks_lds")

_lib = None


def load(path=LIB_PATH):
    global _lib
    if _lib is None:
        if not os.path.exists(path):
            raise RuntimeError("libgs_peaks.so not built (run __graft_entry__.build())")
        lib = ctypes.CDLL(path)
        i64, i32, vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p
        lib.gs_peaks_mfma.argtypes = [vp, i64, i32, i32, vp]
        lib.gs_peaks_exp.argtypes = [vp, i64, i32, vp]
        lib.gs_peaks_fma.argtypes = [vp, i64, i32, vp]
        lib.gs_peaks_read.argtypes = [vp, i64, vp, i64, vp]
        lib.gs_peaks_lds.argtypes = [vp, i64, i32, vp]
        for name in EXPORTED:
            getattr(lib, name).restype = ctypes.c_int
        _lib = lib
    return _lib


def _check(rc, name):
    if rc != 0:
        raise RuntimeError("%s failed with status %d" % (name, rc))


def _time(torch, launch, reps, settle_s):
    """Average launch duration (s) over `reps` launches, after repeating the
    launch for `settle_s` seconds of wall time (the shader clock takes some
    tens of milliseconds of sustained load to reach its steady value)."""
    stream = torch.cuda.current_stream()
    t0 = time.perf_counter()
    while True:
        launch(stream.cuda_stream)
        torch.cuda.synchronize()
        if time.perf_counter() - t0 >= settle_s:
            break
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        launch(stream.cuda_stream)
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e-3 / reps


def measure(read_bytes=4 << 30, reps=20, settle_s=0.3):
    """Measured rates on cuda:0: fp16 MFMA flop/s (both shapes), exp2/s,
    fp32 FMA flop/s (unpacked), streaming-read bytes/s and LDS-read bytes/s
    (whole device)."""
    import torch

    lib = load()
    if not torch.cuda.is_available():
        raise RuntimeError("rate measurement needs a GPU")
    dev = torch.device("cuda:0")
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    wg = cus * 16
    out = torch.empty(wg * THREADS, dtype=torch.float32, device=dev)
    res = {"compute_units": cus, "workgroups": wg}

    iters = 4096
    for shape, key, flop in ((0, "mfma_f16_32x32x16", 32 * 32 * 16 * 2),
                             (1, "mfma_f16_16x16x32", 16 * 16 * 32 * 2)):
        t = _time(torch, lambda s, shape=shape: _check(
            lib.gs_peaks_mfma(out.data_ptr(), wg, iters // 4, shape, s), "gs_peaks_mfma"), reps, settle_s)
        res[key + "_flop_per_s"] = wg * (THREADS // 64) * (iters // 4) * MFMA_CHAINS * flop / t
    t = _time(torch, lambda s: _check(lib.gs_peaks_exp(out.data_ptr(), wg, iters, s), "gs_peaks_exp"), reps, settle_s)
    res["exp2_per_s"] = wg * THREADS * iters * CHAINS / t
    t = _time(torch, lambda s: _check(lib.gs_peaks_fma(out.data_ptr(), wg, iters, s), "gs_peaks_fma"), reps, settle_s)
    res["fma_f32_flop_per_s"] = 2.0 * wg * THREADS * iters * CHAINS / t

    # LDS reads: 8 workgroups per CU (at most 5 resident with 32 KiB each)
    lds_wg, lds_iters = cus * 8, 512
    rd = out.view(torch.int32)
    t = _time(torch, lambda s: _check(lib.gs_peaks_lds(rd.data_ptr(), lds_wg, lds_iters, s), "gs_peaks_lds"),
              reps, settle_s)
    res["lds_read_bytes_per_s"] = lds_wg * THREADS * lds_iters * LDS_READS * 16 / t

    # streaming read: the best of three grid sizes (4, 8, 16 workgroups per CU)
    buf = torch.ones(read_bytes // 4, dtype=torch.int32, device=dev)
    rd = out.view(torch.int32)
    best = None
    for per_cu in (4, 8, 16):
        g = cus * per_cu
        t = _time(torch, lambda s, g=g: _check(
            lib.gs_peaks_read(buf.data_ptr(), read_bytes, rd.data_ptr(), g, s), "gs_peaks_read"), reps, settle_s)
        if best is None or t < best[0]:
            best = (t, g)
    res["read_bytes_per_s"] = read_bytes / best[0]
    res["read_bytes"] = read_bytes
    res["read_workgroups"] = best[1]
    del buf
    return res
