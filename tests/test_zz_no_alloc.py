"""gauss_sum_fwd_noalloc (the forward entry point that allocates nothing and
uses the library's built-in scratch array) through the C ABI: bitwise equal
to gauss_sum_fwd with a caller workspace, and within the stated tolerance
of the fp64 oracle, on two calls in a row with the second problem smaller
(the scratch keeps the first call's contents), plus its argument checks on
the device."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from paper_2609_04910_amd import gauss_sum as gs

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _problem(seed, M, N, D, C, qk=np.float16, vdt=np.float32):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((M, D)).astype(qk)
    k = rng.standard_normal((N, D)).astype(qk)
    v = rng.standard_normal((N, C)).astype(vdt)
    return q, k, v, np.float32(1.0 / D)


def _noalloc(tq, tk, tv, tau, out):
    lib = gs.load()
    M, D = tq.shape
    N, C = tv.shape
    p = gs.make_problem(M, N, D, C, gs._dtype_code(tq.dtype), gs._dtype_code(tv.dtype))
    return lib.gauss_sum_fwd_noalloc(ctypes.byref(p), gs._ptr(tq), gs._ptr(tk), gs._ptr(tv), float(tau),
                                     gs._ptr(out), ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))


def test_two_calls_in_a_row_second_smaller():
    shapes = [(3001, 2600, 64, 3), (700, 513, 20, 1)]
    for seed, (M, N, D, C) in enumerate(shapes):
        q, k, v, tau = _problem(seed, M, N, D, C)
        tq, tk, tv = (torch.from_numpy(a).to(DEV) for a in (q, k, v))
        out = torch.full((M, C), float("nan"), dtype=torch.float32, device=DEV)
        assert _noalloc(tq, tk, tv, tau, out) == 0
        ref = gs.gauss_sum_fwd(tq, tk, tv, float(tau))   # caller workspace
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        assert np.array_equal(got.view(np.uint32), ref.cpu().numpy().view(np.uint32)), (M, N, D, C)
        val, scale = oracle.fwd(q, k, v, float(tau))
        err = np.abs(got.astype(np.float64) - val)
        assert np.all(err <= 2e-3 * scale + 1e-30), float(np.max(err / scale))


def test_same_array_for_q_and_k_and_bf16():
    q, _, v, tau = _problem(7, 1500, 1500, 33, 5)
    bits = (q.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    tq = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(DEV)
    tv = torch.from_numpy(v).to(DEV)
    out = torch.empty((1500, 5), dtype=torch.float32, device=DEV)
    assert _noalloc(tq, tq, tv, tau, out) == 0
    ref = gs.gauss_sum_fwd(tq, tq, tv, float(tau))
    torch.cuda.synchronize()
    assert torch.equal(out, ref)


def test_device_side_validation_and_limit():
    q, k, v, tau = _problem(3, 64, 64, 8, 2)
    tq, tk, tv = (torch.from_numpy(a).to(DEV) for a in (q, k, v))
    out = torch.zeros((64, 2), dtype=torch.float32, device=DEV)
    lib = gs.load()
    p = gs.make_problem(64, 64, 8, 2, gs.GS_F16, gs.GS_F32)
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    assert lib.gauss_sum_fwd_noalloc(ctypes.byref(p), gs._ptr(tq), gs._ptr(tk), gs._ptr(tv), float(tau),
                                     None, s) == 1
    assert lib.gauss_sum_fwd_noalloc(ctypes.byref(p), ctypes.c_void_p(tq.data_ptr() + 1), gs._ptr(tk),
                                     gs._ptr(tv), float(tau), gs._ptr(out), s) == 5
    # an output overlapping an input
    assert lib.gauss_sum_fwd_noalloc(ctypes.byref(p), gs._ptr(tq), gs._ptr(tk), gs._ptr(tv), float(tau),
                                     ctypes.c_void_p(tv.data_ptr()), s) == 9
    big = gs.make_problem(1 << 22, 1 << 22, 256, 16, gs.GS_F16, gs.GS_F32)
    assert lib.gauss_sum_fwd_noalloc(ctypes.byref(big), gs._ptr(tq), gs._ptr(tk), gs._ptr(tv), float(tau),
                                     gs._ptr(out), s) == 10
    torch.cuda.synchronize()
    assert torch.count_nonzero(out) == 0      # nothing was launched
    # M = 0 is a no-op, N = 0 writes zeros (no scratch needed)
    z = gs.make_problem(64, 0, 8, 2, gs.GS_F16, gs.GS_F32)
    out.fill_(5.0)
    assert lib.gauss_sum_fwd_noalloc(ctypes.byref(z), gs._ptr(tq), gs._ptr(tk), gs._ptr(tv), float(tau),
                                     gs._ptr(out), s) == 0
    torch.cuda.synchronize()
    assert torch.count_nonzero(out) == 0
