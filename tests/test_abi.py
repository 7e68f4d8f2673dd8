"""The C-ABI library on the CPU: it loads, exports every symbol the header
declares, and rejects bad arguments before enqueuing any GPU work (these
calls use fake device addresses; validation never dereferences them)."""
import ctypes
import math
import os
import re
import subprocess

import pytest

from paper_2609_04910_amd import gauss_sum as gs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gauss_sum.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gauss_sum_\w+)\s*\(", text)))


def test_library_loads_and_exports_every_declared_symbol():
    lib = gs.load()
    names = declared_functions()
    assert set(names) == set(gs.EXPORTED), names
    out = subprocess.run(["nm", "-D", "--defined-only", gs.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (\w+)", out))
    for n in names:
        assert n in exported, n
        assert hasattr(lib, n)


def test_abi_version_and_status_strings():
    assert gs.gauss_sum_abi_version() == 1
    seen = set()
    for code in range(11):
        s = gs.status_string(code)
        assert s and s != "unknown status"
        seen.add(s)
    assert len(seen) == 11
    assert gs.status_string(1234) == "unknown status"


FAKE = 0x100000  # a 256-aligned fake device address, never dereferenced


def _fwd(M=8, N=8, D=4, C=2, qk=gs.GS_F16, vd=gs.GS_F32, q=FAKE, k=FAKE + 0x10000,
         v=FAKE + 0x20000, tau=1.0, out=FAKE + 0x30000, ws=FAKE + 0x100000, wsb=1 << 40, p=True):
    lib = gs.load()
    prob = gs.make_problem(M, N, D, C, qk, vd)
    pp = ctypes.byref(prob) if p else None
    return lib.gauss_sum_fwd(pp, q, k, v, ctypes.c_float(tau), out, ws, wsb, None)


def _bwd(M=8, N=8, D=4, C=2, qk=gs.GS_F16, vd=gs.GS_F32, gd=gs.GS_F32, tau=1.0,
         dq=FAKE + 0x40000, dk=FAKE + 0x50000, dv=FAKE + 0x60000, dout=FAKE + 0x70000,
         ws=FAKE + 0x100000, wsb=1 << 40):
    lib = gs.load()
    prob = gs.make_problem(M, N, D, C, qk, vd)
    return lib.gauss_sum_bwd(ctypes.byref(prob), FAKE, FAKE + 0x10000, FAKE + 0x20000,
                             ctypes.c_float(tau), dout, gd, dq, dk, dv, ws, wsb, None)


@pytest.mark.parametrize("kw,status", [
    (dict(p=False), 1),
    (dict(q=None), 1), (dict(k=None), 1), (dict(v=None), 1), (dict(out=None), 1),
    (dict(M=-1), 2), (dict(N=-3), 2), (dict(D=0), 2), (dict(D=257), 2), (dict(C=0), 2),
    (dict(C=300), 2), (dict(M=1 << 40), 2), (dict(M=(1 << 30) + 1), 2), (dict(N=(1 << 30) + 1), 2),
    (dict(tau=0.0), 3), (dict(tau=-1.0), 3), (dict(tau=float("nan")), 3),
    (dict(tau=float("inf")), 3),
    (dict(qk=gs.GS_F32, q=FAKE + 2), 5), (dict(qk=7), 4), (dict(vd=9), 4),
    (dict(q=FAKE + 1), 5), (dict(v=FAKE + 0x20002), 5), (dict(out=FAKE + 0x30002), 5),
    (dict(ws=FAKE + 0x100010), 5),
    (dict(ws=None), 6), (dict(wsb=16), 6),
    (dict(out=FAKE + 0x10000), 9), (dict(out=FAKE + 0x20004), 9), (dict(ws=FAKE + 0x30000 - 256), 9),
])
def test_fwd_validation(kw, status):
    assert _fwd(**kw) == status


@pytest.mark.parametrize("kw,status", [
    (dict(dq=None, dk=None, dv=None), 1), (dict(dout=None), 1),
    (dict(gd=5), 4), (dict(D=300), 2), (dict(tau=-2.0), 3),
    (dict(dq=FAKE + 0x40002), 5), (dict(dout=FAKE + 0x70002), 5),
    (dict(dq=FAKE + 0x10000), 9), (dict(dk=FAKE + 0x40000), 9), (dict(dv=FAKE + 0x70000), 9),
    (dict(wsb=1), 6), (dict(ws=None), 6),
])
def test_bwd_validation(kw, status):
    assert _bwd(**kw) == status


def _fb(M=8, N=8, D=4, C=2, out=FAKE + 0x30000, dq=FAKE + 0x40000, dk=None, dv=None,
        dout=FAKE + 0x70000, wsb=1 << 40):
    lib = gs.load()
    prob = gs.make_problem(M, N, D, C, gs.GS_F16, gs.GS_F32)
    return lib.gauss_sum_fwd_bwd(ctypes.byref(prob), FAKE, FAKE + 0x10000, FAKE + 0x20000,
                                 ctypes.c_float(1.0), dout, gs.GS_F32, out, dq, dk, dv,
                                 FAKE + 0x100000, wsb, None)


@pytest.mark.parametrize("kw,status", [
    (dict(out=None), 1), (dict(dout=None), 1), (dict(out=FAKE + 0x40000), 9),
    (dict(out=FAKE + 0x70000), 9), (dict(wsb=8), 6), (dict(D=0), 2),
])
def test_fwd_bwd_validation(kw, status):
    assert _fb(**kw) == status


def _flow(M=8, N=8, D=4, C=1, x=FAKE, v=FAKE + 0x20000, tau=1.0, s=FAKE + 0x30000,
          grad=FAKE + 0x40000, mmd2=FAKE + 0x50000, ws=FAKE + 0x100000, wsb=1 << 40, p=True):
    lib = gs.load()
    prob = gs.make_problem(M, N, D, C, gs.GS_F16, gs.GS_F32)
    pp = ctypes.byref(prob) if p else None
    return lib.gauss_sum_mmd_flow(pp, x, v, ctypes.c_float(tau), s, grad, mmd2, ws, wsb, None)


@pytest.mark.parametrize("kw,status", [
    (dict(p=False), 1), (dict(s=None, grad=None, mmd2=None), 1), (dict(x=None), 1),
    (dict(v=None), 1),
    (dict(N=9), 2), (dict(D=0), 2), (dict(C=2), 4), (dict(tau=0.0), 3),
    (dict(mmd2=FAKE + 0x50004), 5), (dict(s=FAKE + 0x30002), 5), (dict(wsb=64), 6), (dict(ws=None), 6),
    (dict(s=FAKE + 0x10), 9), (dict(grad=FAKE + 0x20000), 9), (dict(mmd2=FAKE + 0x30010), 9),
    (dict(mmd2=FAKE + 0x100100), 9), (dict(grad=FAKE + 0x30000), 9),
])
def test_mmd_flow_validation(kw, status):
    assert _flow(**kw) == status


def _fwd_b(count=3, qs=8 * 4, ks=8 * 4, vs=8 * 2, outs=8 * 2, M=8, N=8, D=4, C=2, q=FAKE,
           k=FAKE + 0x10000, v=FAKE + 0x20000, out=FAKE + 0x30000, ws=FAKE + 0x100000, wsb=1 << 40,
           batch=True):
    lib = gs.load()
    prob = gs.make_problem(M, N, D, C, gs.GS_F16, gs.GS_F32)
    b = gs.Batch(count, qs, ks, vs, 0, outs, 0, 0, 0)
    bp = ctypes.byref(b) if batch else None
    return lib.gauss_sum_fwd_batched(ctypes.byref(prob), bp, q, k, v, ctypes.c_float(1.0), out, ws,
                                     wsb, None)


@pytest.mark.parametrize("kw,status", [
    (dict(batch=False), 1), (dict(out=None), 1), (dict(count=-1), 2), (dict(qs=-8), 2),
    (dict(outs=15), 2), (dict(count=0), 0), (dict(count=0, out=None), 0), (dict(q=FAKE + 1), 5),
    (dict(out=FAKE + 0x20000 + 2 * 8 * 2 * 4), 9),  # third problem's out meets the v span
    (dict(outs=16, out=FAKE + 0x100000 - 64), 9),    # out span runs into the workspace
    (dict(wsb=16), 6), (dict(D=0), 2),
])
def test_fwd_batched_validation(kw, status):
    assert _fwd_b(**kw) == status


def test_bwd_batched_validation():
    lib = gs.load()
    prob = gs.make_problem(8, 8, 4, 2, gs.GS_F16, gs.GS_F32)
    b = gs.Batch(2, 32, 32, 16, 16, 0, 32, 32, 16)
    args = [FAKE, FAKE + 0x10000, FAKE + 0x20000, ctypes.c_float(1.0), FAKE + 0x70000, gs.GS_F32]
    ws = [FAKE + 0x100000, 1 << 40, None]
    assert lib.gauss_sum_bwd_batched(ctypes.byref(prob), ctypes.byref(b), *args, None, None, None,
                                     *ws) == 1
    empty = gs.Batch(0, 32, 32, 16, 16, 0, 32, 32, 16)
    assert lib.gauss_sum_bwd_batched(ctypes.byref(prob), ctypes.byref(empty), *args, None, None,
                                     None, *ws) == 0
    bad = gs.Batch(2, 32, 32, 16, 16, 0, 31, 32, 16)  # dq of problem 1 would overlap problem 0
    assert lib.gauss_sum_bwd_batched(ctypes.byref(prob), ctypes.byref(bad), *args, FAKE + 0x40000,
                                     None, None, *ws) == 2
    assert lib.gauss_sum_bwd_batched(ctypes.byref(prob), ctypes.byref(b), *args, FAKE + 0x40000,
                                     FAKE + 0x40000 + 64, None, *ws) == 9


def test_fwd_bwd_batched_validation():
    lib = gs.load()
    prob = gs.make_problem(8, 8, 4, 2, gs.GS_F16, gs.GS_F32)
    b = gs.Batch(2, 32, 32, 16, 16, 16, 32, 32, 16)
    args = [FAKE, FAKE + 0x10000, FAKE + 0x20000, ctypes.c_float(1.0), FAKE + 0x70000, gs.GS_F32]
    ws = [FAKE + 0x100000, 1 << 40, None]
    fn = lib.gauss_sum_fwd_bwd_batched
    assert fn(ctypes.byref(prob), None, *args, FAKE + 0x30000, None, None, None, *ws) == 1
    assert fn(ctypes.byref(prob), ctypes.byref(b), *args, None, FAKE + 0x40000, None, None, *ws) == 1
    empty = gs.Batch(0, 32, 32, 16, 16, 16, 32, 32, 16)
    assert fn(ctypes.byref(prob), ctypes.byref(empty), *args, None, None, None, None, *ws) == 0
    neg = gs.Batch(-1, 32, 32, 16, 16, 16, 32, 32, 16)
    assert fn(ctypes.byref(prob), ctypes.byref(neg), *args, None, None, None, None, *ws) == 2
    bad = gs.Batch(2, 32, 32, 16, 16, 15, 32, 32, 16)  # s of problem 1 would overlap problem 0
    assert fn(ctypes.byref(prob), ctypes.byref(bad), *args, FAKE + 0x30000, FAKE + 0x40000, None,
              None, *ws) == 2
    assert fn(ctypes.byref(prob), ctypes.byref(b), *args, FAKE + 0x30000, FAKE + 0x30000 + 64, None,
              None, *ws) == 9
    assert fn(ctypes.byref(prob), ctypes.byref(b), *args, FAKE + 0x30000, FAKE + 0x40000, None,
              None, FAKE + 0x100000, 16, None) == 6
    one = gs.gauss_sum_fwd_bwd_workspace_size(1000, 3000, 64, 1, want_dk=False, want_dv=False)
    assert gs.gauss_sum_fwd_bwd_batched_workspace_size(1000, 3000, 64, 1, 1, want_dk=False,
                                                       want_dv=False) == one
    assert gs.gauss_sum_fwd_bwd_batched_workspace_size(1000, 3000, 64, 1, 4, want_dk=False,
                                                       want_dv=False) == 4 * one


def test_svgd_validation():
    lib = gs.load()
    F16 = gs.GS_F16

    def call(M=64, N=64, D=8, C=8, qk=F16, x=FAKE, sc=FAKE + 0x10000, tau=1.0, phi=FAKE + 0x20000,
             ws=FAKE + 0x100000, wsb=1 << 40):
        prob = gs.make_problem(M, N, D, C, qk, gs.GS_F32)
        return lib.gauss_sum_svgd(ctypes.byref(prob), x, sc, ctypes.c_float(tau), phi, ws, wsb, None)

    assert call(N=63) == 2 and call(C=7) == 2 and call(D=300, C=300) == 2
    assert call(tau=0.0) == 3
    assert call(qk=gs.GS_F32) == 4
    assert call(phi=None) == 1 and call(x=None) == 1 and call(sc=None) == 1
    assert call(phi=FAKE + 0x20002) == 5
    assert call(phi=FAKE + 8) == 9               # phi meets x
    assert call(phi=FAKE + 0x100000 + 64) == 9   # phi inside the workspace
    assert call(wsb=16) == 6
    assert call(M=0, N=0, x=None, sc=None, ws=None, wsb=0) == 0
    w = gs.gauss_sum_svgd_workspace_size(1000, 64)
    assert w > 0 and w % 256 == 0
    assert w >= 1000 * 64 * 4 + gs.gauss_sum_fwd_workspace_size(1000, 1000, 64, 64)
    assert gs.gauss_sum_svgd_workspace_size(1000, 64, gs.GS_F32) == 0


def test_empty_query_set_is_a_noop():
    # M = 0: nothing to compute; no pointer is touched and no kernel runs.
    assert _fwd(M=0, q=None, out=None) == 0


def test_workspace_sizes():
    assert gs.gauss_sum_fwd_workspace_size(0, 5, 3, 1) == 0
    assert gs.gauss_sum_fwd_workspace_size(5, 0, 3, 1) == 0
    assert gs.gauss_sum_fwd_workspace_size(5, 5, 0, 1) == 0  # invalid
    a = gs.gauss_sum_fwd_workspace_size(4096, 4096, 16, 1)
    b = gs.gauss_sum_fwd_workspace_size(8192, 8192, 16, 1)
    assert 0 < a < b and a % 256 == 0
    assert gs.gauss_sum_bwd_workspace_size(64, 64, 8, 2, want_dq=False, want_dk=False,
                                           want_dv=False) == 0
    full = gs.gauss_sum_bwd_workspace_size(1000, 3000, 64, 4)
    only_dq = gs.gauss_sum_bwd_workspace_size(1000, 3000, 64, 4, want_dk=False, want_dv=False)
    assert 0 < only_dq < full
    fused = gs.gauss_sum_fwd_bwd_workspace_size(1000, 3000, 64, 4, want_dk=False, want_dv=False)
    assert fused >= only_dq and fused > 0
    assert gs.gauss_sum_fwd_bwd_workspace_size(1000, 3000, 64, 4, want_dq=False, want_dk=False,
                                               want_dv=False) == \
        gs.gauss_sum_fwd_workspace_size(1000, 3000, 64, 4)
    flow = gs.gauss_sum_mmd_flow_workspace_size(5000, 64)
    assert flow > gs.gauss_sum_fwd_bwd_workspace_size(5000, 5000, 64, 1, want_dk=False, want_dv=False)
    assert flow % 256 == 0


def test_f32_tier_validation():
    """fp32 points: the forward only (any C); gradients and the flow are
    unsupported, and points are aligned to 4 bytes."""
    lib = gs.load()
    F = gs.GS_F32
    assert _fwd(qk=F, C=2, q=FAKE + 2) == 5
    assert _fwd(qk=F, C=1, q=FAKE + 2) == 5
    assert _fwd(qk=F, C=1, out=FAKE + 0x10000 + 4 * 8 * 4 - 4) == 9  # out meets the k span (fp32 points)
    assert _bwd(qk=F, C=1) == 4
    prob = gs.make_problem(8, 8, 4, 1, F, gs.GS_F32)
    assert lib.gauss_sum_mmd_flow(ctypes.byref(prob), FAKE, FAKE + 0x20000, ctypes.c_float(1.0),
                                  FAKE + 0x30000, None, None, FAKE + 0x100000, 1 << 40, None) == 4
    assert gs.gauss_sum_mmd_flow_workspace_size(64, 8, F) == 0
    assert gs.gauss_sum_bwd_workspace_size(64, 64, 8, 1, F) == 0
    several = gs.gauss_sum_fwd_workspace_size(1000, 3000, 64, 100, F)
    assert several > gs.gauss_sum_fwd_workspace_size(1000, 3000, 64, 1, F) and several % 256 == 0
    one = gs.gauss_sum_fwd_workspace_size(1000, 3000, 64, 1, F)
    assert one > 0 and one % 256 == 0
    assert gs.gauss_sum_fwd_batched_workspace_size(1000, 3000, 64, 1, 1, F) == one


def test_batched_workspace_sizes():
    # one problem per group: exactly the single-problem workspace
    assert gs.gauss_sum_fwd_batched_workspace_size(1000, 3000, 64, 4, 1) == \
        gs.gauss_sum_fwd_workspace_size(1000, 3000, 64, 4)
    assert gs.gauss_sum_bwd_batched_workspace_size(1000, 3000, 64, 4, 1) == \
        gs.gauss_sum_bwd_workspace_size(1000, 3000, 64, 4)
    one = gs.gauss_sum_fwd_workspace_size(16384, 16384, 32, 1)
    many = gs.gauss_sum_fwd_batched_workspace_size(16384, 16384, 32, 1, 64)
    # 64 slices, each at most the single-problem one (fewer key splits)
    assert 0 < many <= 64 * one and many % (64 * 256) == 0 and many > one
    assert gs.gauss_sum_fwd_batched_workspace_size(64, 64, 8, 1, 0) == 0
    assert gs.gauss_sum_fwd_batched_workspace_size(0, 64, 8, 1, 4) == 0
    assert gs.gauss_sum_fwd_batched_workspace_size(64, 64, 0, 1, 4) == 0
    assert gs.gauss_sum_bwd_batched_workspace_size(64, 64, 8, 1, 4, want_dq=False, want_dk=False,
                                                   want_dv=False) == 0
    # groups stop at 65535 problems
    assert gs.gauss_sum_fwd_batched_workspace_size(64, 64, 8, 1, 1 << 20) == \
        gs.gauss_sum_fwd_batched_workspace_size(64, 64, 8, 1, 65535)


def test_profile_hook_arguments():
    lib = gs.load()
    assert lib.gauss_sum_profile_start(0, 1) == 2
    assert lib.gauss_sum_profile_start(4, 0) == 2
    assert lib.gauss_sum_profile_start(4, 4) == 2
    assert lib.gauss_sum_profile_stop(None, 0) == 0  # nothing started


def _noalloc(M=8, N=8, D=4, C=2, tau=1.0, p=True, out=FAKE + 0x30000):
    lib = gs.load()
    prob = gs.make_problem(M, N, D, C, gs.GS_F16, gs.GS_F32)
    return lib.gauss_sum_fwd_noalloc(ctypes.byref(prob) if p else None, FAKE, FAKE + 0x10000,
                                     FAKE + 0x20000, ctypes.c_float(tau), out, None)


def test_noalloc_validation_and_scratch_limit():
    assert _noalloc(p=False) == 1
    assert _noalloc(D=0) == 2
    assert _noalloc(tau=0.0) == 3
    # the built-in scratch holds GAUSS_SUM_NOALLOC_SCRATCH_BYTES: larger
    # problems are refused before anything is looked up or launched
    for M, N, D, C in ((1 << 22, 1 << 22, 256, 16), (1 << 20, 1 << 20, 64, 1), (4096, 1 << 22, 128, 1)):
        need = gs.gauss_sum_fwd_workspace_size(M, N, D, C)
        assert need > gs.NOALLOC_SCRATCH_BYTES
        assert _noalloc(M, N, D, C) == 10
    assert gs.gauss_sum_fwd_workspace_size(8, 8, 4, 2) <= gs.NOALLOC_SCRATCH_BYTES
    hdr = open(os.path.join(ROOT, "include", "gauss_sum.h")).read()
    assert "#define GAUSS_SUM_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)" in hdr
    assert gs.NOALLOC_SCRATCH_BYTES == 128 << 20


def test_no_device_reports_hip_error():
    # A valid call in a process without a usable GPU fails at launch, and the
    # failure is reported as GS_ERR_HIP rather than crashing.
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is visible")
    assert _fwd() == 7
    assert _noalloc() == 7
    assert _bwd() == 7
    assert _fb() == 7
    assert _flow() == 7
    assert _fwd_b() == 7
