"""GPU: the batched entry points against the fp64 oracle, problem by problem.

Problems of a batch share each launch (grid.z indexes the problem) as far as
the workspace allows.  With a workspace of one problem's slice they run one at
a time through the same kernels as the single-problem calls and equal those bit
for bit; with larger groups the key-range split may differ (another fp32
summation order), so the results are checked against the oracle and for
bitwise reproducibility.  Also: shared key sets (stride 0), q and k the same
array, groups of every size in between, empty batches, and the full-size
benchmark batch on sampled rows of several problems.
"""
import sys

import numpy as np
import pytest

import oracle
import parity
from paper_2609_04910_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    from paper_2609_04910_amd import gauss_sum as gs
    gs.load()
    yield


def clouds(seed, B, M, N, D, C, shared=False):
    """B independent N(0, I)/sqrt(D) clouds (the paper's benchmark inputs), fp16."""
    rng = np.random.default_rng(seed)
    q = (rng.standard_normal((B, M, D)) / np.sqrt(D)).astype(np.float16)
    kb = 1 if shared else B
    k = (rng.standard_normal((kb, N, D)) / np.sqrt(D)).astype(np.float16)
    v = rng.standard_normal((kb, N, C)).astype(np.float32)
    g = rng.standard_normal((B, M, C)).astype(np.float32)
    if shared:
        k, v = k[0], v[0]
    return q, k, v, g


def check_problem(label, b, q, k, v, g, tau, out, dq=None, dk=None, dv=None):
    th = parity.oracle_threads()
    tol = parity.TOL["f16"]
    kb = k if k.ndim == 2 else k[b]
    vb = v if v.ndim == 2 else v[b]
    ref, scale = oracle.fwd(q[b], kb, vb, tau, threads=th)
    if out is not None:
        parity.compare("%s fwd[%d]" % (label, b), out[b].cpu().numpy(), ref, scale, tol)
    for name, got, fn in (("dq", dq, oracle.dq), ("dk", dk, oracle.dk), ("dv", dv, oracle.dv)):
        if got is not None:
            ref, scale = fn(q[b], kb, vb, g[b], tau, threads=th)
            parity.compare("%s %s[%d]" % (label, name, b), got[b].cpu().numpy(), ref, scale, tol)


SHAPES = [(4, 300, 517, 32, 1), (3, 64, 1000, 64, 3), (5, 129, 97, 17, 2), (6, 700, 640, 16, 1)]


@pytest.mark.parametrize("B,M,N,D,C", SHAPES + [(2, 100, 300, 256, 5)])
def test_batched_matches_oracle_every_problem(B, M, N, D, C):
    import torch
    from paper_2609_04910_amd import gauss_sum as gs
    _say("batched", B, M, N, D, C)
    q, k, v, g = clouds(B * 100 + D, B, M, N, D, C)
    tq, tk, tv, tg = (parity.to_torch(a) for a in (q, k, v, g))
    tau = 1.0
    out = gs.gauss_sum_fwd_batched(tq, tk, tv, tau)
    dq, dk, dv = gs.gauss_sum_bwd_batched(tq, tk, tv, tau, tg)
    torch.cuda.synchronize()
    for b in range(B):
        check_problem("all-in-one-group", b, q, k, v, g, tau, out, dq, dk, dv)
    # reproducible bit for bit
    out2 = gs.gauss_sum_fwd_batched(tq, tk, tv, tau)
    d2 = gs.gauss_sum_bwd_batched(tq, tk, tv, tau, tg)
    torch.cuda.synchronize()
    assert torch.equal(out, out2)
    for x, y in zip((dq, dk, dv), d2):
        assert torch.equal(x, y)


@pytest.mark.parametrize("B,M,N,D,C", SHAPES[:2])
def test_one_slice_workspace_equals_single_calls(B, M, N, D, C):
    import torch
    from paper_2609_04910_amd import gauss_sum as gs
    q, k, v, g = clouds(B * 100 + D + 1, B, M, N, D, C)
    tq, tk, tv, tg = (parity.to_torch(a) for a in (q, k, v, g))
    out = gs.gauss_sum_fwd_batched(tq, tk, tv, 1.0, group=1)
    dq, dk, dv = gs.gauss_sum_bwd_batched(tq, tk, tv, 1.0, tg, group=1)
    torch.cuda.synchronize()
    for b in range(B):
        s1 = gs.gauss_sum_fwd(tq[b], tk[b], tv[b], 1.0)
        d1 = gs.gauss_sum_bwd(tq[b], tk[b], tv[b], 1.0, tg[b])
        torch.cuda.synchronize()
        assert torch.equal(out[b], s1)
        for x, y in zip((dq, dk, dv), d1):
            assert torch.equal(x[b], y)


@pytest.mark.parametrize("B,M,N,D,C", [SHAPES[0], SHAPES[1], (4, 257, 1500, 32, 1), (3, 130, 700, 256, 16)])
def test_fwd_bwd_batched(B, M, N, D, C):
    """gauss_sum_fwd_bwd_batched: every problem against the oracle (all four
    outputs, one launch group), bitwise equal to the single-problem
    gauss_sum_fwd_bwd calls with a one-slice workspace, and to a repeat."""
    import torch
    from paper_2609_04910_amd import gauss_sum as gs
    q, k, v, g = clouds(B * 100 + D + 7, B, M, N, D, C)
    tq, tk, tv, tg = (parity.to_torch(a) for a in (q, k, v, g))
    tau = 1.0
    res = gs.gauss_sum_fwd_bwd_batched(tq, tk, tv, tau, tg)
    torch.cuda.synchronize()
    for b in range(B):
        check_problem("fwd_bwd_batched", b, q, k, v, g, tau, *res)
    again = gs.gauss_sum_fwd_bwd_batched(tq, tk, tv, tau, tg)
    one = gs.gauss_sum_fwd_bwd_batched(tq, tk, tv, tau, tg, want=(True, False, False), group=1)
    torch.cuda.synchronize()
    for x, y in zip(res, again):
        assert torch.equal(x, y)
    assert one[2] is None and one[3] is None
    for b in range(B):
        s1, dq1, _, _ = gs.gauss_sum_fwd_bwd(tq[b], tk[b], tv[b], tau, tg[b], want=(True, False, False))
        torch.cuda.synchronize()
        assert torch.equal(one[0][b], s1) and torch.equal(one[1][b], dq1)


def test_every_group_size():
    """B = 5 with room for 1 .. 5 problems per launch: each grouping matches the oracle."""
    import torch
    from paper_2609_04910_amd import gauss_sum as gs
    B, M, N, D, C = 5, 200, 333, 24, 2
    q, k, v, g = clouds(11, B, M, N, D, C)
    tq, tk, tv, tg = (parity.to_torch(a) for a in (q, k, v, g))
    for grp in range(1, B + 1):
        _say("group", grp)
        out = gs.gauss_sum_fwd_batched(tq, tk, tv, 0.5, group=grp)
        dq, dk, dv = gs.gauss_sum_bwd_batched(tq, tk, tv, 0.5, tg, group=grp)
        torch.cuda.synchronize()
        for b in range(B):
            check_problem("group %d" % grp, b, q, k, v, g, 0.5, out, dq, dk, dv)


def test_batched_shared_keys_same_points_and_empty():
    import torch
    from paper_2609_04910_amd import gauss_sum as gs
    q, k, v, g = clouds(7, 6, 200, 333, 48, 2, shared=True)
    tq, tk, tv, tg = (parity.to_torch(a) for a in (q, k, v, g))
    out = gs.gauss_sum_fwd_batched(tq, tk, tv, 1.0)
    dq, _, _ = gs.gauss_sum_bwd_batched(tq, tk, tv, 1.0, tg, want=(True, False, False))
    torch.cuda.synchronize()
    for b in range(6):
        check_problem("shared keys", b, q, k, v, g, 1.0, out, dq)
    # q and k the same array in every problem (one point set per problem)
    x, _, _, gx = clouds(8, 4, 300, 300, 20, 1)
    vx = np.random.default_rng(9).standard_normal((4, 300, 1)).astype(np.float32)
    tx, tvx, tgx = (parity.to_torch(a) for a in (x, vx, gx))
    out = gs.gauss_sum_fwd_batched(tx, tx, tvx, 2.0)
    dq, dk, dv = gs.gauss_sum_bwd_batched(tx, tx, tvx, 2.0, tgx)
    torch.cuda.synchronize()
    for b in range(4):
        check_problem("same points", b, x, x, vx, gx, 2.0, out, dq, dk, dv)
    empty = gs.gauss_sum_fwd_batched(tq[:0], tk, tv, 1.0)
    assert empty.shape == (0, 200, 2)


def test_benchmark_batch_full_size_sampled_rows():
    """The benchmark batch (B = 64 clouds of 16384 points, D = 32) in the launch
    configuration the benchmark times (all problems in one group); sampled
    query rows of the first, a middle and the last problem against all keys."""
    import torch
    from paper_2609_04910_amd import gauss_sum as gs
    q, k, v, tau = wl.make_batch("batch_d32", seed=0)
    B, M = q.shape[0], q.shape[1]
    tq, tk, tv = (torch.from_numpy(a).cuda() for a in (q, k, v))
    out = gs.gauss_sum_fwd_batched(tq, tk, tv, float(tau)).cpu().numpy()
    rows = wl.sample_rows(M, 512, seed=3)
    for b in (0, B // 2 + 1, B - 1):
        ref, scale = oracle.fwd(q[b], k[b], v[b], float(tau), rows=rows, threads=parity.oracle_threads())
        stats = parity.compare("batch_d32[%d]" % b, out[b][rows], ref, scale, parity.TOL["f16"])
        _say("  problem", b, "max err/A, rel-L2", stats)
