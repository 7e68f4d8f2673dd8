"""GPU parity of the fp32-accuracy tier (fp32 points, C = 1, forward) against
the fp64 oracle, element by element.

Pass rule: |gpu - oracle| <= 1e-5 * A + 1e-30 per element (A = sum_n Phi |v_n|,
the oracle's scale).  The bound follows from the arithmetic for exponents of
order one: split scores carry 22 significant bits (3 * 2^-22 of sum_d |q_d k_d|
after dropping lo.lo), the fp32 exponent terms 2^-24 each, exp2 one ulp, and
the fp32 sums at most (N/32 + 16) * 2^-24 of A; about 1e-6 of A for the shapes
here, so 1e-5 leaves a margin of ten.  Relative L2 error of s itself: signed
values cancel (|s_m| is about A_m / sqrt(N) for N(0, 1) values), so the same
per-term errors weigh about sqrt(N) times more relative to s: the checked
rows must stay within 3e-6 (the paper reports about 5e-7 for every fp32
method).  Positive values (s = A): the error of a row is then dominated by
what is fixed for the row -- the query's split error (2^-22 per coordinate,
times tau' and the kernel-weighted mean key), its half norm and tau' in fp32
-- about one fp32 ulp rms; the checked rows must stay within 2e-7.
"""
import sys

import numpy as np
import pytest

import oracle
import parity
from paper_2609_04910_amd import workloads as wl

pytestmark = pytest.mark.gpu

TOL32 = 1e-5
REL_L2 = 3e-6
REL_L2_POSITIVE = 2e-7


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


def points(seed, M, N, D, spread=1.0, vdt=np.float32):
    rng = np.random.default_rng(seed)
    q = (spread * rng.standard_normal((M, D))).astype(np.float32)
    k = (spread * rng.standard_normal((N, D))).astype(np.float32)
    v = rng.standard_normal((N, 1)).astype(vdt)
    return q, k, v


def check(label, got, q, k, v, tau, rows=None, rel_l2=True, bound=REL_L2):
    ref, scale = oracle.fwd(q, k, v, tau, rows=rows, threads=parity.oracle_threads())
    worst, rl2 = parity.compare(label, got if rows is None else got[rows], ref, scale, TOL32)
    _say("  %s: max err/A %.2e, rel-L2 %.2e" % (label, worst, rl2))
    if rel_l2:
        assert rl2 <= bound, (label, rl2)
    return worst, rl2


# (M, N, D, tau or None (= 1/D))
SHAPES = [
    (1, 1, 1, 0.7), (7, 5, 3, None), (63, 65, 16, None), (64, 64, 32, None), (65, 129, 17, None),
    (129, 300, 64, None), (300, 257, 128, None), (100, 150, 255, None), (96, 200, 256, None),
    (33, 1000, 15, None), (1000, 33, 1, 2.0), (768, 777, 64, None), (1300, 600, 32, None),
    (517, 2000, 40, None),
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "M%d_N%d_D%d" % s[:3])
def test_f32_small_shapes_all_outputs(shape):
    import torch
    from paper_2609_04910_amd import gauss_sum as gs
    M, N, D, tau = shape
    tau = np.float32(1.0 / D if tau is None else tau)
    q, k, v = points(SHAPES.index(shape), M, N, D)
    out = gs.gauss_sum_fwd(*(torch.from_numpy(a).cuda() for a in (q, k, v)), float(tau))
    torch.cuda.synchronize()
    check("f32 %s" % (shape,), out.cpu().numpy(), q, k, v, float(tau), rel_l2=M * N > 1000)


def test_f32_value_dtypes_zeros_signs_and_same_points():
    import torch
    from paper_2609_04910_amd import gauss_sum as gs
    q, k, v = points(21, 400, 700, 24, vdt=np.float16)
    v[::5] = 0
    v[1::7] = -np.abs(v[1::7])
    tq, tk, tv = (torch.from_numpy(a).cuda() for a in (q, k, v))
    out = gs.gauss_sum_fwd(tq, tk, tv, 1.0 / 24)
    torch.cuda.synchronize()
    check("f32 fp16 values", out.cpu().numpy(), q, k, v, float(np.float32(1.0 / 24)))
    # q and k the same array
    x = q[:300]
    tx = torch.from_numpy(x).cuda()
    vx = np.random.default_rng(3).standard_normal((300, 1)).astype(np.float32)
    s = gs.gauss_sum_fwd(tx, tx, torch.from_numpy(vx).cuda(), 0.5)
    s2 = gs.gauss_sum_fwd(tx, tx.clone(), torch.from_numpy(vx).cuda(), 0.5)
    torch.cuda.synchronize()
    assert torch.equal(s, s2)
    check("f32 same points", s.cpu().numpy(), x, x, vx, 0.5)


def test_f32_large_and_tiny_coordinates():
    """Scale invariance of the split: points scaled by 2^20 with tau by 2^-40
    give the same sums (the power-of-two scales are exact)."""
    import torch
    from paper_2609_04910_amd import gauss_sum as gs
    q, k, v = points(5, 300, 500, 20)
    tv = torch.from_numpy(v).cuda()
    a = gs.gauss_sum_fwd(torch.from_numpy(q).cuda(), torch.from_numpy(k).cuda(), tv, 0.05)
    for e in (20, -20):
        f = np.float32(2.0 ** e)
        b = gs.gauss_sum_fwd(torch.from_numpy(q * f).cuda(), torch.from_numpy(k * f).cuda(), tv,
                             float(0.05 / float(f) ** 2))
        torch.cuda.synchronize()
        assert torch.equal(a, b), e
    check("f32 scaled", a.cpu().numpy(), q, k, v, 0.05)


def test_f32_deterministic_and_batched():
    import torch
    from paper_2609_04910_amd import gauss_sum as gs
    q, k, v, tau = wl.make_batch("batch_d32_f32", seed=4, B=5, M=1100)
    tq, tk, tv = (torch.from_numpy(a).cuda() for a in (q, k, v))
    a = gs.gauss_sum_fwd_batched(tq, tk, tv, float(tau))
    b = gs.gauss_sum_fwd_batched(tq, tk, tv, float(tau))
    one = gs.gauss_sum_fwd_batched(tq, tk, tv, float(tau), group=1)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    for i in range(5):
        assert torch.equal(one[i], gs.gauss_sum_fwd(tq[i], tk[i], tv[i], float(tau)))
        check("f32 batch[%d]" % i, a[i].cpu().numpy(), q[i], k[i], v[i], float(tau))


def test_f32_unsupported_requests_raise():
    import torch
    from paper_2609_04910_amd import gauss_sum as gs
    q = torch.randn(10, 4, device="cuda")
    v = torch.randn(10, 1, device="cuda")
    with pytest.raises(gs.GaussSumError):
        gs.gauss_sum_bwd(q, q, v, 1.0, torch.randn(10, 1, device="cuda"))
    with pytest.raises(gs.GaussSumError):
        gs.gauss_sum_fwd(q, q, torch.randn(10, 2, device="cuda"), 1.0)


def test_f32_benchmark_batch_full_size_sampled_rows():
    """B = 64 fp32 clouds of 16384 points, D = 32 (the paper's single-precision
    D sweep), all problems in one launch group; sampled rows of three problems
    against all keys."""
    import torch
    from paper_2609_04910_amd import gauss_sum as gs
    q, k, v, tau = wl.make_batch("batch_d32_f32", seed=0)
    B, M = q.shape[0], q.shape[1]
    tq, tk, tv = (torch.from_numpy(a).cuda() for a in (q, k, v))
    out = gs.gauss_sum_fwd_batched(tq, tk, tv, float(tau)).cpu().numpy()
    rows = wl.sample_rows(M, 512, seed=3)
    for b in (0, B // 2 + 1, B - 1):
        check("batch_d32_f32[%d]" % b, out[b], q[b], k[b], v[b], float(tau), rows=rows)


def test_f32_positive_values_full_size():
    """Positive values (a density estimate): no cancellation, so the relative
    L2 error of s is the per-term error itself."""
    import torch
    from paper_2609_04910_amd import gauss_sum as gs
    q, k, v, tau = wl.make_batch("batch_d32_f32", seed=6, B=2)
    v = np.abs(v)
    tq, tk, tv = (torch.from_numpy(a).cuda() for a in (q, k, v))
    out = gs.gauss_sum_fwd_batched(tq, tk, tv, float(tau)).cpu().numpy()
    rows = wl.sample_rows(q.shape[1], 512, seed=5)
    for b in range(2):
        check("positive[%d]" % b, out[b], q[b], k[b], v[b], float(tau), rows=rows,
              bound=REL_L2_POSITIVE)
