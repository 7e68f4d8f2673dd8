"""GPU parity of the fp32-accuracy tier (fp32 points, forward; one channel and
several) against the fp64 oracle, element by element.

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


def points(seed, M, N, D, spread=1.0, vdt=np.float32, C=1):
    rng = np.random.default_rng(seed)
    q = (spread * rng.standard_normal((M, D))).astype(np.float32)
    k = (spread * rng.standard_normal((N, D))).astype(np.float32)
    v = rng.standard_normal((N, C)).astype(vdt)
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
        gs.gauss_sum_fwd_bwd(q, q, v, 1.0, torch.randn(10, 1, device="cuda"))


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


# (M, N, D, C, tau or None (= 1/D)): channel counts around the 16-row tiles
# and the 64-channel launches
SHAPES_C = [
    (7, 5, 3, 2, None), (65, 129, 17, 15, None), (129, 300, 64, 16, None), (300, 257, 32, 17, None),
    (517, 700, 40, 32, None), (200, 333, 128, 64, None), (100, 150, 255, 65, None), (96, 200, 16, 100, 0.3),
    (64, 500, 8, 256, None),
]


@pytest.mark.parametrize("shape", SHAPES_C, ids=lambda s: "M%d_N%d_D%d_C%d" % s[:4])
def test_f32_several_channels_all_outputs(shape):
    import torch
    from paper_2609_04910_amd import gauss_sum as gs
    M, N, D, C, tau = shape
    tau = np.float32(1.0 / D if tau is None else tau)
    q, k, v = points(100 + SHAPES_C.index(shape), M, N, D, C=C)
    out = gs.gauss_sum_fwd(*(torch.from_numpy(a).cuda() for a in (q, k, v)), float(tau))
    torch.cuda.synchronize()
    check("f32 %s" % (shape,), out.cpu().numpy(), q, k, v, float(tau), rel_l2=M * N > 1000)


def test_f32_several_channels_tiny_kernel_values():
    """Rows whose kernel values are all far below 1 (sums down to ~1e-20): the
    exact row-maximum shift keeps full precision; checked relative to A with
    no absolute floor.  The exponent terms here are far from order one
    (tau' (||q||^2 + ||k||^2) up to ~190), and the fp32 rounding of the
    expanded exponent scales with them, so the bound per row is
    1e-5 * max(1, M_m / 2) with M_m = tau' (||q_m||^2 + max_n ||k_n||^2)."""
    import torch
    from paper_2609_04910_amd import gauss_sum as gs
    q, k, v = points(31, 300, 400, 8, spread=2.0, C=5)
    tau = 2.0
    out = gs.gauss_sum_fwd(*(torch.from_numpy(a).cuda() for a in (q, k, v)), tau).cpu().numpy()
    ref, A = oracle.fwd(q, k, v, tau, threads=parity.oracle_threads())
    assert 1e-36 < A.min() < 1e-12, (A.min(), A.max())  # rows with tiny sums are present
    rel = np.abs(out.astype(np.float64) - ref) / A
    tau2 = tau * np.log2(np.e)
    mag = tau2 * ((q.astype(np.float64) ** 2).sum(1) + (k.astype(np.float64) ** 2).sum(1).max())
    bound = TOL32 * np.maximum(1.0, mag / 2)[:, None]
    _say("  tiny values: A in [%.1e, %.1e], max err/A %.2e, max err/bound %.2f" %
         (A.min(), A.max(), rel.max(), (rel / bound).max()))
    assert np.all(rel <= bound)


def test_f32_several_channels_positive_and_batched():
    import torch
    from paper_2609_04910_amd import gauss_sum as gs
    q, k, v, tau = wl.make_batch("batch_c32_f32", seed=7, B=3, M=2000)
    v = np.abs(v)
    tq, tk, tv = (torch.from_numpy(a).cuda() for a in (q, k, v))
    a = gs.gauss_sum_fwd_batched(tq, tk, tv, float(tau))
    b = gs.gauss_sum_fwd_batched(tq, tk, tv, float(tau))
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    for i in range(3):
        check("c32 positive[%d]" % i, a[i].cpu().numpy(), q[i], k[i], v[i], float(tau),
              bound=REL_L2_POSITIVE)


def test_f32_several_channels_benchmark_batch_full_size():
    """B = 4 fp32 clouds, N = 16384, D = C = 32 (the paper's single-precision
    N sweep), all problems in one launch group; sampled rows of two problems."""
    import torch
    from paper_2609_04910_amd import gauss_sum as gs
    q, k, v, tau = wl.make_batch("batch_c32_f32", seed=0)
    tq, tk, tv = (torch.from_numpy(a).cuda() for a in (q, k, v))
    out = gs.gauss_sum_fwd_batched(tq, tk, tv, float(tau)).cpu().numpy()
    rows = wl.sample_rows(q.shape[1], 256, seed=3)
    for b in (0, 3):
        check("batch_c32_f32[%d]" % b, out[b], q[b], k[b], v[b], float(tau), rows=rows)
