"""GPU parity of gauss_sum_svgd (Sec. 3: the SVGD direction, whose kernel
part has the form of the query gradient) against the fp64 oracle:
phi[m] = sum_n Phi(x_m, x_n) score_n + tau sum_n Phi(x_m, x_n) (x_m - x_n),
i.e. the forward sum with values score minus the query gradient with unit
weights and unit upstream gradient.  Tolerance per element: tol times the sum
of the two oracle scales (sum_n Phi |score_nd| and tau sum_n Phi |x_nd - x_md|).
A small case is also checked against the definition written out in numpy."""
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


def particles(seed, N, D, qk, sdt):
    """x ~ N(0, I); score = -x + 0.1 eps (the score of N(0, I) plus noise)."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((N, D)).astype(np.float32)
    if qk == "f16":
        xs = x.astype(np.float16)
        xv = xs
    else:
        xs, xv = wl.bf16_round(x)
    score = (-xv.astype(np.float32) + 0.1 * rng.standard_normal((N, D))).astype(np.float32)
    if sdt == "f16":
        score = score.astype(np.float16)
    return xs, xv, score


def reference(xv, score, tau, rows=None):
    th = parity.oracle_threads()
    ones = np.ones((xv.shape[0], 1), np.float32)
    s, a = oracle.fwd(xv, xv, score, tau, rows=rows, threads=th)
    dq, aq = oracle.dq(xv, xv, ones, ones, tau, rows=rows, threads=th)
    return s - dq, a + aq


def run(xs, score, tau):
    import torch
    from paper_2609_04910_amd import gauss_sum as gs
    phi = gs.gauss_sum_svgd(parity.to_torch(xs), parity.to_torch(score), float(tau))
    torch.cuda.synchronize()
    return phi.cpu().numpy()


@pytest.mark.parametrize("N,D,qk,sdt,tau", [
    (1, 4, "f16", "f32", 0.5), (300, 64, "f16", "f32", 1.0 / 64), (777, 128, "f16", "f16", 1.0 / 128),
    (1000, 32, "bf16", "f32", 1.0 / 32), (517, 17, "f16", "f32", 0.3),
    # the D > 128 instance (one query tile per wave, 16 tiles of score values)
    # and bf16 points beyond D = 32
    (400, 256, "f16", "f32", 1.0 / 256), (350, 200, "bf16", "f16", 1.0 / 200),
    (640, 100, "bf16", "f32", 1.0 / 100), (1000, 129, "f16", "f16", 1.0 / 129)])
def test_svgd_matches_oracle(N, D, qk, sdt, tau):
    xs, xv, score = particles(N + D, N, D, qk, sdt)
    got = run(xs, score, tau)
    ref, scale = reference(xv, score, tau)
    _say("svgd", N, D, qk, parity.compare("svgd", got, ref, scale, parity.TOL[qk]))


def test_svgd_small_case_against_the_definition():
    N, D, tau = 40, 3, 0.7
    xs, xv, score = particles(3, N, D, "f16", "f32")
    got = run(xs, score, tau)
    x = xv.astype(np.float64)
    diff = x[:, None, :] - x[None, :, :]                       # x_m - x_n
    phi_k = np.exp(-0.5 * float(np.float32(tau)) * (diff ** 2).sum(-1))
    ref = phi_k @ score.astype(np.float64) + float(np.float32(tau)) * (phi_k[:, :, None] * diff).sum(1)
    scale = phi_k @ np.abs(score.astype(np.float64)) + float(np.float32(tau)) * (phi_k[:, :, None] * np.abs(diff)).sum(1)
    _say("svgd definition", parity.compare("svgd definition", got, ref, scale, parity.TOL["f16"]))


def test_svgd_workload_full_size_sampled_rows():
    """The svgd workload's points and score-like values (N = 16384, D = 128)."""
    w = wl.make("svgd", seed=0)
    got = run(w.q, w.v, w.tau)
    rows = wl.sample_rows(w.M, 256, seed=4)
    ref, scale = reference(w.q_values, w.v, w.tau, rows=rows)
    _say("svgd full size", parity.compare("svgd full", got[rows], ref, scale, parity.TOL["f16"]))
