"""GPU edge cases beyond the benchmark shapes: clouds translated far from
the origin (the expanded exponent tau q.k - tau/2 ||q||^2 - tau/2 ||k||^2
cancels there; Eq. 1 itself is translation invariant, Sec. 2 Remark 2),
and value / upstream-gradient magnitudes near 1e4.  Each case runs the
forward and all three gradients through the C ABI and is compared with the
fp64 oracle element by element."""
import sys

import numpy as np
import pytest

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


def _cloud(seed, M, N, D, C, offset, qk="f16", tau=None, grid=None):
    """N(0, I) clouds shifted by offset * 1 (both q and k), rounded to the
    point dtype; with `grid`, the unshifted draws are first rounded to
    multiples of `grid` (so that a shift by a multiple of 2 grid stays exact
    in fp16)."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((M, D)).astype(np.float32)
    y = rng.standard_normal((N, D)).astype(np.float32)
    if grid:
        x = np.clip(np.round(x / grid) * grid, -3.5, 3.5).astype(np.float32)
        y = np.clip(np.round(y / grid) * grid, -3.5, 3.5).astype(np.float32)
    x += np.float32(offset)
    y += np.float32(offset)
    if qk == "f16":
        q, qv, k, kv = x.astype(np.float16), x.astype(np.float16), y.astype(np.float16), y.astype(np.float16)
    else:
        q, qv = wl.bf16_round(x)
        k, kv = wl.bf16_round(y)
    v = rng.standard_normal((N, C)).astype(np.float32)
    g = rng.standard_normal((M, C)).astype(np.float32)
    t = np.float32(1.0 / D if tau is None else tau)
    return wl.Workload("offset%g" % offset, M, N, D, C, t, qk, q, k, v, g, ("fwd", "dq", "dk", "dv"), False,
                       qv, kv)


# (D, C, qk, offset): tau * max ||x||^2 stays within the documented domain
# (at most 2^13), up to offset 64 at D = 16 (tau ||x||^2 about 4100)
OFFSETS = [(16, 3, "f16", 8.0), (16, 3, "f16", 32.0), (16, 3, "f16", 64.0), (64, 1, "f16", 16.0),
           (64, 5, "f16", 48.0), (32, 4, "bf16", 24.0), (128, 16, "f16", 24.0), (256, 16, "f16", 12.0)]


@pytest.mark.parametrize("case", OFFSETS, ids=lambda c: "D%d_C%d_%s_off%g" % c)
def test_translated_clouds_match_oracle(case):
    import parity
    D, C, qk, off = case
    w = _cloud(11, 700, 900, D, C, off, qk)
    dom = float(w.tau) * max(float(np.max(np.sum(w.q_values.astype(np.float64) ** 2, 1))),
                             float(np.max(np.sum(w.k_values.astype(np.float64) ** 2, 1))))
    _say("case", case, "tau max||x||^2 = %.0f" % dom)
    assert dom <= 2.0 ** 13
    stats = parity.check_workload(w, passes=("fwd", "dq", "dk", "dv"))
    _say("  stats", stats)


def test_exact_translation_leaves_results_unchanged():
    """Points on a 2^-5 grid in [-3.5, 3.5] translated by 32 are exact in fp16
    (ulp 2^-5 on [32, 64), 2^-6 below), so both runs see the same sums;
    the translated run agrees with the centred one within twice the stated
    tolerance (each is within it of the same exact value)."""
    import parity
    a = _cloud(3, 600, 650, 16, 2, 0.0, grid=2.0 ** -5)
    b = _cloud(3, 600, 650, 16, 2, 32.0, grid=2.0 ** -5)
    assert np.array_equal(b.q_values.astype(np.float64) - 32.0, a.q_values.astype(np.float64))
    assert np.array_equal(b.k_values.astype(np.float64) - 32.0, a.k_values.astype(np.float64))
    ra = parity.run(a, ("fwd", "dq", "dk", "dv"))
    rb = parity.run(b, ("fwd", "dq", "dk", "dv"))
    for p in ("fwd", "dq", "dk", "dv"):
        rows = None
        ref, scale = parity.oracle_ref(a, p, rows=rows)
        err = np.abs(rb[p].astype(np.float64) - ra[p].astype(np.float64))
        assert np.all(err <= 2 * 2e-3 * scale + 1e-30), (p, float(np.max(err / scale)))
        _say(p, "max |translated - centred| / A = %.2e" % float(np.max(err / scale)))
    parity.check_workload(b, passes=("fwd", "dq", "dk", "dv"))


@pytest.mark.parametrize("vdt", ["f32", "f16"])
def test_value_and_gradient_magnitudes_near_1e4(vdt):
    import parity
    w = parity.random_workload(21, 500, 700, 24, 6, "f16", vdt, "f32")
    scale = np.float32(1.0e4)
    v = w.v.astype(np.float32) * scale
    w.v = v.astype(np.float16) if vdt == "f16" else v
    w.g = (w.g.astype(np.float32) * np.float32(0.7e4)).astype(np.float32)
    assert np.max(np.abs(w.v.astype(np.float32))) > 2e4
    stats = parity.check_workload(w, passes=("fwd", "dq", "dk", "dv"))
    _say("  stats", stats)


@pytest.mark.parametrize("tiny", [1e-5, 1e-7])
def test_bf16_points_with_a_tiny_coordinate(tiny):
    """bf16 points whose last coordinate is `tiny` times the others: the fp16
    copy that the gradient contraction reads is scaled so its largest
    magnitude lies in [2^14, 2^15), and the tiny coordinate keeps its 11
    bits.  Scaled to [1, 2), as before, it fell into fp16 subnormals, and the
    gradients' last coordinate (a sum of the small differences q - k there)
    was off by 4.8e-4 / 5.2e-4 of its scale (dq / dk) at 1e-5, 2.6e-2 /
    3.1e-2 at 1e-7; now 3.9e-5 / 5.0e-5 at either."""
    import parity
    rng = np.random.default_rng(11)
    M, N, D, C = 300, 500, 16, 4
    x = rng.standard_normal((M, D)).astype(np.float32)
    y = rng.standard_normal((N, D)).astype(np.float32)
    x[:, -1] *= np.float32(tiny)
    y[:, -1] *= np.float32(tiny)
    q, qv = wl.bf16_round(x)
    k, kv = wl.bf16_round(y)
    v = rng.standard_normal((N, C)).astype(np.float32)
    g = rng.standard_normal((M, C)).astype(np.float32)
    w = wl.Workload("tiny%g" % tiny, M, N, D, C, np.float32(1.0 / D), "bf16", q, k, v, g,
                    ("fwd", "dq", "dk", "dv"), False, qv, kv)
    _say("bf16 points, last coordinate scaled by", tiny)
    stats = parity.check_workload(w, passes=("fwd", "dq", "dk", "dv"))
    _say("  stats", stats)


def test_dominant_pair_with_an_equal_coordinate():
    """The limit of the per-element gradient scale: where the one pair that
    dominates a row of dq (a column of dk) has exactly equal coordinate d,
    that pair's term drops out of the element and of its scale, and the rest
    lies far below the pair's share of the two fp32 sums of the expanded
    form tau (sum P k_d - q_d sum P).  In this seeded case (fp16, spread 3,
    tau 3, kernel values near 1e-15) such elements exist: every other
    element meets the usual bound, and every element beyond it has that
    structure and an error within 2^-20 of the dominant pair's term
    tau Phi sum_c |g_c v_c| |q_d|."""
    import oracle
    import parity
    w = parity.random_workload(21, 150, 400, 8, 4, "f16", "f32", "f32", 3.0, 3.0)
    got = parity.run(w, ("dq", "dk"))
    qv = w.q_values.astype(np.float64)
    kv = w.k_values.astype(np.float64)
    d2 = ((qv[:, None, :] - kv[None, :, :]) ** 2).sum(-1)
    tol = parity.TOL["f16"]
    special = 0
    for pas in ("dq", "dk"):
        ref, scale = parity.oracle_ref(w, pas)
        err = np.abs(got[pas].astype(np.float64) - ref)
        for r, d in np.argwhere(err > tol * scale + 1e-30):
            m, n = (r, int(np.argmin(d2[r]))) if pas == "dq" else (int(np.argmin(d2[:, r])), r)
            assert qv[m, d] == kv[n, d], (pas, r, d)
            phi = oracle.fwd(w.q_values[m:m + 1], w.k_values[n:n + 1], np.ones((1, 1), np.float32),
                             float(w.tau))[0][0, 0]
            term = float(w.tau) * phi * np.abs(w.g[m].astype(np.float64) * w.v[n]).sum() * abs(qv[m, d])
            assert err[r, d] <= 2.0 ** -20 * term, (pas, r, d, err[r, d], term)
            _say("  %s[%d, %d]: err %.3e, scale %.3e, dominant term %.3e" % (pas, r, d, err[r, d], scale[r, d],
                                                                          term))
            special += 1
    assert special >= 1
