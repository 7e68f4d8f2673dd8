"""Pins for the fp64 oracle: checks against facts fixed by the paper and by
mathematics, none of which re-types the oracle's own double loop.

Each ``pin_*`` takes an oracle object (``fwd/dq/dk/dv`` methods, see
``oracle.Oracle``) and raises AssertionError on failure.  ``test_oracle.py``
runs every pin against the real oracle; ``test_oracle_mutants.py`` runs them
against deliberately broken copies of the oracle and requires each copy to
fail at least one pin.

Independent routes used here:
  * the kernel matrix from ``scipy.spatial.distance.cdist`` in the expanded
    (Gram) form, with numpy long double, times a library matmul;
  * the paper's two attention routes in fp64: prescale (Alg. 1, built on the
    un-normalisation identity Eq. 3 and the factorisation Eq. 4) and reweight
    (Alg. 2, identity Eq. 5) with the bounds of Prop. 1;
  * closed forms (one key; a point against itself; tau -> 0; well separated
    points; a dyadic lattice where tau = 2 ln 2 makes every kernel value an
    exact power of two, summed in exact rational arithmetic);
  * invariants (joint translation, linearity in v, permutation, the adjoint
    relation, MMD^2 >= 0 from Sec. 3);
  * central finite differences for all gradients, the query-gradient formula
    of Sec. 3 evaluated through the dense kernel matrix, and the identities
    that follow from Eq. 1 being symmetric in (q, k) and linear in v.
"""
import math
from fractions import Fraction

import numpy as np
from scipy.spatial.distance import cdist
from scipy.special import logsumexp


def _rng(seed):
    return np.random.default_rng(seed)


def _close(a, b, rtol, atol=0.0, what=""):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    assert a.shape == b.shape, "%s: shape %s vs %s" % (what, a.shape, b.shape)
    err = np.abs(a - b)
    bound = rtol * np.maximum(np.abs(b), np.abs(a)) + atol
    bad = err > bound
    assert not bad.any(), "%s: max err %.3e (bound %.3e) at %s" % (
        what, err.max(), bound.flat[int(np.argmax(err - bound))], np.argwhere(bad)[0])


def _kernel_matrix(q, k, tau):
    """exp(-tau/2 * d2) with d2 from scipy's cdist (sqeuclidean), in long double."""
    d2 = cdist(np.asarray(q, np.float64), np.asarray(k, np.float64), "sqeuclidean")
    return np.exp(np.longdouble(-0.5 * tau) * d2.astype(np.longdouble))


def _problem(seed, M, N, D, C, spread=1.0):
    r = _rng(seed)
    return (spread * r.standard_normal((M, D)), spread * r.standard_normal((N, D)),
            r.standard_normal((N, C)), r.standard_normal((M, C)))


# ---------------------------------------------------------------- forward

def pin_library_kernel_matrix(orc):
    """Eq. 1 as a long-double kernel matrix (cdist) times v (matmul)."""
    for seed, (M, N, D, C, tau) in enumerate([(5, 7, 3, 2, 0.7), (9, 4, 1, 1, 2.5),
                                              (3, 11, 8, 3, 0.05), (6, 6, 5, 4, 1.0)]):
        q, k, v, _ = _problem(seed, M, N, D, C)
        Kmat = _kernel_matrix(q, k, tau)
        ref = (Kmat @ v.astype(np.longdouble)).astype(np.float64)
        ref_abs = (Kmat @ np.abs(v).astype(np.longdouble)).astype(np.float64)
        s, a = orc.fwd(q, k, v, tau)
        _close(s, ref, 1e-12, 1e-300, "fwd vs kernel matrix")
        _close(a, ref_abs, 1e-12, 1e-300, "abs scale vs kernel matrix")


def _attention(qt, kt, vt, tau):
    """Softmax attention Att_tau and lse_tau of Eq. 2, stable fp64."""
    logits = tau * (qt @ kt.T)
    lse = logsumexp(logits, axis=1)
    att = np.exp(logits - lse[:, None]) @ vt
    return att, lse


def pin_prescale_alg1(orc):
    """Alg. 1: s = Att(q,k,v~) exp(lse) exp(-tau/2||q||^2), v~ = v exp(-tau/2||k||^2)."""
    q, k, v, _ = _problem(11, 8, 13, 4, 3, spread=0.8)
    tau = 1.3
    vt = v * np.exp(-0.5 * tau * np.sum(k * k, axis=1))[:, None]
    att, lse = _attention(q, k, vt, tau)
    s_ref = att * np.exp(lse)[:, None] * np.exp(-0.5 * tau * np.sum(q * q, axis=1))[:, None]
    s, _ = orc.fwd(q, k, v, tau)
    _close(s, s_ref, 1e-11, 1e-300, "prescale route (Alg. 1)")


def pin_reweight_alg2(orc):
    """Alg. 2 with kappa = sqrt(N+1): s = kappa*alpha/beta, and Prop. 1's bounds."""
    M, N, D, C = 7, 10, 3, 2
    q, k, v, _ = _problem(12, M, N, D, C, spread=0.9)
    tau = 0.8
    kappa = math.sqrt(N + 1)
    qt = np.concatenate([q, np.ones((M, 1)), 0.5 * np.sum(q * q, axis=1, keepdims=True)], axis=1)
    kt = np.concatenate([k, -0.5 * np.sum(k * k, axis=1, keepdims=True), np.zeros((N, 1))], axis=1)
    k0 = np.zeros((1, D + 2))
    k0[0, D + 1] = 1.0
    vt = np.concatenate([v, np.zeros((N, 1))], axis=1)
    v0 = np.zeros((1, C + 1))
    v0[0, C] = kappa
    att, _ = _attention(qt, np.concatenate([k0, kt]), np.concatenate([v0, vt]), tau)
    alpha, beta = att[:, :C], att[:, C]
    s, _ = orc.fwd(q, k, v, tau)
    _close(s, kappa * alpha / beta[:, None], 1e-11, 1e-300, "reweight route (Alg. 2)")
    # Prop. 1: kappa/(N+1) <= beta <= kappa, beta = kappa/(1 + sum_n Phi),
    # ||alpha_m||_inf <= max_n ||v_n||_inf.  sum_n Phi is the oracle with v = 1.
    sum_phi, _ = orc.fwd(q, k, np.ones((N, 1)), tau)
    assert np.all(beta >= kappa / (N + 1) * (1 - 1e-12)) and np.all(beta <= kappa * (1 + 1e-12))
    _close(beta, kappa / (1.0 + sum_phi[:, 0]), 1e-11, 0.0, "Prop. 1 beta identity")
    assert np.max(np.abs(alpha)) <= np.max(np.abs(v)) * (1 + 1e-12)


def pin_single_key(orc):
    """N = 1: s = exp(-tau/2 ||q - k||^2) v with a hand-computed distance."""
    q = np.array([[0.0, 0.0], [1.0, 1.0], [3.0, 4.0]])
    k = np.array([[3.0, 4.0]])
    v = np.array([[2.0, -0.5]])
    tau = 0.25
    d2 = np.array([25.0, 13.0, 0.0])
    ref = np.exp(-tau / 2 * d2)[:, None] * v
    s, a = orc.fwd(q, k, v, tau)
    _close(s, ref, 1e-15, 0.0, "single key")
    _close(a, np.abs(ref), 1e-15, 0.0, "single key abs")


def pin_self_point(orc):
    """q = k, one point: Phi = 1, so s = v exactly (any tau)."""
    x = np.array([[0.3, -1.7, 2.2, 5.0]])
    v = np.array([[1.5, -2.25, 0.0]])
    for tau in (1e-3, 1.0, 1e6):
        s, _ = orc.fwd(x, x, v, tau)
        assert np.array_equal(s, v), (tau, s)


def pin_tau_to_zero(orc):
    """tau -> 0: every Phi -> 1, so s_m = sum_n v_n for every m."""
    q, k, v, _ = _problem(13, 4, 9, 3, 2)
    s, _ = orc.fwd(q, k, v, 1e-300)
    ref = np.broadcast_to(np.sum(v, axis=0), s.shape)
    _close(s, ref, 1e-14, 1e-14, "tau -> 0")


def pin_separated(orc):
    """Far-apart lattice points with large tau: s_m = sum of v_n with k_n == q_m."""
    grid = 10.0 * np.array([[i, j] for i in range(3) for j in range(3)], dtype=np.float64)
    r = _rng(14)
    kidx = r.integers(0, 9, size=20)
    k = grid[kidx]
    q = grid[[0, 4, 8, 2]]
    v = r.standard_normal((20, 2))
    s, _ = orc.fwd(q, k, v, 5.0)
    ref = np.array([v[kidx == i].sum(axis=0) for i in (0, 4, 8, 2)])
    _close(s, ref, 1e-14, 1e-100, "separated points")


def pin_dyadic_lattice(orc):
    """Integer points, tau = 2 ln 2: Phi = 2^(-d2) exactly, summed as fractions."""
    r = _rng(15)
    q = r.integers(-2, 3, size=(6, 3)).astype(np.float64)
    k = r.integers(-2, 3, size=(9, 3)).astype(np.float64)
    v = r.integers(-8, 9, size=(9, 2)).astype(np.float64) / 4.0
    tau = 2.0 * math.log(2.0)
    s, _ = orc.fwd(q, k, v, tau)
    ref = np.zeros((6, 2))
    for m in range(6):
        for c in range(2):
            tot = Fraction(0)
            for n in range(9):
                d2 = int(sum((int(q[m, d]) - int(k[n, d])) ** 2 for d in range(3)))
                tot += Fraction(1, 2 ** d2) * Fraction(v[n, c])
            ref[m, c] = float(tot)
    _close(s, ref, 1e-13, 1e-15, "dyadic lattice")


def pin_translation(orc):
    """Joint translation of q and k leaves Eq. 1 unchanged."""
    q, k, v, _ = _problem(16, 6, 8, 4, 2)
    a = np.array([0.75, -2.0, 1.5, 3.0])
    s0, _ = orc.fwd(q, k, v, 0.9)
    s1, _ = orc.fwd(q + a, k + a, v, 0.9)
    _close(s1, s0, 1e-11, 1e-14, "translation")


def pin_linearity(orc):
    """s(q, k, alpha v + beta u) = alpha s(v) + beta s(u)."""
    q, k, v, _ = _problem(17, 5, 7, 3, 2)
    u = _rng(18).standard_normal(v.shape)
    s = orc.fwd(q, k, 1.5 * v - 0.25 * u, 0.6)[0]
    ref = 1.5 * orc.fwd(q, k, v, 0.6)[0] - 0.25 * orc.fwd(q, k, u, 0.6)[0]
    _close(s, ref, 1e-12, 1e-13, "linearity in v")


def pin_permutation(orc):
    """Permuting keys (with v) changes nothing; permuting queries permutes rows."""
    q, k, v, _ = _problem(19, 6, 9, 3, 2)
    pk = _rng(20).permutation(9)
    pq = _rng(21).permutation(6)
    s0, _ = orc.fwd(q, k, v, 0.7)
    s1, _ = orc.fwd(q[pq], k[pk], v[pk], 0.7)
    _close(s1, s0[pq], 1e-13, 1e-15, "permutation")


def pin_adjoint(orc):
    """<u, s(q,k,v)> = <v, s(k,q,u)> (the kernel matrix is transposed)."""
    q, k, v, u = _problem(22, 7, 5, 3, 2)
    lhs = np.sum(u * orc.fwd(q, k, v, 1.1)[0])
    rhs = np.sum(v * orc.fwd(k, q, u, 1.1)[0])
    assert abs(lhs - rhs) <= 1e-12 * (abs(lhs) + abs(rhs) + 1e-300), (lhs, rhs)


def pin_rows_subset(orc):
    """Row-subset mode returns exactly the selected rows of the full result."""
    q, k, v, g = _problem(23, 9, 6, 3, 2)
    rows = np.array([8, 0, 3, 3])
    s_all, a_all = orc.fwd(q, k, v, 0.5)
    s, a = orc.fwd(q, k, v, 0.5, rows=rows)
    assert np.array_equal(s, s_all[rows]) and np.array_equal(a, a_all[rows])
    d_all, _ = orc.dk(q, k, v, g, 0.5)
    d, _ = orc.dk(q, k, v, g, 0.5, rows=[5, 1])
    assert np.array_equal(d, d_all[[5, 1]])


def pin_threads_bitwise(orc):
    """Each row is summed by one thread in index order: thread count is invisible."""
    q, k, v, g = _problem(24, 37, 20, 4, 3)
    for fn in (lambda t: orc.fwd(q, k, v, 0.4, threads=t), lambda t: orc.dq(q, k, v, g, 0.4, threads=t),
               lambda t: orc.dk(q, k, v, g, 0.4, threads=t), lambda t: orc.dv(q, k, v, g, 0.4, threads=t)):
        a1, b1 = fn(1)
        a7, b7 = fn(7)
        assert np.array_equal(a1, a7) and np.array_equal(b1, b7)


def pin_mmd_nonnegative(orc):
    """Sec. 3: MMD^2 = v^T s(x, x, v) >= 0 for signed v; identical measures give 0."""
    r = _rng(25)
    for trial in range(5):
        x = r.standard_normal((12, 2))
        v = r.standard_normal((12, 1))
        val = float(np.sum(v * orc.fwd(x, x, v, 0.5 + trial)[0]))
        assert val >= -1e-13, val
    x = r.standard_normal((6, 3))
    xx = np.concatenate([x, x])
    w = np.concatenate([np.full((6, 1), 1 / 6), np.full((6, 1), -1 / 6)])
    assert abs(float(np.sum(w * orc.fwd(xx, xx, w, 1.0)[0]))) < 1e-15


# -------------------------------------------------------------- gradients

def _loss(orc, q, k, v, g, tau):
    return float(np.sum(g * orc.fwd(q, k, v, tau)[0]))


def _fd(orc, f, x, h):
    grad = np.zeros_like(x)
    for idx in np.ndindex(*x.shape):
        xp = x.copy()
        xm = x.copy()
        xp[idx] += h
        xm[idx] -= h
        grad[idx] = (f(xp) - f(xm)) / (2 * h)
    return grad


def pin_dq_finite_difference(orc):
    q, k, v, g = _problem(26, 4, 6, 3, 2)
    tau = 0.7
    fd = _fd(orc, lambda x: _loss(orc, x, k, v, g, tau), q, 1e-5)
    _close(orc.dq(q, k, v, g, tau)[0], fd, 1e-6, 1e-9, "dq vs finite differences")


def pin_dk_finite_difference(orc):
    q, k, v, g = _problem(27, 5, 4, 3, 2)
    tau = 0.9
    fd = _fd(orc, lambda x: _loss(orc, q, x, v, g, tau), k, 1e-5)
    _close(orc.dk(q, k, v, g, tau)[0], fd, 1e-6, 1e-9, "dk vs finite differences")


def pin_dv_finite_difference(orc):
    q, k, v, g = _problem(28, 5, 4, 3, 3)
    tau = 0.6
    fd = _fd(orc, lambda x: _loss(orc, q, k, x, g, tau), v, 1e-3)
    _close(orc.dv(q, k, v, g, tau)[0], fd, 1e-9, 1e-12, "dv vs finite differences")


def pin_query_gradient_formula(orc):
    """Sec. 3: grad_{q_m} s_m = tau (sum Phi v_n k_n - q_m sum Phi v_n) for C = 1,
    evaluated through the dense long-double kernel matrix; with g = 1 the
    oracle's dq is exactly this gradient."""
    q, k, v, _ = _problem(29, 6, 9, 4, 1)
    tau = 1.2
    Kmat = _kernel_matrix(q, k, tau)
    vk = v.astype(np.longdouble) * k.astype(np.longdouble)
    ref = tau * ((Kmat @ vk) - q * (Kmat @ v.astype(np.longdouble)))
    _close(orc.dq(q, k, v, np.ones((6, 1)), tau)[0], ref.astype(np.float64), 1e-11, 1e-14,
           "query gradient formula")


def pin_gradient_scales(orc):
    """The absolute scales equal the sums of |terms| built from the dense matrix;
    the q and k gradients are double sums over (n, c) of tau Phi g_c v_c (k - q)."""
    q, k, v, g = _problem(30, 5, 7, 3, 2)
    tau = 0.8
    Kmat = _kernel_matrix(q, k, tau).astype(np.float64)
    W = np.abs(g) @ np.abs(v).T                    # sum_c |g_mc v_nc|
    diff = k[None, :, :] - q[:, None, :]           # k_n - q_m
    aq = tau * np.einsum("mn,mnd->md", Kmat * W, np.abs(diff))
    ak = tau * np.einsum("mn,mnd->nd", Kmat * W, np.abs(diff))
    av = Kmat.T @ np.abs(g)
    _close(orc.dq(q, k, v, g, tau)[1], aq, 1e-12, 1e-300, "dq scale")
    _close(orc.dk(q, k, v, g, tau)[1], ak, 1e-12, 1e-300, "dk scale")
    _close(orc.dv(q, k, v, g, tau)[1], av, 1e-12, 1e-300, "dv scale")


def pin_net_scales(orc):
    """The net scales tau sum Phi |sum_c g_c v_c| |k - q| of the q and k
    gradients: from the dense kernel matrix; equal to the absolute scales for
    one channel; zero where every w_mn vanishes although its channel terms do
    not (g_m = (a, a), v_n = (b, -b)), unlike the absolute scale; never above the absolute
    scale; and the gradients themselves unchanged."""
    q, k, v, g = _problem(31, 6, 8, 3, 3)
    tau = 0.7
    Kmat = _kernel_matrix(q, k, tau).astype(np.float64)
    Wn = np.abs(g @ v.T)                           # |sum_c g_mc v_nc|
    diff = k[None, :, :] - q[:, None, :]
    nq = tau * np.einsum("mn,mnd->md", Kmat * Wn, np.abs(diff))
    nk = tau * np.einsum("mn,mnd->nd", Kmat * Wn, np.abs(diff))
    dq, aq, netq = orc.dq_scales(q, k, v, g, tau)
    dk, ak, netk = orc.dk_scales(q, k, v, g, tau)
    _close(netq, nq, 1e-12, 1e-300, "dq net scale")
    _close(netk, nk, 1e-12, 1e-300, "dk net scale")
    assert np.all(netq <= aq * (1 + 1e-12)) and np.all(netk <= ak * (1 + 1e-12))
    _close(dq, orc.dq(q, k, v, g, tau)[0], 0.0, 0.0, "dq value")
    _close(dk, orc.dk(q, k, v, g, tau)[0], 0.0, 0.0, "dk value")
    # one channel: |g v| = |g| |v|, the two scales agree
    q1, k1, v1, g1 = _problem(32, 5, 7, 2, 1)
    _, a1, n1 = orc.dq_scales(q1, k1, v1, g1, 0.9)
    _close(n1, a1, 1e-14, 0.0, "one-channel dq scales")
    _, a1k, n1k = orc.dk_scales(q1, k1, v1, g1, 0.9)
    _close(n1k, a1k, 1e-14, 0.0, "one-channel dk scales")
    # w = a_m b_n - a_m b_n = 0 for every pair while each channel's term is not
    a = _rng(33).standard_normal((6, 1))
    b = _rng(34).standard_normal((8, 1))
    g2 = np.hstack([a, a])
    v2 = np.hstack([b, -b])
    d2, a2, n2 = orc.dq_scales(q, k, v2, g2, tau)
    assert np.all(n2 == 0.0) and np.all(d2 == 0.0) and np.all(a2 > 0.0)
    d2k, a2k, n2k = orc.dk_scales(q, k, v2, g2, tau)
    assert np.all(n2k == 0.0) and np.all(d2k == 0.0) and np.all(a2k > 0.0)


def pin_swap_identities(orc):
    """Eq. 1 is symmetric in (q, k) and linear in v, so
    dv(q,k,v,g) = s(k,q,g) and dk(q,k,v,g) = dq(k,q,g,v)."""
    q, k, v, g = _problem(31, 6, 8, 3, 2)
    tau = 0.75
    _close(orc.dv(q, k, v, g, tau)[0], orc.fwd(k, q, g, tau)[0], 1e-13, 1e-15, "dv = fwd swapped")
    _close(orc.dk(q, k, v, g, tau)[0], orc.dq(k, q, g, v, tau)[0], 1e-13, 1e-15, "dk = dq swapped")


def pin_gradient_translation(orc):
    """Translation invariance: sum_m dq_m + sum_n dk_n = 0."""
    q, k, v, g = _problem(32, 7, 9, 3, 2)
    tot = orc.dq(q, k, v, g, 0.5)[0].sum(axis=0) + orc.dk(q, k, v, g, 0.5)[0].sum(axis=0)
    scale = orc.dq(q, k, v, g, 0.5)[1].sum()
    assert np.all(np.abs(tot) <= 1e-12 * scale), tot


def pin_gradient_degenerate(orc):
    """tau -> 0 gives dq, dk -> 0 (proportional to tau); a point against
    itself has zero query gradient."""
    q, k, v, g = _problem(33, 4, 5, 2, 2)
    tiny = 1e-200
    dq0 = orc.dq(q, k, v, g, tiny)[0]
    assert np.all(np.abs(dq0) <= 1e-195), dq0
    x = np.array([[0.5, -1.0, 2.0]])
    assert np.array_equal(orc.dq(x, x, np.ones((1, 2)), np.ones((1, 2)), 3.0)[0], np.zeros((1, 3)))


def pin_empty_sum(orc):
    """N = 0 is the empty sum; M = 0 selects nothing."""
    s, a = orc.fwd(np.zeros((3, 2)), np.zeros((0, 2)), np.zeros((0, 1)), 1.0)
    assert np.array_equal(s, np.zeros((3, 1))) and np.array_equal(a, np.zeros((3, 1)))
    s, _ = orc.fwd(np.zeros((0, 2)), np.ones((4, 2)), np.ones((4, 1)), 1.0)
    assert s.shape == (0, 1)


ALL_PINS = [v for k_, v in sorted(globals().items()) if k_.startswith("pin_")]
