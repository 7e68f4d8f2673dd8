"""Seeded synthetic workloads shaped like the paper's experiments.

This module only draws random inputs and rounds them to storage precision.
It holds none of the Gauss-sum arithmetic, and both the GPU tests and the
CPU oracle consume exactly the arrays it returns (the oracle upcasts them to
fp64).  The paper evaluates on synthetic Gaussian point clouds only
(Sec. 4); no dataset is involved.

Five named workloads (sizes and recipes as listed in ``WORKLOADS``):

``dense_d16``   forward, M=N=4096, D=16, C=1, independent N(0,I) clouds in fp16,
                v ~ N(0,1) fp32, tau = 1/16.
``mmd_flow``    forward + dq, M=N=65536, D=64, C=1, q = k = x: 32768 source points
                N(0,I) followed by 32768 target points N(0.5*1, I), fp16; signed
                two-sample weights v = +1/N (source) / -1/N (target), exact in fp16;
                tau = 1/median squared pairwise distance over 4096 sampled points
                (all pairs i<j); upstream gradient g = v (fp32).
``svgd``        forward + dq, dk, dv, M=N=16384, D=128, C=128, q = k = x ~ N(0,I) fp16,
                v = -x + 0.1*eps (score-like) in fp16, tau = 1/128, g ~ N(0,1) fp32.
``mixture_d32`` forward, M=N=2^20, D=32, C=4, q and k drawn independently from the
                same 32-component isotropic mixture (centres ~ N(0,4I) drawn once,
                component std 0.3, equal weights), bf16; v ~ U[-1,1) fp32;
                tau in {0.1, 1, 10}.
``rect_d256``   forward + dq, dk, dv, M=2^17 queries, N=2^21 keys, D=256, C=16,
                independent unit-normalised N(0,I) vectors in fp16; v ~ N(0,1) fp16
                with exactly floor(0.1 N) zero rows (seeded permutation); tau = 4;
                g ~ N(0,1) fp32.

Random numbers come from ``numpy.random.default_rng(seed)`` (PCG64).  Draw
order: points (centres, labels, noise), then v, then g.  Reduced sizes
(``M``/``N`` overrides) follow the same recipe, for parity tests the oracle
can finish in seconds.
"""
from dataclasses import dataclass, field
from typing import Optional

import numpy as np

WORKLOADS = {
    "dense_d16": dict(M=4096, N=4096, D=16, C=1, passes=("fwd",)),
    "mmd_flow": dict(M=65536, N=65536, D=64, C=1, passes=("fwd", "dq")),
    "svgd": dict(M=16384, N=16384, D=128, C=128, passes=("fwd", "dq", "dk", "dv")),
    "mixture_d32": dict(M=1 << 20, N=1 << 20, D=32, C=4, passes=("fwd",)),
    "rect_d256": dict(M=1 << 17, N=1 << 21, D=256, C=16, passes=("fwd", "dq", "dk", "dv")),
}
ORDER = ("dense_d16", "mmd_flow", "svgd", "mixture_d32", "rect_d256")
MIXTURE_TAUS = (0.1, 1.0, 10.0)


def bf16_round(x: np.ndarray):
    """Round float32 values to bfloat16 with round-to-nearest-even.

    Returns ``(bits, values)``: the uint16 bit patterns and the same numbers as
    float32.  NaN is kept quiet; infinities pass through.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16).astype(np.uint32)
    nan = np.isnan(x)
    r[nan] = (u[nan] >> 16).astype(np.uint32) | 0x40
    bits = r.astype(np.uint16)
    vals = (bits.astype(np.uint32) << 16).view(np.float32)
    return bits, vals


@dataclass
class Workload:
    """One synthetic problem instance.

    ``q``, ``k``: storage arrays (float16, or uint16 bf16 bits when
    ``qk_dtype == 'bf16'``); ``q_values``/``k_values`` the same numbers as
    float16/float32 arrays for the oracle.  ``v`` and ``g`` are stored in ``v_dtype``/``g_dtype``
    (float16 or float32).  ``same_points`` marks q and k as the same array.
    """
    name: str
    M: int
    N: int
    D: int
    C: int
    tau: np.float32
    qk_dtype: str
    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    g: Optional[np.ndarray]
    passes: tuple
    same_points: bool
    q_values: np.ndarray = field(repr=False, default=None)
    k_values: np.ndarray = field(repr=False, default=None)

    @property
    def pairs(self) -> int:
        return self.M * self.N


def _store_points(x32: np.ndarray, dtype: str):
    if dtype == "f16":
        h = x32.astype(np.float16)
        return h, h
    bits, vals = bf16_round(x32)
    return bits, vals


def _median_tau(x16: np.ndarray, rng: np.random.Generator, samples: int = 4096) -> np.float32:
    """tau = 1 / median of the squared pairwise distances (all pairs i<j) of
    ``samples`` distinct points drawn without replacement (median heuristic)."""
    n = x16.shape[0]
    s = min(samples, n)
    idx = rng.choice(n, size=s, replace=False)
    X = x16[idx].astype(np.float64)
    sq = np.einsum("ij,ij->i", X, X)
    d2 = sq[:, None] + sq[None, :] - 2.0 * (X @ X.T)
    iu = np.triu_indices(s, k=1)
    med = float(np.median(d2[iu]))
    return np.float32(1.0 / med)


def make(name: str, seed: int = 0, M: Optional[int] = None, N: Optional[int] = None,
         tau: Optional[float] = None) -> Workload:
    """Build workload ``name`` (see module doc) with optional reduced sizes."""
    spec = WORKLOADS[name]
    D, C = spec["D"], spec["C"]
    M = spec["M"] if M is None else int(M)
    N = spec["N"] if N is None else int(N)
    rng = np.random.default_rng(seed)
    f32 = np.float32

    if name == "dense_d16":
        q, qv = _store_points(rng.standard_normal((M, D), dtype=f32), "f16")
        k, kv = _store_points(rng.standard_normal((N, D), dtype=f32), "f16")
        v = rng.standard_normal((N, C), dtype=f32)
        return Workload(name, M, N, D, C, f32(1.0 / D if tau is None else tau), "f16", q, k, v,
                        None, spec["passes"], False, qv, kv)

    if name == "mmd_flow":
        if M != N:
            raise ValueError("mmd_flow uses q = k, so M must equal N")
        half = N // 2
        x32 = rng.standard_normal((N, D), dtype=f32)
        x32[half:] += f32(0.5)
        x, xv = _store_points(x32, "f16")
        w = np.float16(1.0 / N)
        v = np.empty((N, C), dtype=np.float16)
        v[:half] = w
        v[half:] = -w
        t = _median_tau(x, rng) if tau is None else f32(tau)
        g = v.astype(f32)
        return Workload(name, M, N, D, C, t, "f16", x, x, v, g, spec["passes"], True, xv, xv)

    if name == "svgd":
        if M != N:
            raise ValueError("svgd uses q = k, so M must equal N")
        x, xv = _store_points(rng.standard_normal((N, D), dtype=f32), "f16")
        eps = rng.standard_normal((N, C), dtype=f32)
        v = (-x.astype(f32) + f32(0.1) * eps).astype(np.float16)
        g = rng.standard_normal((M, C), dtype=f32)
        return Workload(name, M, N, D, C, f32(1.0 / D if tau is None else tau), "f16", x, x, v, g,
                        spec["passes"], True, xv, xv)

    if name == "mixture_d32":
        K = 32
        centres = f32(2.0) * rng.standard_normal((K, D), dtype=f32)
        lq = rng.integers(0, K, size=M)
        lk = rng.integers(0, K, size=N)
        q32 = centres[lq] + f32(0.3) * rng.standard_normal((M, D), dtype=f32)
        k32 = centres[lk] + f32(0.3) * rng.standard_normal((N, D), dtype=f32)
        q, qv = _store_points(q32, "bf16")
        k, kv = _store_points(k32, "bf16")
        v = rng.uniform(-1.0, 1.0, size=(N, C)).astype(f32)
        t = f32(1.0 if tau is None else tau)
        return Workload(name, M, N, D, C, t, "bf16", q, k, v, None, spec["passes"], False, qv, kv)

    if name == "rect_d256":
        def unit(n):
            # N(0, I) rows divided by their norm (computed in fp64), stored
            # fp16; drawn in blocks of rows into reused buffers (the same
            # stream of draws as one call for all n rows)
            blk_rows = 4096
            h = np.empty((n, D), dtype=np.float16)
            x = np.empty((blk_rows, D), dtype=f32)
            buf = np.empty((blk_rows, D), dtype=np.float64)
            for a in range(0, n, blk_rows):
                m = min(blk_rows, n - a)
                rng.standard_normal(out=x[:m], dtype=f32)
                blk = buf[:m]
                blk[...] = x[:m]
                blk /= np.sqrt(np.einsum("ij,ij->i", blk, blk))[:, None]
                h[a:a + m] = blk
            return h
        q = qv = unit(M)
        k = kv = unit(N)
        v = rng.standard_normal((N, C), dtype=f32).astype(np.float16)
        zero = rng.permutation(N)[: N // 10]
        v[zero] = 0
        g = rng.standard_normal((M, C), dtype=f32)
        return Workload(name, M, N, D, C, f32(4.0 if tau is None else tau), "f16", q, k, v, g,
                        spec["passes"], False, qv, kv)

    raise KeyError(name)


BATCHED = {
    # Sec. 4 benchmark layout: B independent standard Gaussian clouds scaled by
    # D^(-1/2), M = N, tau = 1, fp16 (the D sweep uses B = 64, N = 16384, C = 1)
    "batch_d32": dict(B=64, M=16384, N=16384, D=32, C=1),
    # the same layout in single precision (App. A.2, the D sweep in fp32)
    "batch_d32_f32": dict(B=64, M=16384, N=16384, D=32, C=1, qk="f32"),
    # the N sweep with several channels (B = 4, D = C = 32), at N = 16384
    "batch_c32": dict(B=4, M=16384, N=16384, D=32, C=32),
    "batch_c32_f32": dict(B=4, M=16384, N=16384, D=32, C=32, qk="f32"),
    # the N sweep of the forward-plus-backward benchmark (B = 4, D = 32,
    # C = 1, fp16) at N = 65536: s and the gradients with respect to q, k, v
    "batch_grad_d32": dict(B=4, M=65536, N=65536, D=32, C=1, grad=True),
}


def make_batch(name: str, seed: int = 0, B: Optional[int] = None, M: Optional[int] = None):
    """Batched workload ``name``: (q, k, v, tau) with q, k of shape B x M x D
    (fp16, or fp32 where the entry says qk="f32"; N(0, I / D)) and v of shape
    B x N x C (fp32, N(0, 1)); draws in the order points (q then k, problem by
    problem), then values."""
    cfg = dict(BATCHED[name])
    if B is not None:
        cfg["B"] = B
    if M is not None:
        cfg["M"] = cfg["N"] = M
    B_, M_, N_, D_, C_ = cfg["B"], cfg["M"], cfg["N"], cfg["D"], cfg["C"]
    pt = np.float32 if cfg.get("qk") == "f32" else np.float16
    rng = np.random.default_rng(seed)
    s = np.float32(1.0 / np.sqrt(D_))
    q = np.empty((B_, M_, D_), pt)
    k = np.empty((B_, N_, D_), pt)
    for b in range(B_):
        q[b] = (rng.standard_normal((M_, D_), dtype=np.float32) * s).astype(pt)
        k[b] = (rng.standard_normal((N_, D_), dtype=np.float32) * s).astype(pt)
    v = rng.standard_normal((B_, N_, C_), dtype=np.float32)
    return q, k, v, np.float32(1.0)


def batch_dout(name: str, seed: int = 0, M: Optional[int] = None) -> np.ndarray:
    """Upstream gradient dout ~ N(0, 1) fp32 (B x M x C) of a batched
    workload's backward pass, from its own generator (seed + 1), so the
    points and values of make_batch stay the same draws."""
    cfg = BATCHED[name]
    rng = np.random.default_rng(seed + 1)
    return rng.standard_normal((cfg["B"], M or cfg["M"], cfg["C"]), dtype=np.float32)


def sample_rows(n_total: int, count: int, seed: int = 1, tile: int = 256) -> np.ndarray:
    """Seeded sample of ``count`` distinct row indices plus tile-boundary rows
    (0, 63, 64, 127, 128, 255 modulo ``tile`` near the start and end) and the
    last row; sorted, unique."""
    rng = np.random.default_rng(seed)
    c = min(count, n_total)
    base = rng.choice(n_total, size=c, replace=False)
    extra = []
    for start in (0, max(0, (n_total // tile - 1) * tile)):
        for off in (0, 63, 64, 127, 128, 255):
            if start + off < n_total:
                extra.append(start + off)
    extra.append(n_total - 1)
    return np.unique(np.concatenate([base, np.array(extra, dtype=np.int64)]))
