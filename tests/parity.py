"""Helpers shared by the GPU parity tests: move a workload to the GPU, run the
library through the C ABI binding, and compare with the fp64 oracle.

Pass rule (per element): |gpu - oracle| <= tol * A + 1e-30, where A is the
oracle's sum of absolute terms (sum_n Phi |v_n| for the forward pass and the
analogous sums for the gradients) and tol = 2e-3 for fp16 points, 5e-3 for
bf16 points.
"""
import os

import numpy as np

import oracle
from paper_2609_04910_amd import gauss_sum as gs
from paper_2609_04910_amd import workloads as wl

TOL = {"f16": 2e-3, "bf16": 5e-3}


def oracle_threads():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, int(os.environ.get("GS_ORACLE_THREADS", n))))


def to_torch(arr, device="cuda"):
    import torch
    if arr.dtype == np.uint16:  # bf16 bit patterns
        return torch.from_numpy(arr.view(np.int16).copy()).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(arr)).to(device)


def gpu_inputs(w, alias=True):
    q = to_torch(w.q)
    k = q if (alias and w.same_points) else to_torch(w.k)
    v = to_torch(w.v)
    g = to_torch(w.g) if w.g is not None else None
    return q, k, v, g


def run(w, passes, alias=True, g=None, fused=False):
    """Runs the requested passes on the GPU (separate gauss_sum_fwd /
    gauss_sum_bwd calls, or one gauss_sum_fwd_bwd call when fused); returns
    numpy fp32 results."""
    import torch
    q, k, v, gd = gpu_inputs(w, alias)
    if g is not None:
        gd = to_torch(g)
    res = {}
    want = tuple(p in passes for p in ("dq", "dk", "dv"))
    if fused:
        s, dq, dk, dv = gs.gauss_sum_fwd_bwd(q, k, v, float(w.tau), gd, want=want)
        res.update({"fwd": s, "dq": dq, "dk": dk, "dv": dv})
    else:
        if "fwd" in passes:
            res["fwd"] = gs.gauss_sum_fwd(q, k, v, float(w.tau))
        if any(want):
            dq, dk, dv = gs.gauss_sum_bwd(q, k, v, float(w.tau), gd, want=want)
            res.update({"dq": dq, "dk": dk, "dv": dv})
    torch.cuda.synchronize()
    return {k_: t.cpu().numpy() for k_, t in res.items() if t is not None}


def oracle_ref(w, pas, rows=None, g=None):
    g = w.g if g is None else g
    qv, kv = w.q_values, w.k_values
    th = oracle_threads()
    if pas == "fwd":
        return oracle.fwd(qv, kv, w.v, float(w.tau), rows=rows, threads=th)
    if pas in ("dq", "dk"):
        # value and absolute scale; the net scale (w summed over channels
        # before the magnitude) is kept for net_ratio
        fn = oracle.dq_scales if pas == "dq" else oracle.dk_scales
        val, absscale, net = fn(qv, kv, w.v, g, float(w.tau), rows=rows, threads=th)
        NET_SCALES[id(val)] = (val, net)  # the array is held, so its id is not reused
        return val, absscale
    fn = {"dv": oracle.dv}[pas]
    return fn(qv, kv, w.v, g, float(w.tau), rows=rows, threads=th)


# (reference array, net scale) of the gradient references oracle_ref returned,
# by id of the reference array
NET_SCALES = {}


def net_ratio(got, ref):
    """max |gpu - oracle| / net scale over the elements whose net scale is at
    least 1e-3 of the row's largest (the other reading of the gradient
    tolerance; elements whose w cancel almost completely are left out)."""
    entry = NET_SCALES.get(id(ref))
    if entry is None or entry[0] is not ref or not entry[1].size:
        return None
    net = entry[1]
    err = np.abs(np.asarray(got, dtype=np.float64) - ref)
    keep = net >= 1e-3 * np.max(net, axis=1, keepdims=True)
    return float(np.max(np.where(keep, err / np.maximum(net, 1e-300), 0.0)))


def compare(label, got, ref, scale, tol):
    """Asserts the pass rule; returns (max err/A, rel-L2)."""
    got = np.asarray(got, dtype=np.float64)
    assert got.shape == ref.shape, (label, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), "%s: non-finite GPU output" % label
    err = np.abs(got - ref)
    bound = tol * scale + 1e-30
    ratio = err / np.maximum(scale, 1e-300)
    worst = float(ratio.max()) if ratio.size else 0.0
    rel_l2 = float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300)) if ref.size else 0.0
    bad = err > bound
    if bad.any():
        idx = tuple(np.argwhere(bad)[0])
        raise AssertionError("%s: %d elements out of tolerance; first %s gpu=%r oracle=%r A=%r "
                             "(max err/A %.3e, rel-L2 %.3e)" % (label, int(bad.sum()), idx, got[idx],
                                                                ref[idx], scale[idx], worst, rel_l2))
    return worst, rel_l2


def check_workload(w, passes=None, rows=None, key_rows=None, alias=True, label=None, fused=None):
    """Runs ``passes`` on the GPU and checks them against the oracle (all rows,
    or the given query rows / key rows).  With passes holding the forward and
    a gradient, both the separate calls and the fused gauss_sum_fwd_bwd call
    are checked (fused=None), or only one of them (fused=False / True).
    Returns a dict of (max err/A, rel-L2)."""
    passes = passes or w.passes
    label = label or w.name
    grads = any(p in passes for p in ("dq", "dk", "dv"))
    if w.g is None and grads:
        w.g = np.random.default_rng(99).standard_normal((w.M, w.C)).astype(np.float32)
    modes = [False, True] if fused is None and grads and "fwd" in passes else [bool(fused)]
    results = [(f, run(w, passes, alias=alias, fused=f)) for f in modes]
    tol = TOL[w.qk_dtype]
    stats = {}
    for p in passes:
        r = key_rows if p in ("dk", "dv") else rows
        ref, scale = oracle_ref(w, p, rows=r)
        for f, got in results:
            g = got[p] if r is None else got[p][np.asarray(r)]
            key = p + ("/fused" if f else "")
            stats[key] = compare("%s/%s" % (label, key), g, ref, scale, tol)
            nr = net_ratio(g, ref)
            if nr is not None:
                stats[key + "/net"] = nr
    NET_SCALES.clear()
    if len(results) == 2:
        sep, fus = results[0][1], results[1][1]
        for p in ("dk", "dv"):
            if p in sep:
                assert np.array_equal(sep[p], fus[p]), "%s: fused %s differs" % (label, p)
    return stats


def random_workload(seed, M, N, D, C, qk="f16", vdt="f32", gdt="f32", tau=None, spread=1.0,
                    same=False):
    """Small seeded problem for shape sweeps: N(0, spread^2 I) points."""
    rng = np.random.default_rng(seed)
    f32 = np.float32
    x = (spread * rng.standard_normal((M, D))).astype(f32)
    y = x.copy() if same else (spread * rng.standard_normal((N, D))).astype(f32)
    if qk == "f16":
        q, qv = x.astype(np.float16), x.astype(np.float16)
        k, kv = (q, qv) if same else (y.astype(np.float16), y.astype(np.float16))
    else:
        q, qv = wl.bf16_round(x)
        k, kv = (q, qv) if same else wl.bf16_round(y)
    v = rng.standard_normal((N, C)).astype(f32)
    g = rng.standard_normal((M, C)).astype(f32)
    conv = {"f32": lambda a: a, "f16": lambda a: a.astype(np.float16)}
    v = conv[vdt](v)
    g = conv[gdt](g)
    t = np.float32(1.0 / max(D, 1) if tau is None else tau)
    return wl.Workload("rand", M, N, D, C, t, qk, q, k, v, g, ("fwd", "dq", "dk", "dv"), same, qv, kv)
