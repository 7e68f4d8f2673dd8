"""Benchmark: exact Gauss-sum pair interactions per second on one MI355X.

Default workload (one "step" = the whole hot path over one batch):
  mmd_flow -- MMD-gradient-flow shape, M = N = 65536 points in 64-D (two
  Gaussian clouds, means 0 and 0.5*1, fp16), signed two-sample weights
  v = +-1/N (C = 1), tau = 1/median squared pairwise distance; a step is the
  forward sum s = sum_n Phi v_n plus its query gradient dq (upstream gradient
  g = v), i.e. what one MMD-flow iteration evaluates.  By default a step is
  one gauss_sum_fwd_bwd call (the forward and dq from one pass over the pairs);
  --separate times gauss_sum_fwd followed by gauss_sum_bwd instead.

Other workloads (--workload) use the same JSON format: dense_d16 (forward),
svgd (forward + dq, dk, dv), mixture_d32 (forward, --tau), rect_d256
(forward + dq, dk, dv).

Protocol: inputs are generated on the host (seeded), copied to HBM before
timing; W untimed warm-up steps, then exactly K steps bracketed by device
synchronisation, timed with HIP events on the stream the library runs on.
The dominant kernel's per-launch duration is measured with the library's
event hook over the same timed steps.  The fp64 CPU oracle is timed on a
bounded sample of query rows of the same workload (rank 0, one GPU only).

Prints one JSON line.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "Gauss-sum pair interactions/sec (M·N/s) fwd+bwd; % of fp16 MFMA peak"
PEAK_MFMA_F16 = 2.5e15  # MI355X dense fp16 / bf16 matrix peak, flop/s

PASSES = {
    "dense_d16": ("fwd",),
    "mmd_flow": ("fwd", "dq"),
    "svgd": ("fwd", "dq", "dk", "dv"),
    "mixture_d32": ("fwd",),
    "rect_d256": ("fwd", "dq", "dk", "dv"),
}


def flops_per_pair(passes, D, C, fused):
    """Algorithmic flops per (query, key) pair: the matrix contractions of each
    pass (q.k, the value or gradient contraction and, for gradients, the sum
    over keys of P k), no padding or recomputation counted.  A fused forward +
    dq pass computes q.k once: 2D (q.k) + 2C (values) + 2C (w) + 2D (P k)."""
    f = 0
    ps = list(passes)
    if fused and "fwd" in ps and "dq" in ps:
        f += 4 * D + 4 * C
        ps.remove("fwd")
        ps.remove("dq")
    for p in ps:
        if p in ("fwd", "dv"):
            f += 2 * D + 2 * C
        else:  # dq or dk
            f += 4 * D + 2 * C
    return f


def describe(w, passes):
    return ("%s: M=%d queries, N=%d keys, D=%d, C=%d, %s points, tau=%.6g, passes %s"
            % (w.name, w.M, w.N, w.D, w.C, w.qk_dtype, float(w.tau), "+".join(passes)))


def cpu_baseline(w, passes, budget_s=15.0):
    """The fp64 oracle as it stands, on a bounded sample of query rows."""
    import numpy as np

    import oracle

    threads = oracle.default_threads()
    threads = min(threads, 16)
    g = w.g
    if g is None and any(p != "fwd" for p in passes):
        g = np.random.default_rng(99).standard_normal((w.M, w.C)).astype(np.float32)

    def run(rows_q, rows_k):
        t0 = time.perf_counter()
        for p in passes:
            if p == "fwd":
                oracle.fwd(w.q_values, w.k_values, w.v, float(w.tau), rows=rows_q, threads=threads)
            elif p == "dq":
                oracle.dq(w.q_values, w.k_values, w.v, g, float(w.tau), rows=rows_q, threads=threads)
            elif p == "dk":
                oracle.dk(w.q_values, w.k_values, w.v, g, float(w.tau), rows=rows_k, threads=threads)
            else:
                oracle.dv(w.q_values, w.k_values, w.v, g, float(w.tau), rows=rows_k, threads=threads)
        return time.perf_counter() - t0

    # warm up (library load, thread start), calibrate on a few rows, then size
    # the sample to about budget_s seconds
    run(np.arange(1), np.arange(1))
    nq = min(w.M, max(threads, 16))
    nk = min(w.N, max(1, int(nq * w.M / max(w.N, 1)) or 1))
    t = run(np.arange(nq), np.arange(nk))
    scale = max(1.0, budget_s / max(t, 1e-3))
    nq2 = int(min(w.M, max(nq, nq * scale)))
    nk2 = int(min(w.N, max(nk, nk * scale)))
    rng = np.random.default_rng(3)
    rows_q = np.sort(rng.choice(w.M, size=nq2, replace=False))
    rows_k = np.sort(rng.choice(w.N, size=nk2, replace=False))
    t = run(rows_q, rows_k)
    # every pass over the sample costs (sampled rows x all partners) pairs; the
    # metric counts a pair once per step, so the rate is sample pairs / time
    has_q = any(p in ("fwd", "dq") for p in passes)
    has_k = any(p in ("dk", "dv") for p in passes)
    frac = ((nq2 / w.M) if has_q else 0.0) + ((nk2 / w.N) if has_k else 0.0)
    frac /= (int(has_q) + int(has_k))
    pairs = frac * w.M * w.N
    return {
        "value": pairs / t,
        "unit": "pairs/s",
        "cores": threads,
        "kind": "oracle",
        "sample": "fp64 oracle, passes %s on %d of %d query rows%s, each against all partners, %.1f s"
                  % ("+".join(passes), nq2 if has_q else 0, w.M,
                     (" and %d of %d key rows" % (nk2, w.N)) if has_k else "", t),
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=8)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="mmd_flow", choices=sorted(PASSES))
    ap.add_argument("--tau", type=float, default=None, help="mixture_d32 bandwidth (0.1, 1, 10)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-budget", type=float, default=15.0)
    ap.add_argument("--separate", action="store_true",
                    help="time separate gauss_sum_fwd + gauss_sum_bwd calls instead of one "
                         "gauss_sum_fwd_bwd call")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2609_04910_amd import gauss_sum as gs
    from paper_2609_04910_amd import workloads as wl

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    gs.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    passes = PASSES[args.workload]
    tau = args.tau if args.workload == "mixture_d32" else None
    w = wl.make(args.workload, seed=0, tau=tau)
    if w.g is None and any(p != "fwd" for p in passes):
        w.g = np.random.default_rng(99).standard_normal((w.M, w.C)).astype(np.float32)

    def t(a):
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    q = t(w.q)
    k = q if w.same_points else t(w.k)
    v = t(w.v)
    g = t(w.g) if w.g is not None else None
    grads = tuple(p in passes for p in ("dq", "dk", "dv"))
    do_fwd = "fwd" in passes
    fused = do_fwd and any(grads) and not args.separate
    qk_code = gs.GS_F16 if w.qk_dtype == "f16" else gs.GS_BF16
    v_code = {np.dtype(np.float32): gs.GS_F32, np.dtype(np.float16): gs.GS_F16}[w.v.dtype]
    ws_f = gs.gauss_sum_fwd_workspace_size(w.M, w.N, w.D, w.C, qk_code, v_code) if do_fwd else 0
    ws_b = gs.gauss_sum_bwd_workspace_size(w.M, w.N, w.D, w.C, qk_code, v_code, *grads) if any(grads) else 0
    ws_fb = gs.gauss_sum_fwd_bwd_workspace_size(w.M, w.N, w.D, w.C, qk_code, v_code, *grads) if fused else 0
    ws = torch.empty(max(ws_f, ws_b, ws_fb, 1), dtype=torch.uint8, device=dev)
    out = torch.empty((w.M, w.C), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()

    def step():
        if fused:
            gs.gauss_sum_fwd_bwd(q, k, v, float(w.tau), g, want=grads, out=out, workspace=ws,
                                 stream=stream)
            return
        if do_fwd:
            gs.gauss_sum_fwd(q, k, v, float(w.tau), out=out, workspace=ws, stream=stream)
        if any(grads):
            gs.gauss_sum_bwd(q, k, v, float(w.tau), g, want=grads, workspace=ws, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    kind = gs.PROFILE_GRAD if any(grads) else gs.PROFILE_FWD
    launches_per_step = sum(grads[:2]) if any(grads) else 1
    cap = args.steps * max(1, launches_per_step)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    gs.gauss_sum_profile_start(cap, kind)
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    kernel_ms = gs.gauss_sum_profile_stop(cap)
    total_ms = e0.elapsed_time(e1)
    ms_per_step = total_ms / args.steps
    pairs = float(w.M) * float(w.N)
    value = pairs / (ms_per_step * 1e-3)

    # dominant kernel: the gradient kernel when gradients are taken (with the
    # forward sum fused into the dq launch by default), else the forward
    # kernel; one launch processes M*N pairs.  With dk also taken the launches
    # alternate dq (fused) and dk; the per-launch work is averaged.
    if any(grads):
        per_launch = []
        if grads[0]:
            per_launch.append(4 * w.D + (4 if fused else 2) * w.C)
        if grads[1]:
            per_launch.append(4 * w.D + 2 * w.C)
        dom_flops = float(np.mean(per_launch)) * pairs
    else:
        dom_flops = (2 * w.D + 2 * w.C) * pairs
    avg_kernel_ms = float(np.mean(kernel_ms)) if kernel_ms else float("nan")
    achieved = dom_flops / (avg_kernel_ms * 1e-3) / 1e12
    step_flops = flops_per_pair(passes, w.D, w.C, fused) * pairs

    res = {
        "metric": METRIC,
        "value": value,
        "unit": "pairs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16" if w.qk_dtype == "f16" else "bf16",
        "data": "synthetic",
        "config": {"workload": describe(w, passes), "M": w.M, "N": w.N, "D": w.D, "C": w.C,
                   "tau": float(w.tau), "passes": "+".join(passes),
                   "api": "gauss_sum_fwd_bwd" if fused else
                          "+".join(n for n, u in (("gauss_sum_fwd", do_fwd),
                                                  ("gauss_sum_bwd", any(grads))) if u)},
        "mfma_frac_of_peak": step_flops / (ms_per_step * 1e-3) / PEAK_MFMA_F16,
        "roofline": {
            "bound": "mfma",
            "kernel": ("k_dq (forward fused)" if fused else "k_dq") if any(grads) else "k_fwd",
            "achieved": achieved,
            "peak": PEAK_MFMA_F16 / 1e12,
            "unit": "TFLOP/s",
            "frac": achieved / (PEAK_MFMA_F16 / 1e12),
            "traffic": None,
            "avg_launch_ms": avg_kernel_ms,
            "launches": len(kernel_ms),
            "flops_per_launch": dom_flops,
        },
    }
    if not args.no_cpu:
        res["cpu_baseline"] = cpu_baseline(w, passes, args.cpu_budget)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
