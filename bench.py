"""Benchmark: exact Gauss-sum pair interactions per second on one MI355X.

Default workload (one "step" = the whole hot path over one batch):
  rect_d256 -- M = 2^17 queries against N = 2^21 keys in 256-D (independent
  unit-normalised Gaussian vectors, fp16), C = 16 signed values (10 % zero
  rows), tau = 4; a step is the forward sum s and the gradients dq, dk, dv
  of sum(dout * s) for dout ~ N(0, 1): one gauss_sum_fwd_bwd call.  It is the
  largest configuration and the one that runs the forward and all three
  gradients.  The same JSON line carries compact records of the other
  configurations (dense_d16 -- also timed as 1000 back-to-back calls per
  event pair and as single calls --, mmd_flow, svgd, mixture_d32 at
  tau = 0.1, 1, 10); --no-configs leaves them out.

Other workloads (--workload) print one line of the same format for that
workload alone: dense_d16 (forward), mmd_flow (forward + dq, fused; --flow
times gauss_sum_mmd_flow, --separate gauss_sum_fwd + gauss_sum_bwd), svgd
(forward + dq, dk, dv), mixture_d32 (forward, --tau), and the batched
layouts of Sec. 4.

Protocol: inputs are generated on the host (seeded), copied to HBM before
timing.  The step is first repeated, untimed, for --settle-ms of wall time:
under sustained matrix-core load the MI355X takes some tens of milliseconds
to reach its steady shader clock (short bursts run up to ~15 % slower), and a
production loop runs at the steady clock.  Then W untimed warm-up steps and
exactly K steps bracketed by device synchronisation, timed with HIP events on
the stream the library runs on.  The dominant kernel's per-launch duration is
measured with the library's event hook over the same timed steps.  The fp64
CPU oracle is timed on a bounded sample of query rows of the same workload
(rank 0, one GPU only).

roofline.traffic: HBM bytes per launch of the dominant kernel (the mean over
its dispatches, as for the launch time), from the
rocprofv3 FETCH_SIZE and WRITE_SIZE counters (one --pmc run each), scaled by
what the same counters read for a device copy of known size run in the same
process (--calibrate-copy); recorded by --traffic-from into
profiles/traffic_<workload>.json together with a hash of the kernel sources,
and reported only while that hash matches the sources (else null).

Prints one JSON line.
"""
import argparse
import csv
import ctypes
import glob
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "Gauss-sum pair interactions/sec (M·N/s) fwd+bwd; % of fp16 MFMA peak"
PEAK_MFMA_F16 = 2.5e15  # MI355X dense fp16 / bf16 matrix peak, flop/s
# v_exp_f32 at a quarter of the fp32 lane rate: the published 157.3 TFLOP/s fp32
# vector peak is 256 CUs x 4 SIMDs x 32 lanes x 2 flop x 2.4 GHz, so a quarter
# rate is 8 exponentials per SIMD and clock
EXP_NOMINAL = 256 * 4 * 32 / 4 * 2.4e9
PEAKS_FILE = os.path.join(ROOT, "profiles", "peaks_mi355x.json")

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


def algorithmic_flops_per_pair(passes, D, C):
    """The step's algorithmic flops per pair, independent of how the library
    splits it into launches: the forward 2D+2C (q.k and the value
    contraction); the backward 2D for its own q.k, 2C for <g, v> (dq or dk),
    2D each for the sums of P k (dq) and P q (dk), 2C for dv -- the full
    backward 6D+4C, so forward plus full backward is 8D+6C.  With dq the
    only gradient the forward and dq are one pass over the same q.k tiles,
    counted once: 4D+4C."""
    dq, dk, dv, fwd = "dq" in passes, "dk" in passes, "dv" in passes, "fwd" in passes
    f = 2 * D + 2 * C if fwd else 0
    if dq or dk or dv:
        f += 2 * D + (2 * C if (dq or dk) else 0) + 2 * D * dq + 2 * D * dk + 2 * C * dv
        if fwd and dq and not dk and not dv:
            f -= 2 * D
    return f


KERNELS = {"fused": "k_dq", "grad": "k_dq", "fwd": "k_fwd"}
COPY_KERNEL_HINT = "copy"  # torch's device-to-device copy kernel name contains it


def kernel_sources_hash():
    """sha256 over the HIP sources of the library (the kernels the counters measured)."""
    h = hashlib.sha256()
    d = os.path.join(ROOT, "paper_2609_04910_amd", "csrc")
    for f in sorted(os.listdir(d)):
        with open(os.path.join(d, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()


def dominant_kernel_name(workload):
    """Name fragment of the kernel the roofline of `workload` is reported for
    (the one whose traffic --traffic-from records)."""
    if workload == "batch_grad_d32":
        return "k_dq"
    if workload.startswith("batch_"):
        return "k_fwd32" if workload.endswith("_f32") else "k_fwd"
    return "k_dq" if any(p != "fwd" for p in PASSES[workload]) else "k_fwd"


def traffic_file(workload):
    return os.path.join(ROOT, "profiles", "traffic_%s.json" % workload)


def read_counter_csv(d, counter):
    """{kernel name: [value per dispatch]} for `counter` from a rocprofv3 csv output dir."""
    out = {}
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        with open(f) as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] == counter:
                    out.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
    return out


def traffic_from(workload, fetch_dir, write_dir, copy_bytes, dominant):
    """Record HBM bytes per launch of the dominant kernel from two --pmc runs."""
    rec = {"workload": workload, "kernel": dominant, "kernel_sources_sha256": kernel_sources_hash()}
    for key, d, counter in (("fetch", fetch_dir, "FETCH_SIZE"), ("write", write_dir, "WRITE_SIZE")):
        vals = read_counter_csv(d, counter)
        dom = [v for name, vs in vals.items() if dominant in name for v in vs]
        cpy = [v for name, vs in vals.items() if COPY_KERNEL_HINT in name.lower() for v in vs]
        if not dom or not cpy:
            raise SystemExit("traffic: no %s samples for %s / the copy kernel in %s" % (counter, dominant, d))
        kib_dom = sum(dom) / len(dom)                 # mean over dispatches, as the launch time
        kib_cpy = max(cpy)                            # the calibration copies are the largest
        factor = copy_bytes / (kib_cpy * 1024.0)      # bytes moved per counted byte
        rec[key] = {"counter_kib_per_launch": kib_dom, "copy_counter_kib": kib_cpy,
                    "copy_bytes_each_way": copy_bytes, "scale": factor,
                    "bytes_per_launch": kib_dom * 1024.0 * factor}
    rec["bytes_per_launch"] = rec["fetch"]["bytes_per_launch"] + rec["write"]["bytes_per_launch"]
    with open(traffic_file(workload), "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")
    print(json.dumps(rec))


def recorded_traffic(workload, dominant):
    """Bytes per launch recorded for these kernel sources, else None."""
    try:
        with open(traffic_file(workload)) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None
    if rec.get("kernel") != dominant or rec.get("kernel_sources_sha256") != kernel_sources_hash():
        return None
    return rec.get("bytes_per_launch")


def measured_peaks():
    """Rates measured on an MI355X by `bench.py --peaks` (libgs_peaks.so), or None."""
    try:
        with open(PEAKS_FILE) as fh:
            return json.load(fh)
    except (OSError, ValueError):
        return None


def measured_mfma(achieved_tflops):
    """The dominant kernel's throughput against the measured 16x16x32 f16 MFMA rate."""
    pk = measured_peaks()
    if not pk:
        return {}
    m = pk["mfma_f16_16x16x32_flop_per_s"] / 1e12
    return {"peak_measured": m, "frac_of_measured": achieved_tflops / m}


def exp_rate(pairs_per_launch, avg_ms):
    """Exponentials per second of the dominant kernel (one exp2 per pair and
    launch) against the nominal and the measured v_exp_f32 rates."""
    got = pairs_per_launch / (avg_ms * 1e-3)
    out = {"achieved": got, "unit": "exp/s", "peak_nominal": EXP_NOMINAL, "frac_nominal": got / EXP_NOMINAL}
    pk = measured_peaks()
    if pk:
        out["peak_measured"] = pk["exp2_per_s"]
        out["frac_measured"] = got / pk["exp2_per_s"]
    return out


def bench_peaks(args):
    """Measure the device's own rates with libgs_peaks.so and print them as one
    JSON line (the record profiles/peaks_mi355x.json holds)."""
    import torch

    from paper_2609_04910_amd import peaks

    rec = peaks.measure()
    rec.update({"device": torch.cuda.get_device_name(0), "mfma_nominal_flop_per_s": PEAK_MFMA_F16,
                "exp2_nominal_per_s": EXP_NOMINAL, "hbm_nominal_bytes_per_s": 8e12})
    print(json.dumps(rec), flush=True)


def describe(w, passes):
    return ("%s: M=%d queries, N=%d keys, D=%d, C=%d, %s points, tau=%.6g, passes %s"
            % (w.name, w.M, w.N, w.D, w.C, w.qk_dtype, float(w.tau), "+".join(passes)))


def cpu_baseline(w, passes, budget_s=15.0):
    """The fp64 oracle as it stands, on a bounded sample of query rows."""
    import numpy as np

    import oracle

    threads = oracle.default_threads()   # every host core this process may run on
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
    rng = np.random.default_rng(3)
    t = run(np.arange(nq), np.arange(nk))
    # grow the sample until it takes at least half the budget (the first
    # calls include thread start-up, so one extrapolation can undershoot)
    for _ in range(4):
        if t >= 0.5 * budget_s or (nq >= w.M and nk >= w.N):
            break
        scale = min(64.0, max(1.5, budget_s / max(t, 1e-3)))
        nq = int(min(w.M, max(nq + 1, nq * scale)))
        nk = int(min(w.N, max(nk + 1, nk * scale)))
        rows_q = np.sort(rng.choice(w.M, size=nq, replace=False))
        rows_k = np.sort(rng.choice(w.N, size=nk, replace=False))
        t = run(rows_q, rows_k)
    nq2, nk2 = nq, nk
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
        "cpu_model": cpu_model(),
        "kind": "oracle",
        "sample": "fp64 oracle, passes %s on %d of %d query rows%s, each against all partners, %.1f s"
                  % ("+".join(passes), nq2 if has_q else 0, w.M,
                     (" and %d of %d key rows" % (nk2, w.N)) if has_k else "", t),
        # the whole step (all M x N pairs of every pass) at the sampled rate
        "full_problem_s_extrapolated": w.M * float(w.N) / (pairs / t),
    }


def cpu_model():
    """The host CPU's model name (from /proc/cpuinfo), or None."""
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def fused_passes(D, C):
    """Which forward-type sums the library computes inside a gradient launch
    (the fusion rule of gauss_sum_fwd_bwd): (forward inside the dq pass, dv
    inside the dk pass)."""
    f = C <= 16
    return f, f


def dominant_flops(passes, D, C, fused_call):
    """Algorithmic flops per pair of one launch of the dominant kernel: a
    gradient launch (dq or dk, averaged over the gradient launches of a step)
    when gradients are taken, else the forward launch."""
    fwd_in_dq, dv_in_dk = fused_passes(D, C)
    per_launch = []
    if "dq" in passes:
        per_launch.append(4 * D + (4 if (fused_call and "fwd" in passes and fwd_in_dq) else 2) * C)
    if "dk" in passes:
        per_launch.append(4 * D + (4 if ("dv" in passes and dv_in_dk) else 2) * C)
    if per_launch:
        return sum(per_launch) / len(per_launch)
    return 2 * D + 2 * C


def calibration_copy(mib, dev):
    """Three device copies of `mib` MiB (the known-size kernel that --pmc runs
    scale FETCH_SIZE / WRITE_SIZE by); nothing for mib = 0."""
    if not mib:
        return
    import torch
    src = torch.empty(mib * 1024 * 1024, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def clean(res):
    """The result without the private (underscore) entries."""
    return {k: v for k, v in res.items() if not k.startswith("_")}


def measure_workload(args, name, tau, steps, warmup, settle_ms, graph=False, flow=False, separate=False,
                     calibrate_copy=0, calls_per_pair=0):
    """Times `steps` steps of workload `name` on cuda:0 (inputs resident in
    HBM; untimed settle and warm-up first) and returns the benchmark record:
    pairs/s, ms per step, the dominant kernel's roofline from the library's
    HIP-event hook.  calls_per_pair > 0 also times that many back-to-back
    steps between one pair of events and single steps one at a time (the
    launch-latency floor of the smallest problem)."""
    import numpy as np
    import torch

    from paper_2609_04910_amd import gauss_sum as gs
    from paper_2609_04910_amd import workloads as wl

    dev = torch.device("cuda:0")
    passes = PASSES[name]
    w = wl.make(name, seed=0, tau=tau)
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
    if flow and name != "mmd_flow":
        print("--flow applies to the mmd_flow workload only", file=sys.stderr)
        sys.exit(2)
    fused = do_fwd and any(grads) and not separate
    qk_code = gs.GS_F16 if w.qk_dtype == "f16" else gs.GS_BF16
    v_code = {np.dtype(np.float32): gs.GS_F32, np.dtype(np.float16): gs.GS_F16}[w.v.dtype]
    ws_f = gs.gauss_sum_fwd_workspace_size(w.M, w.N, w.D, w.C, qk_code, v_code) if do_fwd else 0
    ws_b = gs.gauss_sum_bwd_workspace_size(w.M, w.N, w.D, w.C, qk_code, v_code, *grads) if any(grads) else 0
    ws_fb = gs.gauss_sum_fwd_bwd_workspace_size(w.M, w.N, w.D, w.C, qk_code, v_code, *grads) if fused else 0
    ws_fl = gs.gauss_sum_mmd_flow_workspace_size(w.N, w.D, qk_code, v_code) if flow else 0
    ws = torch.empty(max(ws_f, ws_b, ws_fb, ws_fl, 1), dtype=torch.uint8, device=dev)
    out = torch.empty((w.M, w.C), dtype=torch.float32, device=dev)
    dq = torch.empty((w.M, w.D), dtype=torch.float32, device=dev) if grads[0] else None
    dk = torch.empty((w.N, w.D), dtype=torch.float32, device=dev) if grads[1] else None
    dv = torch.empty((w.N, w.C), dtype=torch.float32, device=dev) if grads[2] else None
    stream = torch.cuda.current_stream()
    lib = gs.load()
    prob = gs.make_problem(w.M, w.N, w.D, w.C, qk_code, v_code)
    g_code = gs.GS_F32 if g is None else gs._dtype_code(g.dtype)
    nbytes = ws.numel()
    P = gs._ptr

    # the step calls the C ABI directly (outputs and workspace preallocated),
    # so the timed region holds library work only
    def step(on=None):
        s_ = (stream if on is None else on).cuda_stream
        if flow:
            gs.gauss_sum_mmd_flow(q, v, float(w.tau), workspace=ws, stream=stream if on is None else on)
            return
        if fused:
            st = lib.gauss_sum_fwd_bwd(ctypes.byref(prob), P(q), P(k), P(v), float(w.tau), P(g), g_code,
                                       P(out), P(dq), P(dk), P(dv), P(ws), nbytes, ctypes.c_void_p(s_))
        else:
            st = 0
            if do_fwd:
                st = lib.gauss_sum_fwd(ctypes.byref(prob), P(q), P(k), P(v), float(w.tau), P(out), P(ws), nbytes,
                                       ctypes.c_void_p(s_))
            if any(grads) and st == 0:
                st = lib.gauss_sum_bwd(ctypes.byref(prob), P(q), P(k), P(v), float(w.tau), P(g), g_code, P(dq),
                                       P(dk), P(dv), P(ws), nbytes, ctypes.c_void_p(s_))
        if st != 0:
            raise gs.GaussSumError(st, "benchmark step")

    calibration_copy(calibrate_copy, dev)

    settle_steps = 0
    t_settle = time.perf_counter()
    while settle_steps == 0 or (time.perf_counter() - t_settle) * 1e3 < settle_ms:
        step()
        settle_steps += 1
        torch.cuda.synchronize()
    settle_ms_done = (time.perf_counter() - t_settle) * 1e3
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()

    kind = gs.PROFILE_GRAD if any(grads) else gs.PROFILE_FWD
    launches_per_step = sum(grads[:2]) if any(grads) else 1
    cap = steps * max(1, launches_per_step)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    gs.gauss_sum_profile_start(cap, kind)
    e0.record(stream)
    for _ in range(steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    kernel_ms = gs.gauss_sum_profile_stop(cap)
    ms_per_step = e0.elapsed_time(e1) / steps
    eager_ms = ms_per_step
    extra = {}
    if calls_per_pair:
        e0.record(stream)
        for _ in range(calls_per_pair):
            step()
        e1.record(stream)
        torch.cuda.synchronize()
        extra["ms_per_call_back_to_back"] = e0.elapsed_time(e1) / calls_per_pair
        extra["calls_per_event_pair"] = calls_per_pair
        single = []
        for _ in range(20):
            torch.cuda.synchronize()
            e0.record(stream)
            step()
            e1.record(stream)
            torch.cuda.synchronize()
            single.append(e0.elapsed_time(e1))
        extra["ms_single_call_median"] = float(np.median(single))
        ms_per_step = extra["ms_per_call_back_to_back"]
    if graph:
        # the same step captured once in a HIP graph and replayed
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            step(side)
        stream.wait_stream(side)
        torch.cuda.synchronize()
        cg = torch.cuda.CUDAGraph()
        with torch.cuda.graph(cg):
            step(torch.cuda.current_stream())
        for _ in range(max(1, warmup)):
            cg.replay()
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(steps):
            cg.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        ms_per_step = e0.elapsed_time(e1) / steps
    pairs = float(w.M) * float(w.N)
    value = pairs / (ms_per_step * 1e-3)

    # dominant kernel: the gradient kernel when gradients are taken, else the
    # forward kernel; one launch processes M*N pairs
    fwd_in_dq, _ = fused_passes(w.D, w.C)
    dom_flops = dominant_flops(passes, w.D, w.C, fused) * pairs
    avg_kernel_ms = float(np.mean(kernel_ms)) if kernel_ms else float("nan")
    achieved = dom_flops / (avg_kernel_ms * 1e-3) / 1e12
    step_flops = flops_per_pair(passes, w.D, w.C, fused) * pairs
    alg_flops = algorithmic_flops_per_pair(passes, w.D, w.C) * pairs

    res = {
        "metric": METRIC,
        "value": value,
        "unit": "pairs/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "settle": {"ms": settle_ms_done, "steps": settle_steps},
        "ms_per_step": ms_per_step,
        # device memory beyond inputs and outputs (the caller-owned workspace)
        "workspace_bytes": int(ws.numel()),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16" if w.qk_dtype == "f16" else "bf16",
        "data": "synthetic",
        "config": {"workload": describe(w, passes), "M": w.M, "N": w.N, "D": w.D, "C": w.C,
                   "tau": float(w.tau), "passes": "+".join(passes),
                   "api": "gauss_sum_mmd_flow" if flow else "gauss_sum_fwd_bwd" if fused else
                          "+".join(n for n, u in (("gauss_sum_fwd", do_fwd),
                                                  ("gauss_sum_bwd", any(grads))) if u),
                   "graph": bool(graph)},
        "mfma_frac_of_peak": step_flops / (ms_per_step * 1e-3) / PEAK_MFMA_F16,
        "step_roofline": {"flops_per_pair": algorithmic_flops_per_pair(passes, w.D, w.C),
                          "basis": "algorithmic flops per pair of the step (forward 2D+2C, full "
                                   "backward 6D+4C; fwd+dq 4D+4C) over the step time",
                          "achieved": alg_flops / (ms_per_step * 1e-3) / 1e12, "unit": "TFLOP/s",
                          "peak": PEAK_MFMA_F16 / 1e12,
                          "frac": alg_flops / (ms_per_step * 1e-3) / PEAK_MFMA_F16},
        "roofline": {
            "bound": "mfma",
            "kernel": ("k_dq (forward fused)" if (fused and fwd_in_dq) else "k_dq") if any(grads) else "k_fwd",
            "achieved": achieved,
            "peak": PEAK_MFMA_F16 / 1e12,
            "unit": "TFLOP/s",
            "frac": achieved / (PEAK_MFMA_F16 / 1e12),
            "traffic": recorded_traffic(name, "k_dq" if any(grads) else "k_fwd"),
            "avg_launch_ms": avg_kernel_ms,
            "std_launch_ms": float(np.std(kernel_ms)) if kernel_ms else float("nan"),
            "launches": len(kernel_ms),
            "flops_per_launch": dom_flops,
        },
    }
    res["roofline"].update(measured_mfma(achieved))
    res["roofline"]["exp"] = exp_rate(pairs, avg_kernel_ms)
    res.update(extra)
    if graph:
        res["eager_ms_per_step"] = eager_ms
    res["_workload"] = w
    res["_passes"] = passes
    del q, k, v, g, ws, out, dq, dk, dv
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res


def sub_record(res, tau=None):
    """The compact form of a workload's record that the headline line carries."""
    pk = measured_peaks()
    c = res["config"]
    pairs = float(c["M"]) * c["N"]
    out = {"workload": c["workload"].split(":")[0], "M": c["M"], "N": c["N"], "D": c["D"], "C": c["C"],
           "tau": c["tau"], "passes": c["passes"], "api": c["api"], "steps": res["steps"],
           "ms_per_step": res["ms_per_step"], "pairs_per_s": res["value"],
           "step_frac_of_mfma_peak": res["step_roofline"]["frac"],
           "kernel": res["roofline"]["kernel"], "avg_launch_ms": res["roofline"]["avg_launch_ms"],
           "kernel_frac_of_mfma_peak": res["roofline"]["frac"],
           "workspace_bytes": res.get("workspace_bytes")}
    if c["D"] <= 32:
        # one exponential per pair and pass: the target for D <= 32 is stated
        # against the exponential rate
        out["exp_per_s_step"] = pairs * len(c["passes"].split("+")) / (res["ms_per_step"] * 1e-3)
        out["exp_per_s_kernel"] = res["roofline"]["exp"]["achieved"]
        if pk:
            out["step_frac_of_measured_exp_rate"] = out["exp_per_s_step"] / pk["exp2_per_s"]
            out["kernel_frac_of_measured_exp_rate"] = out["exp_per_s_kernel"] / pk["exp2_per_s"]
    for key in ("ms_per_call_back_to_back", "calls_per_event_pair", "ms_single_call_median"):
        if key in res:
            out[key] = res[key]
    return out


def bench_headline(args):
    """The benchmark line: rect_d256 (the largest configuration, forward and
    all three gradients) as the headline, with compact records of the other
    configurations (dense_d16 with back-to-back and single calls, mmd_flow,
    svgd, mixture_d32 at each tau) in the same JSON line."""
    import torch

    configs = []
    if not args.no_configs:
        for name, tau, steps in (("dense_d16", None, 20), ("mmd_flow", None, 20), ("svgd", None, 20),
                                 ("mixture_d32", 0.1, 5), ("mixture_d32", 1.0, 5), ("mixture_d32", 10.0, 5)):
            print("config", name, tau, flush=True, file=sys.stderr)
            r = measure_workload(args, name, tau, steps, 2, 200.0,
                                 calls_per_pair=1000 if name == "dense_d16" else 0)
            configs.append(sub_record(r))
            del r
            torch.cuda.empty_cache()
    print("headline rect_d256", flush=True, file=sys.stderr)
    res = measure_workload(args, "rect_d256", None, args.steps, args.warmup, args.settle_ms,
                           calibrate_copy=args.calibrate_copy)
    if configs:
        res["configs"] = configs
    if not args.no_cpu:
        res["cpu_baseline"] = cpu_baseline(res.pop("_workload"), res.pop("_passes"), args.cpu_budget)
    print(json.dumps(clean(res)), flush=True)


def bench_batched(args):
    """Batched forward (the paper's benchmark layout): one gauss_sum_fwd_batched
    call per step over B independent clouds; pairs/s counts B M N per step."""
    import numpy as np
    import torch

    import oracle
    from paper_2609_04910_amd import gauss_sum as gs
    from paper_2609_04910_amd import workloads as wl

    dev = torch.device("cuda:0")
    cfg = wl.BATCHED[args.workload]
    q, k, v, tau = wl.make_batch(args.workload, seed=0)
    B, M, D = q.shape
    N, C = v.shape[1], v.shape[2]
    tq, tk, tv = (torch.from_numpy(a).to(dev) for a in (q, k, v))
    # room for every problem in one launch group
    f32 = q.dtype == np.float32
    qk_code = gs.GS_F32 if f32 else gs.GS_F16
    p_ws = gs.gauss_sum_fwd_batched_workspace_size(M, N, D, C, B, qk_code, gs.GS_F32)
    ws = torch.empty(max(p_ws, 1), dtype=torch.uint8, device=dev)
    out = torch.empty((B, M, C), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()

    def step():
        gs.gauss_sum_fwd_batched(tq, tk, tv, float(tau), out=out, workspace=ws, stream=stream)

    calibration_copy(args.calibrate_copy, dev)
    settle_steps, t0 = 0, time.perf_counter()
    while settle_steps == 0 or (time.perf_counter() - t0) * 1e3 < args.settle_ms:
        step()
        settle_steps += 1
        torch.cuda.synchronize()
    settle_ms = (time.perf_counter() - t0) * 1e3
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    cap = args.steps * B
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    gs.gauss_sum_profile_start(cap, gs.PROFILE_FWD)
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    kernel_ms = gs.gauss_sum_profile_stop(cap)
    ms_per_step = e0.elapsed_time(e1) / args.steps
    pairs = float(B) * M * N
    per_step = max(1, len(kernel_ms) // args.steps)     # forward launches per step
    per_launch = float(B) / per_step * M * N * (2 * D + 2 * C)
    avg = float(np.mean(kernel_ms)) if kernel_ms else float("nan")
    achieved = per_launch / (avg * 1e-3) / 1e12
    # fp32 points: every fp32-accurate product of the scores is three fp16
    # MFMA products (split operands), so the ceiling of that contraction is a
    # third of the fp16 peak
    peak = PEAK_MFMA_F16 / (3.0 if f32 else 1.0)
    res = {
        "metric": METRIC, "value": pairs / (ms_per_step * 1e-3), "unit": "pairs/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "settle": {"ms": settle_ms, "steps": settle_steps},
        "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32" if f32 else "f16", "data": "synthetic",
        "config": {"workload": "%s: B=%d independent clouds, M=N=%d, D=%d, C=%d, %s points "
                               "N(0, I/D), tau=1, forward" % (args.workload, B, M, D, C,
                                                              "f32" if f32 else "f16"),
                   "B": B, "M": M, "N": N, "D": D, "C": C, "tau": float(tau), "passes": "fwd",
                   "api": "gauss_sum_fwd_batched"},
        "mfma_frac_of_peak": pairs * (2 * D + 2 * C) / (ms_per_step * 1e-3) / peak,
        "roofline": {"bound": "mfma", "kernel": ("k_fwd32" if C == 1 else "k_fwd32c") if f32 else "k_fwd",
                     "achieved": achieved,
                     "peak": peak / 1e12, "unit": "TFLOP/s", "frac": achieved / (peak / 1e12),
                     "peak_basis": "fp16 MFMA peak / 3 (split fp32 products)" if f32 else "fp16 MFMA peak",
                     "traffic": recorded_traffic(args.workload, "k_fwd32" if f32 else "k_fwd"),
                     "avg_launch_ms": avg,
                     "launches": len(kernel_ms), "problems_per_launch": B // per_step,
                     "flops_per_launch": per_launch,
                     "launch_share_of_step": avg * per_step / ms_per_step},
    }
    if not f32:
        res["roofline"].update(measured_mfma(achieved))
    res["roofline"]["exp"] = exp_rate(float(B) / per_step * M * N, avg)
    if not args.no_cpu:
        threads = oracle.default_threads()
        oracle.fwd(q[0], k[0], v[0], float(tau), rows=np.arange(1), threads=threads)
        # whole problems (every query row against every key), in order, until
        # the time budget is spent
        t0, done = time.perf_counter(), 0
        while done < B and (done == 0 or time.perf_counter() - t0 < args.cpu_budget):
            oracle.fwd(q[done], k[done], v[done], float(tau), threads=threads)
            done += 1
        t = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": done * float(M) * N / t, "unit": "pairs/s", "cores": threads,
                               "kind": "oracle",
                               "sample": "fp64 oracle, forward of problems 0..%d of %d (all %d x %d "
                                         "pairs each), %.1f s" % (done - 1, B, M, N, t)}
    print(json.dumps(res), flush=True)


def bench_batched_grad(args):
    """Batched forward plus backward (the paper's forward-and-backward
    benchmark layout, Sec. 4): one gauss_sum_fwd_bwd_batched call per step
    over B independent clouds giving s and dq, dk, dv for an upstream gradient
    dout; pairs/s counts B M N per step."""
    import numpy as np
    import torch

    import oracle
    from paper_2609_04910_amd import gauss_sum as gs
    from paper_2609_04910_amd import workloads as wl

    dev = torch.device("cuda:0")
    q, k, v, tau = wl.make_batch(args.workload, seed=0)
    g = wl.batch_dout(args.workload, seed=0)
    B, M, D = q.shape
    N, C = v.shape[1], v.shape[2]
    tq, tk, tv, tg = (torch.from_numpy(a).to(dev) for a in (q, k, v, g))
    ws = torch.empty(max(gs.gauss_sum_fwd_bwd_batched_workspace_size(M, N, D, C, B), 1),
                     dtype=torch.uint8, device=dev)
    out = torch.empty((B, M, C), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()

    def step():
        gs.gauss_sum_fwd_bwd_batched(tq, tk, tv, float(tau), tg, out=out, workspace=ws, stream=stream)

    calibration_copy(args.calibrate_copy, dev)
    settle_steps, t0 = 0, time.perf_counter()
    while settle_steps == 0 or (time.perf_counter() - t0) * 1e3 < args.settle_ms:
        step()
        settle_steps += 1
        torch.cuda.synchronize()
    settle_ms = (time.perf_counter() - t0) * 1e3
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    cap = args.steps * 4
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    gs.gauss_sum_profile_start(cap, gs.PROFILE_GRAD)
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    kernel_ms = gs.gauss_sum_profile_stop(cap)
    ms_per_step = e0.elapsed_time(e1) / args.steps
    pairs = float(B) * M * N
    # gradient-kind launches per step: the dq pass (forward fused) and the dk
    # pass (dv fused where the forward fusion applies: C <= 16)
    per_step = max(1, len(kernel_ms) // args.steps)
    grad_ms = float(np.sum(kernel_ms)) / args.steps if kernel_ms else float("nan")
    fused_kv = fused_passes(D, C)[1]
    # algorithmic flops per pair: a gradient pass with a forward-type sum fused
    # 4D+4C (4D+2C for the gradient, 2C more for the sum), else 4D+2C for dk
    # and a separate dv pass 2D+2C
    grad_flops = pairs * ((4 * D + 4 * C) + (4 * D + (4 if fused_kv else 2) * C))
    flops = grad_flops + (0 if fused_kv else pairs * (2 * D + 2 * C))
    res = {
        "metric": METRIC, "value": pairs / (ms_per_step * 1e-3), "unit": "pairs/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "settle": {"ms": settle_ms, "steps": settle_steps},
        "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f16", "data": "synthetic",
        "config": {"workload": "%s: B=%d independent clouds, M=N=%d, D=%d, C=%d, f16 points N(0, I/D), "
                               "tau=1, forward and gradients w.r.t. q, k, v" % (args.workload, B, M, D, C),
                   "B": B, "M": M, "N": N, "D": D, "C": C, "tau": float(tau), "passes": "fwd+dq+dk+dv",
                   "api": "gauss_sum_fwd_bwd_batched"},
        "mfma_frac_of_peak": flops / (ms_per_step * 1e-3) / PEAK_MFMA_F16,
        "roofline": {"bound": "mfma", "kernel": "k_dq (dq pass with the forward fused, dk pass with dv fused)",
                     "achieved": grad_flops / (grad_ms * 1e-3) / 1e12, "peak": PEAK_MFMA_F16 / 1e12,
                     "unit": "TFLOP/s",
                     "frac": grad_flops / (grad_ms * 1e-3) / PEAK_MFMA_F16,
                     "traffic": recorded_traffic(args.workload, "k_dq"),
                     "avg_launch_ms": grad_ms / per_step, "launches": len(kernel_ms),
                     "launches_per_step": per_step, "flops_per_step": grad_flops,
                     "launch_share_of_step": grad_ms / ms_per_step},
    }
    res["roofline"].update(measured_mfma(res["roofline"]["achieved"]))
    # two passes over every pair per step (dq, dk), one exponential each
    res["roofline"]["exp"] = exp_rate(2.0 * pairs / per_step, grad_ms / per_step)
    if not args.no_cpu:
        threads = oracle.default_threads()
        rows = wl.sample_rows(M, 64, seed=5)
        oracle.dq(q[0], k[0], v[0], g[0], float(tau), rows=rows[:1], threads=threads)
        t0, done = time.perf_counter(), 0
        while done == 0 or time.perf_counter() - t0 < args.cpu_budget:
            b = done % B
            oracle.fwd(q[b], k[b], v[b], float(tau), rows=rows, threads=threads)
            oracle.dq(q[b], k[b], v[b], g[b], float(tau), rows=rows, threads=threads)
            oracle.dk(q[b], k[b], v[b], g[b], float(tau), rows=rows, threads=threads)
            oracle.dv(q[b], k[b], v[b], g[b], float(tau), rows=rows, threads=threads)
            done += 1
        t = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": done * len(rows) * float(N) / t, "unit": "pairs/s",
                               "cores": threads, "kind": "oracle",
                               "sample": "fp64 oracle, forward, dq, dk and dv on %d sampled rows of a "
                                         "problem (each against all %d partners), %d problems, %.1f s"
                                         % (len(rows), N, done, t)}
    print(json.dumps(res), flush=True)


def bench_svgd_update(args):
    """One gauss_sum_svgd call per step on the svgd workload's particles and
    score-like values (the SVGD direction of Sec. 3: forward sum with values
    score plus the repulsive query-gradient term); prints one JSON line with
    the step time and pairs/s (N^2 per step).  A secondary measurement, not
    the benchmark line."""
    import numpy as np
    import torch

    from paper_2609_04910_amd import gauss_sum as gs
    from paper_2609_04910_amd import workloads as wl

    dev = torch.device("cuda:0")
    w = wl.make("svgd", seed=0)
    x = torch.from_numpy(w.q).to(dev)
    sc = torch.from_numpy(np.ascontiguousarray(w.v)).to(dev)
    ws = torch.empty(max(gs.gauss_sum_svgd_workspace_size(w.N, w.D, gs.GS_F16, gs.GS_F16), 1),
                     dtype=torch.uint8, device=dev)
    out = torch.empty((w.N, w.D), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()

    def step():
        gs.gauss_sum_svgd(x, sc, float(w.tau), out=out, workspace=ws, stream=stream)

    t0 = time.perf_counter()
    while (time.perf_counter() - t0) * 1e3 < args.settle_ms:
        step()
        torch.cuda.synchronize()
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    print(json.dumps({"mode": "svgd_update", "unit": "pairs/s", "data": "synthetic",
                      "config": {"workload": "svgd particles: N=%d, D=%d, f16, score-like values -x + "
                                             "0.1 eps (f16), tau=%g" % (w.N, w.D, float(w.tau)),
                                 "api": "gauss_sum_svgd"},
                      "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
                      "pairs_per_s": float(w.N) * w.N / (ms * 1e-3)}), flush=True)


def compare_attention_grad(args):
    """The paper's gradient route on this GPU, as an external comparison (not
    part of the library): Alg. 2 (reweight) through PyTorch's public
    scaled_dot_product_attention with automatic differentiation, the backward
    pass again in the fused attention kernels (Sec. 2, Remark 1; Alg. 1 needs
    the log-sum-exp output, which the attention backward does not
    differentiate), for s and the gradients of sum(dout * s) with respect to
    q, k and v in fp16, beside one gauss_sum_fwd_bwd_batched call.  Each route
    is timed like the library and checked against the fp64 oracle on sampled
    rows of three problems (relative L2 error of s and of dq).  Prints one
    JSON line."""
    import numpy as np
    import torch
    import torch.nn.functional as F
    from torch.nn.attention import SDPBackend, sdpa_kernel

    import oracle
    from paper_2609_04910_amd import gauss_sum as gs
    from paper_2609_04910_amd import workloads as wl

    dev = torch.device("cuda:0")
    q, k, v, tau = wl.make_batch(args.workload, seed=0, M=args.batch_n)
    g = wl.batch_dout(args.workload, seed=0, M=args.batch_n)
    tau = float(tau)
    B, M, D = q.shape
    N, C = v.shape[1], v.shape[2]
    tq, tk, tv, tg = (torch.from_numpy(a).to(dev) for a in (q, k, v, g))
    stream = torch.cuda.current_stream()
    ceil8 = lambda x: (x + 7) // 8 * 8
    kappa = float(np.sqrt(N + 1))
    lq = tq.clone().requires_grad_(True)
    lk = tk.clone().requires_grad_(True)
    lv = tv.clone().requires_grad_(True)

    def reweight(backend):
        for t in (lq, lk, lv):
            t.grad = None
        mu = torch.cat([lq, lk], 1).float().mean(dim=1, keepdim=True)
        qc = (lq.float() - mu).half()
        kc = (lk.float() - mu).half()
        nq, nk = qc.float().pow(2).sum(-1), kc.float().pow(2).sum(-1)
        w = ceil8(max(D + 2, C + 1))
        Q = torch.zeros((B, M, w), dtype=torch.float16, device=dev)
        Q[..., :D] = qc
        Q[..., D] = 1.0
        Q[..., D + 1] = (0.5 * nq).half()
        K = torch.zeros((B, N + 1, w), dtype=torch.float16, device=dev)
        K[:, 0, D + 1] = 1.0
        K[:, 1:, :D] = kc
        K[:, 1:, D] = (-0.5 * nk).half()
        V = torch.zeros((B, N + 1, w), dtype=torch.float16, device=dev)
        V[:, 1:, :C] = lv.half()
        V[:, 0, C] = kappa
        be = SDPBackend.FLASH_ATTENTION if backend == "flash" else SDPBackend.EFFICIENT_ATTENTION
        with sdpa_kernel([be]):
            o = F.scaled_dot_product_attention(Q.unsqueeze(1), K.unsqueeze(1), V.unsqueeze(1), scale=tau)
        o = o[:, 0].float()
        s = kappa * o[..., :C] / o[..., C:C + 1]
        (s * tg).sum().backward()
        return s.detach(), lq.grad

    ws = torch.empty(max(gs.gauss_sum_fwd_bwd_batched_workspace_size(M, N, D, C, B), 1),
                     dtype=torch.uint8, device=dev)
    out = torch.empty((B, M, C), dtype=torch.float32, device=dev)

    def library():
        s, dq, _, _ = gs.gauss_sum_fwd_bwd_batched(tq, tk, tv, tau, tg, out=out, workspace=ws,
                                                   stream=stream)
        return s, dq

    rows = wl.sample_rows(M, 256, seed=3)
    probs = tuple(sorted({0, B // 2, B - 1}))
    th = min(oracle.default_threads(), 16)
    ref_s = [oracle.fwd(q[b], k[b], v[b], tau, rows=rows, threads=th)[0] for b in probs]
    ref_dq = [oracle.dq(q[b], k[b], v[b], g[b], tau, rows=rows, threads=th)[0] for b in probs]

    def rel(got, refs):
        num = sum(float(np.sum((got[b][rows].astype(np.float64) - r) ** 2)) for b, r in zip(probs, refs))
        den = sum(float(np.sum(r ** 2)) for r in refs)
        return float(np.sqrt(num / den))

    def measure(fn):
        s, dq = fn()
        torch.cuda.synchronize()
        sh, dqh = s.float().cpu().numpy(), dq.float().cpu().numpy()
        acc = {}
        for key, got, refs in (("s", sh, ref_s), ("dq", dqh, ref_dq)):
            bad = float(np.mean(~np.isfinite(got)))
            acc["nonfinite_" + key] = bad   # fraction of non-finite outputs (fp16 overflow)
            acc["rel_l2_" + key] = rel(got, refs) if bad == 0.0 else None
        t0 = time.perf_counter()
        while (time.perf_counter() - t0) * 1e3 < args.settle_ms:
            fn()
            torch.cuda.synchronize()
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        return dict(ms_per_step=ms, pairs_per_s=B * float(M) * N / (ms * 1e-3), **acc)

    routes = {}
    for name, fn in (("gauss_sum_fwd_bwd_batched", library),
                     ("alg2_reweight_flash_autograd", lambda: reweight("flash")),
                     ("alg2_reweight_mem_efficient_autograd", lambda: reweight("efficient"))):
        print("route", name, flush=True, file=sys.stderr)
        try:
            torch.cuda.reset_peak_memory_stats()
            base = torch.cuda.memory_allocated()
            routes[name] = measure(fn)
            routes[name]["peak_mem_gib"] = (torch.cuda.max_memory_allocated() - base) / 2 ** 30
        except RuntimeError as e:  # a backend that does not take these shapes here
            routes[name] = {"error": str(e).splitlines()[0][:200]}
    lib_ms = routes["gauss_sum_fwd_bwd_batched"]["ms_per_step"]
    for r in routes.values():
        if "ms_per_step" in r:
            r["library_speedup"] = r["ms_per_step"] / lib_ms
    print(json.dumps({"mode": "compare_attention", "unit": "pairs/s", "data": "synthetic",
                      "config": {"workload": args.workload, "B": B, "M": M, "N": N, "D": D, "C": C,
                                 "tau": tau, "passes": "fwd+dq+dk+dv", "inputs": "f16 points, f32 values",
                                 "accuracy": "rel-L2 of s and dq vs fp64 oracle, %d rows of problems %s"
                                             % (len(rows), probs)},
                      "steps": args.steps, "warmup": args.warmup, "routes": routes}), flush=True)


def compare_attention(args):
    """The paper's route on this GPU, as an external comparison (it is not part
    of the library and nothing in the library calls it): Alg. 1 (prescale:
    fused attention with its log-sum-exp, values pre-multiplied by
    exp(-tau/2 |k|^2), output rescaled by exp(lse - tau/2 |q|^2)) and Alg. 2
    (reweight: queries and keys extended by two entries, one auxiliary key and
    value channel with kappa = sqrt(N + 1), output kappa alpha / beta), both
    through PyTorch's fused attention kernels (flash and memory-efficient
    backends) in the points' precision (fp16; fp32 for the single-precision
    workload, App. A.2, where only the memory-efficient backend takes fp32)
    with q and k shifted by their common mean and the widths padded to
    multiples of 8 (Sec. 2, Remark 1).  Forward sums of
    the batched workload; each route is timed like the library (settle,
    warm-up, timed steps between events) and checked against the fp64 oracle
    on sampled rows of three problems (relative L2 error).  Prints one JSON
    line."""
    import numpy as np
    import torch
    import torch.nn.functional as F
    from torch.nn.attention import SDPBackend, sdpa_kernel

    import oracle
    from paper_2609_04910_amd import gauss_sum as gs
    from paper_2609_04910_amd import workloads as wl

    dev = torch.device("cuda:0")
    q, k, v, tau = wl.make_batch(args.workload, seed=0)
    tau = float(tau)
    B, M, D = q.shape
    N, C = v.shape[1], v.shape[2]
    tq, tk, tv = (torch.from_numpy(a).to(dev) for a in (q, k, v))
    stream = torch.cuda.current_stream()
    ceil8 = lambda x: (x + 7) // 8 * 8
    pdt = tq.dtype  # the routes compute in the points' precision (fp16, or fp32 for App. A.2)

    def centred():
        mu = torch.cat([tq, tk], 1).float().mean(dim=1, keepdim=True)
        qc = (tq.float() - mu).to(pdt)
        kc = (tk.float() - mu).to(pdt)
        return qc, kc, qc.float().pow(2).sum(-1), kc.float().pow(2).sum(-1)

    def pad(x, width):
        return F.pad(x, (0, width - x.shape[-1]))

    def prescale(backend):
        qc, kc, nq, nk = centred()
        w = ceil8(max(D, C))
        vt = (tv * torch.exp(-0.5 * tau * nk).unsqueeze(-1)).to(pdt)
        Q, K, V = (pad(x, w).unsqueeze(1).contiguous() for x in (qc, kc, vt))
        if backend == "flash":
            r = torch.ops.aten._scaled_dot_product_flash_attention(Q, K, V, 0.0, False, False, scale=tau)
        else:
            r = torch.ops.aten._scaled_dot_product_efficient_attention(Q, K, V, None, True, 0.0, False,
                                                                       scale=tau)
        o, lse = r[0][:, 0, :, :C].float(), r[1][:, 0, :M].float()
        return o * torch.exp(lse - 0.5 * tau * nq).unsqueeze(-1)

    kappa = float(np.sqrt(N + 1))

    def reweight(backend):
        qc, kc, nq, nk = centred()
        w = ceil8(max(D + 2, C + 1))
        Q = torch.zeros((B, M, w), dtype=pdt, device=dev)
        Q[..., :D] = qc
        Q[..., D] = 1.0
        Q[..., D + 1] = (0.5 * nq).to(pdt)
        K = torch.zeros((B, N + 1, w), dtype=pdt, device=dev)
        K[:, 0, D + 1] = 1.0
        K[:, 1:, :D] = kc
        K[:, 1:, D] = (-0.5 * nk).to(pdt)
        V = torch.zeros((B, N + 1, w), dtype=pdt, device=dev)
        V[:, 1:, :C] = tv.to(pdt)
        V[:, 0, C] = kappa
        be = SDPBackend.FLASH_ATTENTION if backend == "flash" else SDPBackend.EFFICIENT_ATTENTION
        with sdpa_kernel([be]):
            o = F.scaled_dot_product_attention(Q.unsqueeze(1), K.unsqueeze(1), V.unsqueeze(1), scale=tau)
        o = o[:, 0].float()
        return kappa * o[..., :C] / o[..., C:C + 1]

    ws = torch.empty(max(gs.gauss_sum_fwd_batched_workspace_size(M, N, D, C, B), 1), dtype=torch.uint8,
                     device=dev)
    out = torch.empty((B, M, C), dtype=torch.float32, device=dev)

    def library():
        gs.gauss_sum_fwd_batched(tq, tk, tv, tau, out=out, workspace=ws, stream=stream)
        return out

    rows = wl.sample_rows(M, 512, seed=3)
    probs = tuple(sorted({0, B // 2, B - 1}))
    refs = [oracle.fwd(q[b], k[b], v[b], tau, rows=rows, threads=min(oracle.default_threads(), 16))[0]
            for b in probs]

    def measure(fn):
        res = fn()
        torch.cuda.synchronize()
        got = res.cpu().numpy()
        num = sum(float(np.sum((got[b][rows].astype(np.float64) - r) ** 2)) for b, r in zip(probs, refs))
        den = sum(float(np.sum(r ** 2)) for r in refs)
        t0 = time.perf_counter()
        while (time.perf_counter() - t0) * 1e3 < args.settle_ms:
            fn()
            torch.cuda.synchronize()
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        return {"ms_per_step": ms, "pairs_per_s": B * float(M) * N / (ms * 1e-3),
                "rel_l2": float(np.sqrt(num / den)), "peak_mem_gib": None}

    routes = {}
    for name, fn in (("gauss_sum_fwd_batched", library),
                     ("alg1_prescale_flash", lambda: prescale("flash")),
                     ("alg1_prescale_mem_efficient", lambda: prescale("efficient")),
                     ("alg2_reweight_flash", lambda: reweight("flash")),
                     ("alg2_reweight_mem_efficient", lambda: reweight("efficient"))):
        print("route", name, flush=True, file=sys.stderr)
        try:
            torch.cuda.reset_peak_memory_stats()
            base = torch.cuda.memory_allocated()
            routes[name] = measure(fn)
            routes[name]["peak_mem_gib"] = (torch.cuda.max_memory_allocated() - base) / 2 ** 30
        except RuntimeError as e:  # a backend that does not take these shapes here
            routes[name] = {"error": str(e).splitlines()[0][:200]}
    lib_ms = routes["gauss_sum_fwd_batched"]["ms_per_step"]
    for r in routes.values():
        if "ms_per_step" in r:
            r["library_speedup"] = r["ms_per_step"] / lib_ms
    print(json.dumps({"mode": "compare_attention", "unit": "pairs/s", "data": "synthetic",
                      "config": {"workload": args.workload, "B": B, "M": M, "N": N, "D": D, "C": C,
                                 "tau": tau, "passes": "fwd",
                                 "inputs": "%s points, f32 values" % ("f32" if pdt == torch.float32 else "f16"),
                                 "accuracy": "rel-L2 vs fp64 oracle, 512 rows of problems %s" % (probs,)},
                      "steps": args.steps, "warmup": args.warmup, "routes": routes}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--settle-ms", type=float, default=400.0,
                    help="untimed repetition of the step before the warm-up, for the steady clock")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="also run a device copy of MIB MiB (counter calibration for --traffic-from)")
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="record roofline traffic from two rocprofv3 --pmc csv outputs and exit")
    ap.add_argument("--workload", default="rect_d256", choices=sorted(PASSES) + ["batch_d32", "batch_d32_f32", "batch_c32", "batch_c32_f32", "batch_grad_d32"])
    ap.add_argument("--tau", type=float, default=None, help="mixture_d32 bandwidth (0.1, 1, 10)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-configs", action="store_true",
                    help="rect_d256: time the headline workload only (no records of the other configurations)")
    ap.add_argument("--cpu-budget", type=float, default=15.0)
    ap.add_argument("--flow", action="store_true",
                    help="mmd_flow: time one gauss_sum_mmd_flow call per step (s, the flow field "
                         "and MMD^2 = v^T s) instead of gauss_sum_fwd_bwd")
    ap.add_argument("--compare-attention", action="store_true",
                    help="batched workloads: time the paper's attention route (Alg. 1 and 2 through "
                         "PyTorch's fused attention; for batch_grad_d32 forward and backward through "
                         "Alg. 2 with autograd) beside the library")
    ap.add_argument("--batch-n", type=int, default=None, metavar="N",
                    help="--compare-attention on batch_grad_d32: M = N = this instead of 65536")
    ap.add_argument("--graph", action="store_true",
                    help="time the step captured in a HIP graph and replayed (the kernel roofline "
                         "still comes from the eager steps)")
    ap.add_argument("--peaks", action="store_true",
                    help="measure the device's MFMA, exp2, FMA and streaming-read rates and exit")
    ap.add_argument("--svgd-update", action="store_true",
                    help="time gauss_sum_svgd (one SVGD direction per step) on the svgd workload's "
                         "particles and score-like values")
    ap.add_argument("--separate", action="store_true",
                    help="time separate gauss_sum_fwd + gauss_sum_bwd calls instead of one "
                         "gauss_sum_fwd_bwd call")
    args = ap.parse_args()
    if args.traffic_from:
        traffic_from(args.workload, args.traffic_from[0], args.traffic_from[1],
                     args.calibrate_copy * 1024 * 1024, dominant_kernel_name(args.workload))
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
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
    if args.peaks:
        bench_peaks(args)
        return
    if args.svgd_update:
        bench_svgd_update(args)
        return
    if args.compare_attention:
        if args.workload not in wl.BATCHED:
            print("--compare-attention takes a batched workload (--workload batch_d32)", file=sys.stderr)
            sys.exit(2)
        if wl.BATCHED[args.workload].get("grad"):
            compare_attention_grad(args)
        else:
            compare_attention(args)
        return
    if args.workload in wl.BATCHED:
        if wl.BATCHED[args.workload].get("grad"):
            bench_batched_grad(args)
        else:
            bench_batched(args)
        return

    if args.workload == "rect_d256" and not args.no_configs and not (args.flow or args.graph or args.separate):
        bench_headline(args)
        return
    res = measure_workload(args, args.workload, args.tau if args.workload == "mixture_d32" else None,
                           args.steps, args.warmup, args.settle_ms, graph=args.graph, flow=args.flow,
                           separate=args.separate, calibrate_copy=args.calibrate_copy)
    if not args.no_cpu:
        res["cpu_baseline"] = cpu_baseline(res.pop("_workload"), res.pop("_passes"), args.cpu_budget)
    print(json.dumps(clean(res)), flush=True)

if __name__ == "__main__":
    main()
