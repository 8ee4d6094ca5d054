#!/usr/bin/env python3
"""Benchmark: one GPU's share of the phase-owned MoE layer, P and D concurrent.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 1]

A step is one pass of the whole layer (route, dispatch, grouped SwiGLU FFN,
combine) for the prefill batch on one stream and, concurrently, for the
decode batch on a second stream.  Inputs (weights, hidden rows, logits) are
seeded synthetic tensors resident in HBM before timing starts.  Prints one
JSON line with:

* value: whole-job layer throughput, (T_P + T_D) * K / wall time of K steps;
* d_latency_us: the D layer's GPU latency (events on the D stream) alone
  (back to back; alone_cold: after clearing the memory-side cache) and while
  P layers keep the other stream busy, p50/p90/p99; graph_*: the same with
  the D layer captured once into a HIP graph and replayed;
* roofline: the kernel with the largest share of GPU time, its algorithmic
  bytes or flops per launch over its mean launch duration, against the MI355X
  peak that bounds it.  Durations come from HIP events recorded around every
  kernel on the stream it runs on, over a second pass of the same K timed
  steps (the events themselves cost stream time, so the throughput pass runs
  without them) with D-first admission off, so that a P kernel's duration is
  its own work and not the waits the admission policy puts in it;
  roofline_phase_alone: the same kernel timed over K layers of its phase
  alone, with no layer of the other phase beside it;
* D-first admission (--d-priority-us, default 500): while a D layer is in
  flight, P grouped-GEMM tiles wait for it (at tile starts and every few K
  slices), up to that bound per tile; value and d_latency_us are measured
  with it, without_d_first repeats both without;
* engine_clock_mhz: the shader clock, idle and beside P layers (the peaks
  stay the datasheet's);
* kernels: mean launch duration of every kernel of both phases;
* cpu_baseline: the CPU oracle timed on this host on a bounded, seeded sample
  of the same workload (a subset of each phase's tokens, at most 4096 P
  tokens and the same fraction of the D batch; the whole batch when it is
  smaller), its P pass timed stage by stage and, for the small configs, one
  thread; cores = the BLAS threads it ran with (the host's CPU share, at most
  the CPUs this process may run on, which are reported beside it).
"""

from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16 matrix-core peak, TFLOP/s
MFMA_FP8_PEAK_TFLOPS = 5000.0  # dense fp8 matrix-core peak, TFLOP/s
FP32_VECTOR_PEAK_TFLOPS = 157.3

METRIC = "MoE-layer tokens/s (P+D concurrent, 1 GPU); D-layer p50 latency under P load"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=3,
                    help="workload id (0..7); 3 (the skewed DeepSeek-V3-shaped share, the largest one-GPU workload) "
                         "is the headline, 4 the agentic trace on the config-2 layer, 5 the config-2 layer in MX FP8, "
                         "6/7 the paper's model shape in FP8/BF16")
    ap.add_argument("--trace-steps", type=int, default=200, help="steps of the agentic trace (config 4)")
    ap.add_argument("--d-iters", type=int, default=200,
                    help="D layers per latency measurement (enough to span some twenty P layers under P)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="least time of the CPU-oracle sample")
    ap.add_argument("--cpu-tokens", type=int, default=4096, help="P tokens in the CPU-oracle sample (at most)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--seg-layers", type=int, default=40,
                    help="MoE layers per P epoch and per D iteration in the segment-policy sweep (0: skip it)")
    ap.add_argument("--seg-epochs", type=int, default=2, help="P epochs per policy in the segment-policy sweep")
    ap.add_argument("--no-router", action="store_true", help="skip the router-GEMM timing")
    ap.add_argument("--d-priority-us", type=int, default=500,
                    help="D-first admission: longest wait of a P GEMM tile for an in-flight D layer (0 = off)")
    ap.add_argument("--solo", choices=("P", "D"), default=None,
                    help="instead of the concurrent bench, run only this phase's layer back to back and report its "
                         "per-kernel durations (for kernel profiles; prints a line of its own, not the headline)")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="instead of the layer, time a plain device copy of this many MiB (the reference kernel "
                         "for scaling the HBM byte counters)")
    return ap.parse_args()


def pct(vals, q):
    s = sorted(vals)
    if not s:
        return None
    i = min(len(s) - 1, max(0, int(math.ceil(q / 100.0 * len(s))) - 1))
    return s[i]


def workload_name(spec):
    skew = (f", router biased to Zipf({spec.zipf_s}) slot shares capped at 1/{spec.k}" if spec.zipf_s else "")
    return (f"{spec.name}: E={spec.E} (resident {spec.E_loc} from e0={spec.e0}) top-{spec.k} H={spec.H} I={spec.I} "
            f"SwiGLU {spec.dtype}{skew}, P {spec.T_P} + D {spec.T_D} tokens concurrent on two streams")


def kernel_units(spec, kernel, T, R, touched, esz, osz=None, t_res=None):
    """(algorithmic bytes, algorithmic flops) of one launch of `kernel` for a
    phase batch of T tokens with R resident rows over `touched` experts, t_res
    of the tokens having a resident slot.  esz: bytes of an x element; osz:
    bytes per element of the GEMM operands (weights, x_perm, h), scales
    included (1 + 1/32 for MX FP8)."""
    H, I, E, k = spec.H, spec.I, spec.E, spec.k
    osz = esz if osz is None else osz
    t_res = T if t_res is None else t_res
    if kernel == "route":
        return T * E * 4 + T * k * 8, 0
    if kernel in ("count", "place"):
        return T * k * 4 * (1 if kernel == "count" else 2) + R * 4, 0
    if kernel == "permute":
        # the rows of the tokens with a resident slot are read once (the
        # others are skipped), each resident row written once
        return int(t_res * H * esz + R * H * osz), 0
    if kernel == "gemm1_swiglu":
        return int(touched * 2 * I * H * osz + R * H * osz + R * I * osz), 4 * R * H * I
    if kernel == "gemm2_down":
        return int(touched * H * I * osz + R * I * osz + R * H * 4), 2 * R * H * I
    if kernel == "combine":
        return R * H * 4 + T * H * 4 + T * k * 8, 0
    return 0, 0


def recorded_traffic(cfg, phase, kernel, lib_path=None):
    """HBM bytes per launch of one kernel from the committed rocprofv3 counter
    record (FETCH_SIZE + WRITE_SIZE, each scaled by a plain copy's reading),
    or None when no record exists or the kernels differ from the profiled
    ones: the record holds for the library file it was taken with (lib_path,
    the library this process loaded) and for the kernel sources it was taken
    on."""
    import hashlib

    def sha(p):
        return hashlib.sha256(open(p, "rb").read()).hexdigest()

    path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    try:
        rec = json.load(open(path))
        same_lib = bool(lib_path) and os.path.exists(lib_path) and rec.get("library_sha256") == sha(lib_path)
        if not same_lib:
            for rel, digest in rec["sources"].items():
                if sha(os.path.join(ROOT, rel)) != digest:
                    return None
        return rec["workloads"][f"cfg{cfg}"][f"{'P' if phase == 0 else 'D'}.{kernel}"]["hbm_bytes"]
    except (OSError, KeyError, ValueError):
        return None


def cpu_threads():
    """BLAS threads for the CPU oracle: the host's CPU share (OMP_NUM_THREADS,
    else 16), never more than the CPUs this process may run on."""
    affinity = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    try:
        share = int(os.environ.get("OMP_NUM_THREADS", "16"))
    except ValueError:
        share = 16
    return max(1, min(affinity, share)), affinity


def cpu_baseline(inp, seconds, max_p_tokens):
    """The oracle as it stands, timed on a seeded sample of the workload's
    tokens: each phase's sub-batch runs the whole layer (route, layout,
    permute, expert FFN, combine); a token's output depends on no other
    token, so the sample is the same work per token as the full batch.
    Passes repeat until `seconds` have elapsed (at least one)."""
    import numpy as np

    import oracle

    spec = inp.spec
    threads, affinity = cpu_threads()
    try:
        from threadpoolctl import threadpool_limits
    except Exception:  # pragma: no cover - threadpoolctl is optional
        threadpool_limits = None
    rng = np.random.default_rng(7)
    T = {0: spec.T_P, 1: spec.T_D}
    n_p = min(T[0], max_p_tokens)
    n = {0: n_p, 1: min(T[1], max(1, round(T[1] * n_p / max(T[0], 1))))}
    toks = {ph: np.sort(rng.choice(T[ph], size=n[ph], replace=False)) for ph in (0, 1)}
    fp8 = inp.w_gu_scales is not None
    if fp8:
        from oracle import mx as oracle_mx

    stages = {}

    def one_pass(ph):
        lg, x = inp.logits[ph][toks[ph]], inp.x[ph][toks[ph]]
        if fp8:
            oracle_mx.layer_mx(lg, x, inp.w_gu_bits, inp.w_gu_scales, inp.w_dn_bits, inp.w_dn_scales, spec.k, spec.e0)
            return
        # oracle.layer's steps, each timed (the P pass's times are reported)
        st = {}
        t = time.perf_counter()
        idx, w = oracle.route(lg, spec.k)
        st["route"] = time.perf_counter() - t
        t = time.perf_counter()
        le = oracle.local_map(idx, spec.e0, spec.E_loc)
        counts, offsets, ros, tor = oracle.layout(le, spec.E_loc)
        st["layout"] = time.perf_counter() - t
        t = time.perf_counter()
        xp = oracle.permute(x, tor)
        st["permute"] = time.perf_counter() - t
        t = time.perf_counter()
        _, y = oracle.expert_ffn(xp, offsets, inp.w_gu, inp.w_dn)
        st["ffn"] = time.perf_counter() - t
        t = time.perf_counter()
        oracle.combine(y, w, ros, n[ph], spec.H)
        st["combine"] = time.perf_counter() - t
        if ph == 0 and not stages:
            stages.update(st)

    import contextlib

    limit = threadpool_limits(threads) if threadpool_limits is not None else contextlib.nullcontext()
    with limit:
        tokens, reps = 0, 0
        t0 = time.perf_counter()
        while True:
            for ph in (0, 1):
                if n[ph]:
                    one_pass(ph)
                    tokens += n[ph]
            reps += 1
            el = time.perf_counter() - t0
            if el >= seconds or reps >= 50:
                break
    res = {
        "value": tokens / el,
        "unit": "tokens/s",
        "cores": int(threads),
        "affinity_cpus": int(affinity),
        "kind": "oracle",
        "sample": f"{reps} pass(es) of the float64 numpy oracle{' (MX FP8)' if fp8 else ''} over a seeded sample "
                  f"of {n[0]} of the {T[0]} P tokens and {n[1]} of the {T[1]} D tokens of the same workload "
                  f"(the whole layer per sub-batch), {el:.1f} s on {threads} BLAS threads",
    }
    if stages:
        res["p_pass_stages_s"] = {kk: round(v, 4) for kk, v in stages.items()}
    if threadpool_limits is not None and not fp8 and spec.T_P * spec.H * spec.I <= 2048 * 2048 * 1024:
        with threadpool_limits(1):
            t = time.perf_counter()
            for ph in (0, 1):
                oracle.layer(inp.logits[ph], inp.x[ph], inp.w_gu, inp.w_dn, spec.k, spec.e0)
            res["one_thread_tokens_per_s"] = (spec.T_P + spec.T_D) / (time.perf_counter() - t)
    return res


def copy_calibration(args):
    """A plain device-to-device copy of known size (reads and writes
    copy_mib MiB each launch), timed with events on its stream."""
    import torch

    n = args.copy_mib * (1 << 20) // 4
    src = torch.randn(n, device="cuda")
    dst = torch.empty_like(src)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        for _ in range(max(1, args.warmup)):
            dst.copy_(src)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(s)
        for _ in range(args.steps):
            dst.copy_(src)
        b.record(s)
    torch.cuda.synchronize()
    us = a.elapsed_time(b) * 1e3 / args.steps
    by = 2 * n * 4
    print(json.dumps({"mode": "copy", "bytes_read": n * 4, "bytes_written": n * 4, "mean_us": round(us, 2),
                      "GB/s": round(by / (us * 1e-6) / 1e9, 1), "launches": args.steps + max(1, args.warmup)}))


def run_trace(args, M, inp, dev):
    """The agentic rollout trace on the config-2 layer: per step, a D batch on
    the D stream (the host waits for it, as a decode iteration needs its
    output before the next) and, when the step has one, a continuation-prefill
    P batch on the P stream, which runs on asynchronously.  Batches are
    windows of the resident token pools.  Reports the per-step D latency
    distribution (events on the D stream) and total tokens/s."""
    import numpy as np
    import torch

    from synth import agentic_trace

    spec = inp.spec
    trace = agentic_trace(steps=args.trace_steps)

    def up(a):
        a = np.ascontiguousarray(a)
        return torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).to(dev)

    w_gu, w_dn = up(inp.w_gu_bits), up(inp.w_dn_bits)
    xs = {ph: up(inp.x_bits[ph]) for ph in (0, 1)}
    lg = {ph: up(inp.logits[ph]) for ph in (0, 1)}
    outs = {ph: torch.empty(((spec.T_P, spec.T_D)[ph], spec.H), dtype=torch.float32, device=dev) for ph in (0, 1)}

    def make_ctx(us):
        cfg = M.make_config(spec.E, spec.e0, spec.E_loc, spec.k, spec.H, spec.I, M.MOE_DTYPE_BF16, spec.T_P, spec.T_D,
                            d_priority_us=us)
        st, c = M.moe_ctx_create(cfg, w_gu, w_dn)
        M.check(st, "moe_ctx_create")
        return c

    ctx = make_ctx(args.d_priority_us)
    ctx_off = make_ctx(0) if args.d_priority_us > 0 else ctx
    sP, sD = torch.cuda.Stream(device=dev), torch.cuda.Stream(device=dev)

    def win(ph, off, T):
        return lg[ph][off:off + T], xs[ph][off:off + T], outs[ph][off:off + T]

    def play(c, with_p, units=None):
        """Run the trace once; returns (wall s, D latencies us)."""
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in trace]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i, st in enumerate(trace):
            if with_p and st.t_p:
                l, x, o = win(0, st.p_off, st.t_p)
                M.layer(c, 0, l, st.t_p, x, o, sP)
            a, b = evs[i]
            l, x, o = win(1, st.d_off, st.t_d)
            a.record(sD)
            M.layer(c, 1, l, st.t_d, x, o, sD)
            b.record(sD)
            sD.synchronize()
            if units is not None:
                units(st, with_p)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        return wall, [a.elapsed_time(b) * 1000.0 for a, b in evs]

    play(ctx, True)  # warmup: every batch size once
    wall, lat_under = play(ctx, True)
    _, lat_alone = play(ctx, False)
    wall_off, lat_under_off = play(ctx_off, True) if ctx_off is not ctx else (wall, lat_under)
    tokens = sum(st.t_d + st.t_p for st in trace)

    # per-kernel events (D-first admission off), with each step's rows and
    # touched experts read back for the algorithmic units
    acc_units = {}

    def units(st, with_p):
        torch.cuda.synchronize()
        for ph, T in ((0, st.t_p), (1, st.t_d)):
            if T == 0 or (ph == 0 and not with_p):
                continue
            R, touched, t_res = layout_counts(M, ctx_off, ph, spec)
            for name in ("route", "count", "place", "permute", "gemm1_swiglu", "gemm2_down", "combine"):
                by, fl = kernel_units(spec, name, T, R, touched, 2, None, t_res)
                b0, f0 = acc_units.get((ph, name), (0, 0))
                acc_units[(ph, name)] = (b0 + by, f0 + fl)

    M.check(M.moe_timing_enable(ctx_off, len(trace)), "moe_timing_enable")
    play(ctx_off, True, units)
    kern = {}
    for ph in (0, 1):
        for kid in range(M.MOE_NUM_KERNELS):
            st_, ms, n = M.moe_timing_read(ctx_off, ph, kid)
            M.check(st_)
            if n:
                kern[(ph, M.moe_kernel_name(kid))] = (ms, n)
    M.check(M.moe_timing_enable(ctx_off, 0))
    dom = max(kern, key=lambda key: kern[key][0])
    ms_d, n_d = kern[dom]
    by, fl = acc_units[dom]
    t_s = ms_d / 1e3
    if fl and fl / (MFMA_BF16_PEAK_TFLOPS * 1e12) >= by / (HBM_PEAK_GBS * 1e9):
        ach = fl / t_s / 1e12
        roof = {"bound": "mfma", "achieved": round(ach, 2), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s"}
    else:
        ach = by / t_s / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s"}
    roof["frac"] = round(ach / roof["peak"], 4)
    roof["traffic"] = None
    roof["kernel"] = f"{dom[1]} ({'P' if dom[0] == 0 else 'D'})"
    roof["per_launch"] = {"bytes": by // n_d, "flops": fl // n_d, "mean_us": round(ms_d / n_d * 1e3, 2),
                          "launches": n_d, "note": "trace totals over launches (batch sizes vary)"}
    kernels = {}
    for (ph, name), (ms, n) in sorted(kern.items()):
        b_, f_ = acc_units.get((ph, name), (0, 0))
        kernels[f"{'P' if ph == 0 else 'D'}.{name}"] = {
            "mean_us": round(ms / n * 1e3, 2),
            "GB/s": round(b_ / (ms / 1e3) / 1e9, 1) if b_ else None,
            "TFLOP/s": round(f_ / (ms / 1e3) / 1e12, 1) if f_ else None,
        }
    n_p = sum(1 for st in trace if st.t_p)
    p50a, p50u = pct(lat_alone, 50), pct(lat_under, 50)
    res = {
        "metric": METRIC,
        "value": round(tokens / wall, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": len(trace),
        "warmup": 1,
        "ms_per_step": round(wall / len(trace) * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{spec.name}: config-2 layer (E={spec.E}, resident {spec.E_loc}, top-{spec.k}, "
                               f"H={spec.H}, I={spec.I}, bf16) under a seeded {len(trace)}-step agentic trace: "
                               f"D U{{32..256}} tokens per step, P log-uniform 512..16384 with p=0.5 on a second stream",
                   "steps_with_p": n_p, "tokens": tokens, "parallelism": "single GPU, P and D on two streams",
                   "d_priority_us": args.d_priority_us},
        "d_latency_us": {
            "p50_alone": round(p50a, 2), "p90_alone": round(pct(lat_alone, 90), 2),
            "p50_under_p": round(p50u, 2), "p90_under_p": round(pct(lat_under, 90), 2),
            "p99_under_p": round(pct(lat_under, 99), 2), "max_under_p": round(max(lat_under), 2),
            "ratio_p50": round(p50u / p50a, 3), "iters": len(trace),
            "note": "per-step D layer latency; alone = the same D steps with no P batches",
        },
        "roofline": roof,
        "kernels": kernels,
        "kernels_pass_note": "per-kernel HIP events over a replay of the trace with D-first admission off",
        "without_d_first": {
            "value": round(tokens / wall_off, 1),
            "ms_per_step": round(wall_off / len(trace) * 1e3, 4),
            "d_p50_under_p_us": round(pct(lat_under_off, 50), 2),
            "d_p90_under_p_us": round(pct(lat_under_off, 90), 2),
            "ratio_p50": round(pct(lat_under_off, 50) / p50a, 3),
        },
    }
    M.check(M.moe_ctx_destroy(ctx))
    if ctx_off is not ctx:
        M.check(M.moe_ctx_destroy(ctx_off))
    print(json.dumps(res), flush=True)


def segment_sweep(args, M, c, lg, xs, T, spec, sP, dev):
    """P epochs of `seg_layers` layers run by the native P-epoch runner through
    the segment turnstile while D iterations (`seg_layers` D layers captured
    into one HIP graph) run back to back, a D iteration being ready as soon
    as the previous one has completed.  Policies (Section 7's ordering
    ladder and Section 7.6's segment sizes): D waits for P's GPU completion
    (complete), for the whole epoch's host enqueue (enqueue), or for the next
    permitted boundary with span K = 1..4 (fine-K).  Reports, per policy, D's
    boundary wait and iteration latency, P's wait for permits and host
    enqueue time, and the P epoch's makespan (start to GPU completion)."""
    import torch

    L = args.seg_layers
    sg = torch.cuda.Stream(device=dev)
    d_out = torch.empty((T[1], spec.H), dtype=torch.float32, device=dev)
    p_out = torch.empty((T[0], spec.H), dtype=torch.float32, device=dev)
    torch.cuda.synchronize()
    M.layer(c, 1, lg[1], T[1], xs[1], d_out, sg)  # the D phase last ran on the capture stream
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=sg):
        for _ in range(L):
            M.layer(c, 1, lg[1], T[1], xs[1], d_out, sg)
    torch.cuda.synchronize()

    def d_iteration():
        with torch.cuda.stream(sg):
            start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            start.record(sg)
            graph.replay()
            end.record(sg)
        return start, end

    alone = []
    for _ in range(5):
        start, end = d_iteration()
        end.synchronize()
        alone.append(start.elapsed_time(end) * 1e3)
    p_alone = []
    for _ in range(2):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(L):
            M.layer(c, 0, lg[0], T[0], xs[0], p_out, sP)
        sP.synchronize()
        p_alone.append((time.perf_counter() - t0) * 1e6)

    # D latency of an iteration = its boundary wait (host, from the moment the
    # previous iteration completed) + its GPU span (events around the replay).
    # P's epoch span is taken on the P stream, from an event enqueued before
    # the runner starts to one enqueued after it has finished.
    policies = [("complete", L + 1), ("enqueue", L + 1)] + [(f"fine-{k}", k) for k in (1, 2, 3, 4)]
    out = {}
    epoch = 0
    for name, K in policies:
        st, ts = M.moe_turnstile_create(K, 0)
        M.check(st, "moe_turnstile_create")
        waits, iters, marks, p_wait, p_enq, rounds = [], [], [], [], [], []
        torch.cuda.synchronize()
        t_policy = time.perf_counter()
        prev = d_iteration()
        try:
            for _ in range(args.seg_epochs):
                p_start = torch.cuda.Event(enable_timing=True)
                p_start.record(sP)
                st, runner = M.moe_p_epoch_start(c, ts, epoch, True, T[0], [lg[0]] * L, [xs[0]] * L, [p_out] * L, sP,
                                                 60_000_000)
                M.check(st, "moe_p_epoch_start")
                epoch += 1
                joined = None
                while True:
                    prev[1].synchronize()  # D is ready once its previous iteration has completed
                    t_ready = time.perf_counter()
                    M.check(M.moe_turnstile_wait_boundary(ts, 60_000_000), "wait_boundary")
                    done = M.moe_turnstile_query(ts)[1].task == M.MOE_TS_DONE
                    if done:
                        joined = M.moe_p_epoch_join(runner)
                        if name == "complete":
                            sP.synchronize()
                    waits.append((time.perf_counter() - t_ready) * 1e6)
                    prev = d_iteration()
                    iters.append(prev)
                    M.check(M.moe_turnstile_release(ts))
                    if done:
                        break
                st, stats = joined
                M.check(st, "P epoch")
                p_end = torch.cuda.Event(enable_timing=True)
                p_end.record(sP)
                marks.append((p_start, p_end))
                rounds.append(M.moe_turnstile_query(ts)[1].rounds)
                p_wait.append(stats.wait_us)
                p_enq.append(stats.enqueue_us)
            # D keeps iterating while the last epoch's P work drains
            while not marks[-1][1].query():
                prev[1].synchronize()
                t_ready = time.perf_counter()
                M.check(M.moe_turnstile_wait_boundary(ts, 60_000_000), "wait_boundary")
                waits.append((time.perf_counter() - t_ready) * 1e6)
                prev = d_iteration()
                iters.append(prev)
                M.check(M.moe_turnstile_release(ts))
            torch.cuda.synchronize()
            wall = time.perf_counter() - t_policy
        finally:
            M.moe_turnstile_destroy(ts)
        lats = [w + a.elapsed_time(b) * 1e3 for w, (a, b) in zip(waits, iters)]
        spans = [a.elapsed_time(b) for a, b in marks]
        out[name] = {
            "span": K if name.startswith("fine") else None,
            "d_wait_us_mean": round(sum(waits) / len(waits), 1), "d_wait_us_p99": round(pct(waits, 99), 1),
            "d_iter_us_p50": round(pct(lats, 50), 1), "d_iter_us_p99": round(pct(lats, 99), 1),
            "d_iters": len(waits),
            "p_epoch_ms": round(sum(spans) / len(spans), 3),
            "p_wait_for_permit_ms": round(sum(p_wait) / len(p_wait) / 1e3, 3),
            "p_enqueue_ms": round(sum(p_enq) / len(p_enq) / 1e3, 3),
            "rounds_per_epoch": sum(rounds) / len(rounds),
            "wall_ms": round(wall * 1e3, 2),
            "p_layer_tokens_per_s": round(T[0] * L * args.seg_epochs / wall, 1),
            "d_layer_tokens_per_s": round(T[1] * L * len(waits) / wall, 1),
        }
        print(f"# segments {name}: {out[name]}", file=sys.stderr, flush=True)
    del graph
    torch.cuda.synchronize()
    return {"layers": L, "epochs_per_policy": args.seg_epochs, "d_iter_alone_us_p50": round(pct(alone, 50), 1),
            "p_epoch_alone_ms": round(min(p_alone) / 1e3, 3), "policies": out,
            "note": "one P epoch = L layers of the P batch (one boundary per layer, after its dispatch layout), "
                    "epochs back to back; one D iteration = L layers of the D batch replayed as one HIP graph, ready "
                    "when the previous one completes, iterating until the last epoch's P work has drained; D-first "
                    "admission as in the bench line; rates count tokens through one layer"}


def router_measure(M, c, xs, T, spec, inp, sP, sD, bf16, reps=20):
    """The fused router GEMM (moe_route_from_hidden) of each phase, timed with
    the per-kernel events: x Wr^T on the matrix cores (float32 partial
    products over K runs), then the top-k kernel that sums the runs.  Units:
    2 T E H flops; x (T H) and Wr (E H) in the operand dtype as bytes."""
    import numpy as np
    import torch

    from synth import f32_to_bf16_bits

    wt = np.ascontiguousarray(inp.wg.T)
    w = torch.from_numpy(f32_to_bf16_bits(wt).view(np.int16) if bf16 else wt).to(xs[0].device)
    esz = 2 if bf16 else 4
    out = {}
    streams = {0: sP, 1: sD}
    M.check(M.moe_timing_enable(c, reps))
    for ph in (0, 1):
        for i in range(reps + 2):
            M.check(M.moe_route_from_hidden(c, ph, xs[ph], w, None, T[ph], streams[ph]), "moe_route_from_hidden")
            streams[ph].synchronize()
            M.check(M.moe_phase_reset(c, ph))
            if i == 1:  # the first two calls are warm-up
                for kid in range(M.MOE_NUM_KERNELS):
                    M.moe_timing_read(c, ph, kid)
        st, ms_g, n_g = M.moe_timing_read(c, ph, M.MOE_KERNEL_ROUTER)
        st, ms_r, n_r = M.moe_timing_read(c, ph, M.MOE_KERNEL_ROUTE)
        us_g, us_r = ms_g / max(n_g, 1) * 1e3, ms_r / max(n_r, 1) * 1e3
        fl = 2.0 * T[ph] * spec.E * spec.H
        by = (T[ph] + spec.E) * spec.H * esz
        out["P" if ph == 0 else "D"] = {
            "tokens": T[ph], "router_gemm_us": round(us_g, 2), "topk_us": round(us_r, 2),
            "TFLOP/s": round(fl / (us_g * 1e-6) / 1e12, 1), "operand_GB/s": round(by / (us_g * 1e-6) / 1e9, 1)}
    M.check(M.moe_timing_enable(c, 0))
    return out


def layout_counts(M, c, ph, spec):
    """Routed rows, touched experts and tokens with a resident slot of the
    phase's latest layout (read from the device once)."""
    import ctypes

    import torch

    st, v = M.moe_phase_view(c, ph)
    M.check(st)
    counts = torch.empty(spec.E_loc, dtype=torch.int32)
    ros = torch.empty((max(v.tokens, 1), spec.k), dtype=torch.int32)
    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
    assert hip.hipMemcpy(counts.data_ptr(), v.counts, spec.E_loc * 4, 2) == 0
    if v.tokens:
        assert hip.hipMemcpy(ros.data_ptr(), v.row_of_slot, v.tokens * spec.k * 4, 2) == 0
    t_res = int((ros[:v.tokens] >= 0).any(dim=1).sum()) if v.tokens else 0
    return int(counts.sum()), int((counts > 0).sum()), t_res


def solo_run(args, M, c, ph, layer, spec, T, esz, osz):
    """One phase alone: `steps` layers back to back on its stream, timed as a
    whole and then again with per-kernel HIP events."""
    import torch

    for _ in range(max(1, args.warmup)):
        layer(ph, c)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        layer(ph, c)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    M.check(M.moe_timing_enable(c, args.steps), "moe_timing_enable")
    for _ in range(args.steps):
        layer(ph, c)
    torch.cuda.synchronize()
    R, touched, t_res = layout_counts(M, c, ph, spec)
    kernels = {}
    for kid in range(M.MOE_NUM_KERNELS):
        st, ms, n = M.moe_timing_read(c, ph, kid)
        M.check(st)
        if not n:
            continue
        name = M.moe_kernel_name(kid)
        by, fl = kernel_units(spec, name, T, R, touched, esz, osz, t_res)
        us = ms / n * 1e3
        kernels[name] = {"mean_us": round(us, 2), "launches": n,
                         "GB/s": round(by / (us * 1e-6) / 1e9, 1) if by else None,
                         "TFLOP/s": round(fl / (us * 1e-6) / 1e12, 1) if fl else None}
    M.check(M.moe_timing_enable(c, 0))
    print(json.dumps({"solo": args.solo, "workload": workload_name(spec), "tokens": T, "tokens_resident": t_res,
                      "rows": R,
                      "touched_experts": touched, "steps": args.steps, "warmup": args.warmup,
                      "ms_per_layer": round(wall / args.steps * 1e3, 4),
                      "tokens_per_s": round(T * args.steps / wall, 1), "kernels": kernels,
                      "note": "one phase alone, D-first admission off; kernels: per-kernel HIP events on the phase's "
                              "stream over a second pass, algorithmic bytes and flops per launch"}), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the library runs the layer on a single "
              f"MI355X and has no multi-GPU step.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2609_00993_amd import moepd as M
    from synth import BF16, FP8, make_config

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.copy_mib:
        copy_calibration(args)
        return
    dev = torch.device("cuda:0")
    inp = make_config(args.config)
    if args.config == 4:
        run_trace(args, M, inp, dev)
        return
    spec = inp.spec
    bf16 = spec.dtype == BF16
    fp8 = spec.dtype == FP8
    packed = bf16 or fp8
    esz = 2 if packed else 4  # bytes of an x element
    osz = 1 + 1 / 32 if fp8 else esz  # bytes per GEMM operand element, scales included
    mma_peak = MFMA_FP8_PEAK_TFLOPS if fp8 else MFMA_BF16_PEAK_TFLOPS

    def up(a):
        a = np.ascontiguousarray(a)
        return torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).to(dev)

    w_gu = up(inp.w_gu_bits if packed else inp.w_gu)
    w_dn = up(inp.w_dn_bits if packed else inp.w_dn)
    w_gu_s = up(inp.w_gu_scales) if fp8 else None
    w_dn_s = up(inp.w_dn_scales) if fp8 else None
    xs = {ph: up(inp.x_bits[ph] if packed else inp.x[ph]) for ph in (0, 1)}
    lg = {ph: up(inp.logits[ph]) for ph in (0, 1)}
    T = {0: spec.T_P, 1: spec.T_D}
    outs = {ph: torch.empty((T[ph], spec.H), dtype=torch.float32, device=dev) for ph in (0, 1)}
    def make_ctx(d_priority_us):
        cfg = M.make_config(spec.E, spec.e0, spec.E_loc, spec.k, spec.H, spec.I,
                            M.MOE_DTYPE_FP8 if fp8 else M.MOE_DTYPE_BF16 if bf16 else M.MOE_DTYPE_F32, T[0], T[1],
                            d_priority_us=d_priority_us)
        st, c = M.moe_ctx_create(cfg, w_gu, w_dn, w_gu_s, w_dn_s)
        M.check(st, "moe_ctx_create")
        return c

    if args.solo:
        sS = torch.cuda.Stream(device=dev)
        c = make_ctx(0)
        ph = 0 if args.solo == "P" else 1
        solo_run(args, M, c, ph, lambda p, cc: M.layer(cc, p, lg[p], T[p], xs[p], outs[p], sS), spec, T[ph], esz,
                 osz)
        M.check(M.moe_ctx_destroy(c))
        return

    # The bench line runs at the D-first admission bound given (ctx); the same
    # layer without it (ctx_off) gives the comparison figures and the
    # per-kernel durations, which must not include P's deliberate waits.
    ctx = make_ctx(args.d_priority_us)
    ctx_off = make_ctx(0) if args.d_priority_us > 0 else ctx
    sP, sD = torch.cuda.Stream(device=dev), torch.cuda.Stream(device=dev)
    streams = {0: sP, 1: sD}

    def layer(ph, c=None):
        M.layer(ctx if c is None else c, ph, lg[ph], T[ph], xs[ph], outs[ph], streams[ph])

    # ---- warmup
    for c in {ctx, ctx_off}:
        for _ in range(max(1, args.warmup)):
            layer(0, c)
            layer(1, c)
    torch.cuda.synchronize()

    # ---- timed concurrent steps: throughput (no per-kernel events, which
    # would add a stream command around every kernel)
    def timed_steps(c):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            layer(0, c)
            layer(1, c)
        torch.cuda.synchronize()
        return time.perf_counter() - t0

    wall = timed_steps(ctx)
    wall_off = timed_steps(ctx_off) if ctx_off is not ctx else wall

    # ---- the same K concurrent steps again with per-kernel HIP events on the
    # launching streams (D-first admission off): per-kernel durations for the
    # roofline
    M.check(M.moe_timing_enable(ctx_off, args.steps), "moe_timing_enable")
    wall_events = timed_steps(ctx_off)
    kern = {}
    for ph in (0, 1):
        for kid in range(M.MOE_NUM_KERNELS):
            st, ms, n = M.moe_timing_read(ctx_off, ph, kid)
            M.check(st)
            if n:
                kern[(ph, M.moe_kernel_name(kid))] = (ms, n)
    M.check(M.moe_timing_enable(ctx_off, 0))

    # ---- the same kernels with each phase alone (K layers back to back on
    # its stream, per-kernel events).  In the concurrent steps the D stream's
    # K layers run beside the first few P layers, and while D's waves hold a
    # CU a P tile that needs the whole CU cannot start there, so those P
    # launches take longer; the launches of a phase alone show what the
    # kernel itself reaches.
    kern_alone = {}
    M.check(M.moe_timing_enable(ctx_off, args.steps), "moe_timing_enable")
    for ph in (0, 1):
        for _ in range(args.steps):
            layer(ph, ctx_off)
        torch.cuda.synchronize()
        for kid in range(M.MOE_NUM_KERNELS):
            st, ms, n = M.moe_timing_read(ctx_off, ph, kid)
            M.check(st)
            if n:
                kern_alone[(ph, M.moe_kernel_name(kid))] = (ms, n)
    M.check(M.moe_timing_enable(ctx_off, 0))

    # rows and touched experts of each phase (device-side layout, read once)
    rows, touched, t_res = {}, {}, {}
    for ph in (0, 1):
        rows[ph], touched[ph], t_res[ph] = layout_counts(M, ctx, ph, spec)

    # ---- D latency alone and under P
    # D alone is measured back to back (the layer's weights partly stay in the
    # 256 MB memory-side cache, as they do under P, whose batch streams the
    # same weights) and, separately, from a cold cache after a 1 GiB fill
    # outside the events (a model returns to a layer's weights only after
    # all its other layers).  The ratio uses the back-to-back figure.
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)

    def flush_mall():
        flush.zero_()
        torch.cuda.current_stream().synchronize()

    def d_latencies(under_p, c, cold=False):
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in
               range(args.d_iters)]
        p_first = torch.cuda.Event(enable_timing=True)
        p_last = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        if under_p:
            p_first.record(sP)
            n_p = 4
            for _ in range(n_p):
                layer(0, c)
        lat = []
        for i in range(args.d_iters):
            a, b = evs[i]
            if under_p:
                layer(0, c)  # keep the P stream one layer ahead
            elif cold:
                flush_mall()
            a.record(sD)
            layer(1, c)
            b.record(sD)
            if not under_p:
                sD.synchronize()
        if under_p:
            p_last.record(sP)
        torch.cuda.synchronize()
        lat = [a.elapsed_time(b) * 1000.0 for a, b in evs]
        overlapped = None
        if under_p:
            overlapped = sum(1 for a, b in evs if p_first.elapsed_time(a) >= 0 and b.elapsed_time(p_last) >= 0)
        return lat, overlapped

    lat_alone, _ = d_latencies(False, ctx)
    lat_cold, _ = d_latencies(False, ctx, cold=True)
    lat_under, overlapped = d_latencies(True, ctx)

    # ---- the same, with the D layer captured once into a HIP graph and
    # replayed against its stable phase buffers (the paper's D graph path)
    def d_graph_latencies(c):
        sg = torch.cuda.Stream(device=dev)
        torch.cuda.synchronize()
        M.layer(c, 1, lg[1], T[1], xs[1], outs[1], sg)  # the phase last ran on the capture stream
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=sg):
            M.layer(c, 1, lg[1], T[1], xs[1], outs[1], sg)
        torch.cuda.synchronize()
        res = {}
        for under_p in (False, True):
            evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                   for _ in range(args.d_iters)]
            torch.cuda.synchronize()
            if under_p:
                for _ in range(4):
                    layer(0, c)
            for a, b in evs:
                if under_p:
                    layer(0, c)
                with torch.cuda.stream(sg):
                    a.record(sg)
                    graph.replay()
                    b.record(sg)
                if not under_p:
                    sg.synchronize()
            torch.cuda.synchronize()
            res[under_p] = [a.elapsed_time(b) * 1000.0 for a, b in evs]
        del graph
        torch.cuda.synchronize()
        return res

    glat = d_graph_latencies(ctx)

    # the shader clock, idle and beside P layers (peaks stay the datasheet's)
    def clock_mhz(under_p):
        buf = torch.zeros(2, dtype=torch.int64, device=dev)
        sc = torch.cuda.Stream(device=dev)
        torch.cuda.synchronize()
        if under_p:
            for _ in range(3):
                layer(0, ctx)
        M.check(M.moe_clock_probe(sc, 400, buf.data_ptr()), "moe_clock_probe")
        torch.cuda.synchronize()
        ticks, ref = buf.tolist()
        return round(ticks * 100.0 / ref, 1)

    clock = {"idle": clock_mhz(False), "beside_p": clock_mhz(True),
             "note": "shader-clock ticks over a 100 MHz reference-clock spin of 400 us (one wave); "
                     "beside_p: while P layers run on the P stream"}
    segments = segment_sweep(args, M, ctx, lg, xs, T, spec, sP, dev) if args.seg_layers > 0 else None
    router = None if args.no_router else router_measure(M, ctx_off, xs, T, spec, inp, sP, sD, packed)
    if ctx_off is not ctx:
        lat_alone_off, _ = d_latencies(False, ctx_off)
        lat_under_off, _ = d_latencies(True, ctx_off)
    else:
        lat_alone_off, lat_under_off = lat_alone, lat_under

    # ---- roofline of the dominant kernel
    tot = {}
    for (ph, name), (ms, n) in kern.items():
        tot[(ph, name)] = ms
    dom = max(tot, key=tot.get)
    ph_d, name_d = dom
    ms_d, n_d = kern[dom]
    avg_s = ms_d / n_d / 1e3
    by, fl = kernel_units(spec, name_d, T[ph_d], rows[ph_d], touched[ph_d], esz, osz, t_res[ph_d])
    t_hbm = by / (HBM_PEAK_GBS * 1e9)
    t_mfma = fl / (mma_peak * 1e12) if packed else fl / (FP32_VECTOR_PEAK_TFLOPS * 1e12)
    if fl and t_mfma >= t_hbm:
        achieved = fl / avg_s / 1e12
        peak = mma_peak if packed else FP32_VECTOR_PEAK_TFLOPS
        roof = {"bound": "mfma" if packed else "alu", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s"}
    else:
        achieved = by / avg_s / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s"}
    roof["frac"] = round(achieved / roof["peak"], 4)
    roof["traffic"] = recorded_traffic(args.config, ph_d, name_d, M.LIB_PATH)
    roof["kernel"] = f"{name_d} ({'P' if ph_d == 0 else 'D'})"
    roof["per_launch"] = {"bytes": by, "flops": fl, "mean_us": round(avg_s * 1e6, 2), "launches": n_d}
    roof_alone = None
    if dom in kern_alone:
        ms_a, n_a = kern_alone[dom]
        avg_a = ms_a / n_a / 1e3
        ach_a = (fl / avg_a / 1e12) if roof["unit"] == "TFLOP/s" else (by / avg_a / 1e9)
        roof_alone = {"achieved": round(ach_a, 2), "frac": round(ach_a / roof["peak"], 4), "unit": roof["unit"],
                      "mean_us": round(avg_a * 1e6, 2), "launches": n_a,
                      "note": "the same kernel and units, its phase's layers alone back to back (per-kernel "
                              "events); the roofline above averages the concurrent steps, where the other phase "
                              "holds some of the CUs during the first few layers"}

    kernels = {}
    for (ph, name), (ms, n) in sorted(kern.items()):
        by_k, fl_k = kernel_units(spec, name, T[ph], rows[ph], touched[ph], esz, osz, t_res[ph])
        us = ms / n * 1e3
        kernels[f"{'P' if ph == 0 else 'D'}.{name}"] = {
            "mean_us": round(us, 2),
            "GB/s": round(by_k / (us * 1e-6) / 1e9, 1) if by_k else None,
            "TFLOP/s": round(fl_k / (us * 1e-6) / 1e12, 1) if fl_k else None,
        }

    ms_per_step = wall / args.steps * 1e3
    value = (T[0] + T[1]) * args.steps / wall
    p50a, p50u = pct(lat_alone, 50), pct(lat_under, 50)
    res = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp8-mx" if fp8 else "bf16" if bf16 else "f32",
        "data": "synthetic",
        "config": {"workload": workload_name(spec), "E": spec.E, "E_loc": spec.E_loc, "top_k": spec.k, "H": spec.H,
                   "I": spec.I, "T_P": spec.T_P, "T_D": spec.T_D, "rows_P": rows[0], "rows_D": rows[1],
                   "parallelism": "single GPU, P and D on two streams", "d_priority_us": args.d_priority_us},
        "d_latency_us": {
            "p50_alone": round(p50a, 2), "p90_alone": round(pct(lat_alone, 90), 2),
            "p50_alone_cold": round(pct(lat_cold, 50), 2),
            "p50_under_p": round(p50u, 2), "p90_under_p": round(pct(lat_under, 90), 2),
            "p99_under_p": round(pct(lat_under, 99), 2), "ratio_p50": round(p50u / p50a, 3),
            "iters": args.d_iters, "overlapped_with_p": overlapped,
            "graph_p50_alone": round(pct(glat[False], 50), 2), "graph_p50_under_p": round(pct(glat[True], 50), 2),
            "graph_p90_under_p": round(pct(glat[True], 90), 2),
            "graph_ratio_p50": round(pct(glat[True], 50) / pct(glat[False], 50), 3),
            "note": "events on the D stream around one D layer; alone: back to back; alone_cold: after a 1 GiB "
                    "fill that clears the memory-side cache; under_p: with the P stream kept one layer ahead "
                    "(P streams the same weights)",
        },
        "roofline": roof,
        "roofline_phase_alone": roof_alone,
        "engine_clock_mhz": clock,
        "segments": segments,
        "router_from_hidden": router,
        "kernels": kernels,
        "kernels_pass_ms_per_step": round(wall_events / args.steps * 1e3, 4),
        "kernels_pass_note": "per-kernel HIP events over a second pass of the same concurrent steps, D-first admission "
                             "off, so P kernel durations hold no deliberate waits",
        "without_d_first": {
            "value": round((T[0] + T[1]) * args.steps / wall_off, 1),
            "ms_per_step": round(wall_off / args.steps * 1e3, 4),
            "d_p50_alone_us": round(pct(lat_alone_off, 50), 2),
            "d_p50_under_p_us": round(pct(lat_under_off, 50), 2),
            "ratio_p50": round(pct(lat_under_off, 50) / pct(lat_alone_off, 50), 3),
        },
    }
    M.check(M.moe_ctx_destroy(ctx))
    if ctx_off is not ctx:
        M.check(M.moe_ctx_destroy(ctx_off))
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(inp, args.cpu_seconds, args.cpu_tokens)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
