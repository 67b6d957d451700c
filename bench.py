#!/usr/bin/env python3
"""MoE-layer tokens/s of the EC2MoE hot path on one MI355X.

One step is the whole path on one batch: route X with the hardware-aware group gate,
compress it with the low-rank encoder, reconstruct it with the decoder, and run the
sparse MoE layer (SwiGLU, or two-layer ReLU experts for the paper-shaped "switch"
workloads) on the reconstruction with the gate's routing (permute, grouped expert
GEMMs, combine). Inputs are seeded synthetic tensors of the workload's
shape, resident in HBM before timing. Default workload: the Mixtral-shaped layer
(T=4096 tokens, d=4096, 8 experts in 2 groups, SwiGLU hidden 14336, top-2, codec
rank 256).

Prints one JSON line with tokens/s over the timed region, the roofline of the dominant
kernel (its HIP-event time inside the timed region, where only that kernel carries
events), a per-kernel breakdown from a separate profiled pass, and the CPU oracle
timed on a bounded sample of the same workload.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def parse():
    from paper_2508_06024_amd.workload import ALL_ORDER
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed steps (default 50; 1000 for 'decode')")
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="mixtral", choices=ALL_ORDER)
    ap.add_argument("--rotate", type=int, default=4, help="distinct copies of X cycled through the steps")
    ap.add_argument("--overlap", action="store_true",
                    help="run the routing (gate, permutation) on a second stream, overlapping the codec")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of HIP graphs of the step (one per input copy) instead of eager launches")
    ap.add_argument("--top-groups", type=int, default=0,
                    help="group-focused gate: keep the top G groups per token (0: every group)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target CPU time of the oracle sample")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="after timing, run one plain device copy of this many MiB (counter calibration)")
    return ap.parse_args()


def blas_info():
    """(threads, vendor) of the BLAS pool numpy calls."""
    try:
        from threadpoolctl import threadpool_info
        pools = [p for p in threadpool_info() if p.get("user_api") == "blas"]
    except Exception:
        pools = []
    threads = max([p["num_threads"] for p in pools] or [1])
    vendor = ", ".join(sorted({f"{p.get('internal_api', '?')} {p.get('version', '')}".strip() for p in pools})) or "unknown"
    return threads, vendor


def cpu_baseline(inp, cfg, target_s, top_groups=0):
    """The oracle's step (gate, encode, decode, experts, combine) on the first S tokens,
    with U restricted to those rows (one codec slice) or on the first S / h whole slices
    (several slices); weights are upcast to float64 before timing."""
    import oracle as O
    from paper_2508_06024_amd import workload as W
    f = inp.f64
    x, u, v = f("x"), f("u"), f("v")
    wg, wl = f("w_global"), f("w_local")
    gu = [W.to_f64(inp.w_gate_up[e], cfg.dtype) for e in range(cfg.n_experts)]
    dn = [W.to_f64(inp.w_down[e], cfg.dtype) for e in range(cfg.n_experts)]

    c, h = cfg.codec_slices, cfg.codec_h

    def run(S):
        t = time.perf_counter()
        uu = u[:S] if c == 1 else u
        O.layer(x[:S], inp.mask, wg, inp.b_global, wl, inp.b_local, gu, dn, uu, v, uu, v,
                cfg.n_groups, cfg.top_k, activation=cfg.activation, codec_slices=max(1, S // h) if c > 1 else 1,
                top_groups=top_groups)
        return time.perf_counter() - t

    T = cfg.n_tokens
    quantum = h if c > 1 else 64
    S0 = min(T, max(cfg.r_h, quantum))
    t0 = run(S0)
    S = int(min(T, max(S0, S0 * target_s / max(t0, 1e-6))))
    S = max(S0, (S // quantum) * quantum) if S < T else T
    t = run(S) if S != S0 else t0
    # the whole workload finishes under the target: repeat it until the target is reached
    reps = 1
    while S == T and t < target_s:
        t += run(S)
        reps += 1
    threads, vendor = blas_info()
    return {"value": S * reps / t, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "host_cores": len(os.sched_getaffinity(0)), "blas_vendor": vendor, "blas_threads": threads,
            "sample": f"oracle step (gate, encode, decode, experts, combine) on the first {S} of {T} tokens "
                      f"of the same inputs" + (", U restricted to those rows" if c == 1 else
                                                f", {S // h} of {c} codec slices") +
                      (f", {reps} runs" if reps > 1 else "") + f", float64, {t:.1f} s",
            "seconds": round(t, 2)}


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        log("bench.py measures one GPU: this implementation has no multi-GPU path "
            "(it would shard over tokens, with one all-reduce of the encoder's Z); run with --gpus 1")
        sys.exit(2)

    import torch
    from paper_2508_06024_amd import ec2moe as E
    from paper_2508_06024_amd import roofline as R
    from paper_2508_06024_amd import workload as W
    from paper_2508_06024_amd.layer import Ec2moeLayer

    cfg = W.CONFIGS[args.workload]
    per_call = cfg.mask == "per_call"
    steps = args.steps or (cfg.n_calls if per_call else 50)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    t_gen = time.perf_counter()
    inp = W.gen_layer(cfg)
    log(f"[bench] {cfg.name}: inputs generated in {time.perf_counter() - t_gen:.1f} s")

    def up(a):
        if cfg.dtype == W.BF16:
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)

    f32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dev)
    if per_call:
        calls = [W.gen_call(cfg, s) for s in range(cfg.first_call_seed, cfg.first_call_seed + min(steps, cfg.n_calls))]
        xs = [up(c[0]) for c in calls]
        masks = [c[1] for c in calls]
    else:
        xs = [up(inp.x) for _ in range(max(1, args.rotate))]
        masks = [inp.mask]
    layer = Ec2moeLayer(xs[0], masks[0], up(inp.w_global), f32(inp.b_global), up(inp.w_local), f32(inp.b_local),
                        up(inp.w_gate_up), up(inp.w_down), up(inp.u), up(inp.v),
                        n_groups=cfg.n_groups, top_k=cfg.top_k, activation=cfg.activation,
                        codec_slices=cfg.codec_slices, top_groups=args.top_groups, overlap=args.overlap)

    def step(i):
        layer.set_input(xs[i % len(xs)], masks[i % len(masks)])
        layer.step()

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # Per-kernel breakdown: a separate pass with the library's HIP events around every
    # kernel (on its launch stream). It also names the dominant kernel.
    prof_steps = min(steps, max(10, steps // 5))
    E.profile_select(None)
    E.profile_enable(True)
    for i in range(prof_steps):
        step(i)
    torch.cuda.synchronize()
    stats = E.profile_collect()
    E.profile_enable(False)
    stage_names = R.kernel_work(cfg, np.ones(cfg.n_experts, np.int64)).keys()
    dom = max((n for n in stats if n in stage_names), key=lambda n: stats[n][1])

    # Timed region: events only around the dominant kernel, so the others run back to back.
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    if args.graph and not per_call:
        # one graph per input copy (captured on a side stream after a warm-up there); the
        # dominant kernel's time comes from an eager pass with its events right after
        graphs = []
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            for i in range(len(xs)):
                step(i)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        for i in range(len(xs)):
            layer.set_input(xs[i], masks[i % len(masks)])
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                layer.step()
            graphs.append(g)
        torch.cuda.synchronize()
        start.record()
        for i in range(steps):
            graphs[i % len(graphs)].replay()
        end.record()
        torch.cuda.synchronize()
        ms = start.elapsed_time(end)
        E.profile_select(dom)
        E.profile_enable(True)
        for i in range(prof_steps):
            step(i)
        torch.cuda.synchronize()
    else:
        E.profile_select(dom)
        E.profile_enable(True)
        torch.cuda.synchronize()
        start.record()
        for i in range(steps):
            step(i)
        end.record()
        torch.cuda.synchronize()
        ms = start.elapsed_time(end)
    dom_stats = E.profile_collect()[dom]
    E.profile_enable(False)
    E.profile_select(None)
    ms_step = ms / steps
    tokens_s = cfg.n_tokens * steps / (ms / 1e3)
    log(f"[bench] {steps} steps in {ms:.2f} ms: {ms_step:.3f} ms/step, {tokens_s:.4g} tokens/s")

    if args.calibrate_copy_mib:
        n = args.calibrate_copy_mib * (1 << 20) // 4
        a = torch.ones(n, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        torch.mul(a, 1.0, out=b)  # one elementwise kernel: reads and writes N MiB
        torch.cuda.synchronize()
        log(f"[bench] calibration copy of {args.calibrate_copy_mib} MiB done")
        del a, b

    # Algorithmic work at the realised routing of the very calls each figure covers. With a
    # candidate mask drawn per call the routing, and with it the set of active experts whose
    # weights the GEMMs stream, changes from call to call: the work is then averaged over
    # the same calls (the gate, which is deterministic, run again alone on each).
    def mean_work(n):
        """(work per kernel, active experts), averaged over calls 0..n-1."""
        tot, active = None, 0
        for i in range(n if per_call else 1):
            layer.set_input(xs[i % len(xs)], masks[i % len(masks)])
            rows_e = R.expert_rows(layer.route()[0].cpu().numpy(), cfg.n_experts)
            w = R.kernel_work(cfg, rows_e)
            active += int(np.count_nonzero(rows_e))
            tot = w if tot is None else {k: (tot[k][0] + w[k][0], tot[k][1] + w[k][1]) for k in w}
        m = n if per_call else 1
        return {k: (f / m, b / m) for k, (f, b) in tot.items()}, active / m

    work, _ = mean_work(prof_steps)  # the calls of the per-kernel pass
    work_timed, active_timed = mean_work(steps) if per_call else (work, None)  # the calls of the timed region

    # per-kernel algorithmic work at the realised routing
    def stage_of(name):
        return R.stage_of(name) or name
    peak_f = R.PEAK_TFLOPS[cfg.dtype]
    kernels = {}
    for name, (n, tot) in stats.items():
        kernels[name] = {"launches_per_step": n / prof_steps, "avg_us": round(1e3 * tot / n, 2)}
    rows = {}
    for name, (n, tot) in stats.items():
        g = stage_of(name)
        rows.setdefault(g, [0.0, 0])
        rows[g][0] += tot / prof_steps  # ms per step
        rows[g][1] += n / prof_steps
    step_roof_ms = 0.0
    for g, (ms_g, _) in rows.items():
        if g in work:
            ft, bt = work_timed[g]
            step_roof_ms += max(ft / (peak_f * 1e12), bt / (R.PEAK_HBM_GBS * 1e9)) * 1e3
            flop, byt = work[g]
            t_f = flop / (peak_f * 1e12) * 1e3
            t_b = byt / (R.PEAK_HBM_GBS * 1e9) * 1e3
            bound = "mfma" if t_f >= t_b else "hbm"
            ach = flop / (ms_g * 1e-3) / 1e12 if bound == "mfma" else byt / (ms_g * 1e-3) / 1e9
            peak = peak_f if bound == "mfma" else R.PEAK_HBM_GBS
            for name in stats:
                if stage_of(name) == g:
                    kernels[name]["stage"] = g
            kernels.setdefault(f"stage:{g}", {})
            kernels[f"stage:{g}"] = {"ms_per_step": round(ms_g, 4), "bound": bound, "achieved": round(ach, 1),
                                     "unit": "TFLOP/s" if bound == "mfma" else "GB/s", "frac": round(ach / peak, 4)}

    n_l, tot = dom_stats  # the dominant kernel's launches inside the timed region
    avg_s = tot / n_l * 1e-3
    flop, byt = work_timed[dom]
    bound = "mfma" if flop / (peak_f * 1e12) >= byt / (R.PEAK_HBM_GBS * 1e9) else "hbm"
    if bound == "mfma":
        achieved, peak, unit = flop / avg_s / 1e12, peak_f, "TFLOP/s"
    else:
        achieved, peak, unit = byt / avg_s / 1e9, R.PEAK_HBM_GBS, "GB/s"
    traffic = R.measured_traffic(dom, cfg.name)
    roof = {"kernel": dom, "bound": bound, "achieved": round(achieved, 1), "peak": peak, "unit": unit,
            "frac": round(achieved / peak, 4), "traffic": traffic,
            "algorithmic": {"flop": flop, "bytes": byt}, "avg_launch_us": round(avg_s * 1e6, 1)}
    if per_call:
        roof["algorithmic_note"] = (f"mean over the {steps} timed calls of each call's work at its own routing "
                                    f"(active experts per call: {active_timed:.1f} on average)")
    # A step whose algorithmic bytes stay below twice the 256 MB Infinity Cache re-reads the same
    # weights every step: its "HBM" rates may be partly cache hits.
    step_bytes = sum(b for _, b in work_timed.values())
    cache_note = (f"the step moves {step_bytes / 1e6:.0f} MB (algorithmic), the same weights every step: below "
                  f"512 MB the per-stage HBM rates may include Infinity Cache (256 MB) hits"
                  if step_bytes < 512e6 and not per_call else None)

    # host planner (candidate mask producer and task scheduler): host time per call
    rng = np.random.default_rng(0)
    comp = rng.gamma(2.0, 2.0, cfg.n_experts)
    st, sp = E.DeviceState(4, 4, 4, 4), E.SelectionParams(1, 1, 1, 1, 1.0, 0.4)
    tc, tm = rng.gamma(2.0, 1.0, 1024), rng.gamma(1.5, 1.0, 1024)
    sch = E.ScheduleParams(0.5, 1.0, 1e-3, 200.0, 0.0, 0.0, 1.0, 4.0)
    t0 = time.perf_counter()
    for _ in range(200):
        E.select_candidates(st, sp, comp)
    t1 = time.perf_counter()
    for _ in range(200):
        E.schedule_tasks(sch, tc, tm)
    t2 = time.perf_counter()
    planner = {"select_candidates_us": round((t1 - t0) / 200 * 1e6, 2), "experts": cfg.n_experts,
               "schedule_tasks_us": round((t2 - t1) / 200 * 1e6, 2), "tasks": 1024,
               "note": "host calls through the Python binding (marshalling included)"}

    cpu = None
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample ...")
        cpu = cpu_baseline(inp, cfg, args.cpu_seconds, args.top_groups)
        log(f"[bench] oracle: {cpu['value']:.4g} tokens/s on {cpu['cores']} threads")

    out = {
        "metric": "MoE-layer tokens/s incl. group gate + low-rank codec",
        "value": round(tokens_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: T={cfg.n_tokens} d={cfg.d_model} experts={cfg.n_experts} "
                               f"groups={cfg.n_groups} {'ReLU' if cfg.activation == 'relu' else 'SwiGLU'} "
                               f"H={cfg.ffn_hidden} top-{cfg.top_k} codec {cfg.r_h}x{cfg.r_w}"
                               + (f" on {cfg.codec_slices} slices of {cfg.codec_h} tokens" if cfg.codec_slices > 1
                                  else "") + f", mask={cfg.mask}" + (f" keeping {cfg.n_keep}" if cfg.n_keep else "")
                               + (f", gate keeps the top {args.top_groups} groups" if args.top_groups else ""),
                   "tokens_per_step": cfg.n_tokens},
        "roofline": roof,
        "layer_roofline_frac": round(step_roof_ms / ms_step, 4),
        "cache_note": cache_note,
        "kernels": kernels,
        "kernels_pass": f"separate pass of {prof_steps} steps with HIP events around every kernel",
        "launch": ("HIP graph replays of the step (the dominant kernel's time from an eager pass)"
                   if args.graph and not per_call else "eager launches")
                  + (", routing on a second stream" if args.overlap else ""),
        "cpu_baseline": cpu,
        "planner": planner,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
