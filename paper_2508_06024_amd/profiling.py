"""Summaries of rocprofv3 output (kernel statistics and HBM counters) as short text.

    python -m paper_2508_06024_amd.profiling stats <run_kernel_stats.csv> --command "<cmd>" [-o out.md]
    python -m paper_2508_06024_amd.profiling traffic --fetch <fetch counter csv> --write <write counter csv>
        --kernel <substring> --copy-mib N --workload NAME --command "<cmd>" [-o out.json]
    python -m paper_2508_06024_amd.profiling counters --mfma <csv> --fetch <csv> --write <csv>
        --copy-mib N --command "<cmd>" [-o out.md]
    python -m paper_2508_06024_amd.profiling dense [--tokens T --d-model d --hidden H --reps R]
        (GPU: the expert GEMMs on one dense expert beside torch.matmul on the same products)

HBM bytes of a kernel come from FETCH_SIZE and WRITE_SIZE (KiB per dispatch), each
scaled by the ratio of the known bytes of a plain elementwise pass over N MiB (the
benchmark's --calibrate-copy-mib: it reads N MiB and writes N MiB) to what the same
counter reads for that pass.
"""
from __future__ import annotations

import argparse
import csv
import datetime
import json
import re
import sys
from collections import defaultdict

from . import roofline as R

# register-staged GEMM instances; a trailing template argument of 16 or 32 marks 256- or 512-byte slab rows
_SHORT = [
    (r"gemm_kernel<ec2moe::bf16_t, ec2moe::bf16_t, (\d+), (\d+), \d, \d, true(?:, (\d+))?>", "gemm swiglu bf16 {0}x{1}"),
    (r"gemm_kernel<ec2moe::bf16_t, ec2moe::bf16_t, (\d+), (\d+), \d, \d, false(?:, (\d+))?>", "gemm store bf16 {0}x{1}"),
    (r"gemm_kernel<ec2moe::bf16_t, float, (\d+), (\d+), \d, \d, false(?:, (\d+))?>", "gemm store bf16->f32 {0}x{1}"),
    (r"gemm_kernel<float, float, (\d+), (\d+), \d, \d, (?:true|false)(?:, (\d+))?>", "gemm f32 {0}x{1}"),
]


def short_name(n: str) -> str:
    n = n.replace("(anonymous namespace)::", "")
    for pat, rep in _SHORT:
        m = re.search(pat, n)
        if m:
            name = rep.format(m.group(1), m.group(2))
            if "float, float" in m.group(0):
                name += " swiglu" if ", true" in m.group(0) else " store"
            if m.group(3) in ("16", "32"):
                name += f" ({int(m.group(3)) * 16}-byte slabs)"
            return name
    n = re.sub(r"\(.*\)$", "", n)
    return n.replace("ec2moe::", "").replace("void ", "")


def stats_summary(path: str, command: str) -> str:
    rows = list(csv.DictReader(open(path)))
    lines = [f"# rocprofv3 kernel statistics", "", f"command: `{command}`", "",
             f"date: {datetime.date.today().isoformat()}", "",
             "| kernel | calls | avg us | min us | max us | % of GPU time |", "|---|---|---|---|---|---|"]
    for r in rows:
        lines.append(f"| {short_name(r['Name'])} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.2f} |")
    return "\n".join(lines) + "\n"


def _counter_per_dispatch(path: str, counter: str):
    """{kernel name: [value per dispatch]} for one counter (summed over its instances)."""
    per = defaultdict(lambda: defaultdict(float))
    names = {}
    for r in csv.DictReader(open(path)):
        if r.get("Counter_Name") != counter:
            continue
        did = r.get("Dispatch_Id") or r.get("Correlation_Id")
        per[did]["v"] += float(r["Counter_Value"])
        names[did] = r["Kernel_Name"]
    out = defaultdict(list)
    for did, v in per.items():
        out[names[did]].append(v["v"])
    return out


def traffic(fetch_csv: str, write_csv: str, kernel: str, copy_mib: int):
    fetch = _counter_per_dispatch(fetch_csv, "FETCH_SIZE")
    write = _counter_per_dispatch(write_csv, "WRITE_SIZE")

    def pick(d, sub):
        ks = [k for k in d if sub in k]
        if not ks:
            raise KeyError(f"no kernel matching {sub!r}")
        vals = [v for k in ks for v in d[k]]
        return sum(vals) / len(vals), len(vals)

    def calib(d):
        # the calibration kernel: the largest elementwise dispatch of the run
        vals = [v for k in d if "elementwise" in k for v in d[k]]
        if not vals:
            raise KeyError("no elementwise calibration dispatch")
        return max(vals)

    copy_kib = copy_mib * 1024.0
    f_copy, w_copy = calib(fetch), calib(write)
    f_kib, nf = pick(fetch, kernel)
    w_kib, nw = pick(write, kernel)
    f_scale, w_scale = copy_kib / f_copy, copy_kib / w_copy
    return {"fetch_kib_raw": f_kib, "write_kib_raw": w_kib, "copy_fetch_kib": f_copy, "copy_write_kib": w_copy,
            "fetch_scale": f_scale, "write_scale": w_scale, "dispatches": [nf, nw],
            "hbm_bytes_per_launch": (f_kib * f_scale + w_kib * w_scale) * 1024.0}


def _per_dispatch(path: str):
    """{dispatch id: (kernel name, duration ns, {counter: value summed over instances})}."""
    out = {}
    for r in csv.DictReader(open(path)):
        did = r.get("Dispatch_Id") or r.get("Correlation_Id")
        if did not in out:
            out[did] = [r["Kernel_Name"], int(r["End_Timestamp"]) - int(r["Start_Timestamp"]), defaultdict(float)]
        out[did][2][r["Counter_Name"]] += float(r["Counter_Value"])
    return out


def counters_summary(mfma_csv: str, fetch_csv: str, write_csv: str, copy_mib: int, command: str,
                     xcds: int = 8, simds: int = 1024) -> str:
    """Per kernel: matrix-core busy fraction and clock (SQ_VALU_MFMA_BUSY_CYCLES, GRBM_GUI_ACTIVE)
    and HBM bytes (FETCH_SIZE, WRITE_SIZE scaled by the copy calibration), averaged over its
    dispatches. GRBM_GUI_ACTIVE sums the active cycles of every XCD, so the kernel's clock is
    GUI / xcds / duration and its SIMD-cycles GUI / xcds * simds; a 32x32x16 bf16 MFMA keeps a
    SIMD's matrix core busy for 32 of them, a 16x16x32 one for 16."""
    m = _per_dispatch(mfma_csv)
    f = _per_dispatch(fetch_csv)
    w = _per_dispatch(write_csv)

    def calib(d, counter):
        vals = [c[counter] for n, _, c in d.values() if "elementwise" in n and counter in c]
        if not vals:
            raise KeyError("no elementwise calibration dispatch")
        return copy_mib * 1024.0 / max(vals)

    fs, ws = calib(f, "FETCH_SIZE"), calib(w, "WRITE_SIZE")
    # one kernel serving launches of very different sizes (the same GEMM for a codec product
    # and an expert layer): its dispatches are split at the geometric mean of the extremes when
    # they differ by more than 5x
    # the passes run the same launch sequence: the i-th dispatch of a kernel is the same launch
    # in every pass, classified by the median of its durations
    def ordered(d):
        out = defaultdict(list)
        for did in sorted(d, key=lambda x: int(x)):
            name, dur, c = d[did]
            out[short_name(name)].append((dur, c))
        return out
    om, of_, ow = ordered(m), ordered(f), ordered(w)
    rows = defaultdict(lambda: defaultdict(list))
    for n in om:
        if "elementwise" in n or "rocclr" in n:
            continue
        per = [om[n], of_.get(n, []), ow.get(n, [])]
        k = min(len(x) for x in per)
        med = [sorted(x[i][0] for x in per)[1] for i in range(k)]
        lo, hi = (min(med), max(med)) if med else (0, 0)
        cut = (lo * hi) ** 0.5 if lo > 0 and hi > 5 * lo else None
        for i in range(k):
            name = n if cut is None else n + (" (long launches)" if med[i] > cut else " (short launches)")
            r = rows[name]
            for (dur, c), key in zip((per[0][i], per[1][i], per[2][i]), ("m", "f", "w")):
                r["dur_" + key].append(dur)
                for cn, v in c.items():
                    r[cn].append(v)
    avg = lambda v: sum(v) / len(v) if v else float("nan")
    lines = ["# rocprofv3 counters per kernel", "", f"command: `{command}`", "",
             f"date: {datetime.date.today().isoformat()}", "",
             f"FETCH_SIZE scaled by {fs:.3f} and WRITE_SIZE by {ws:.3f} (a plain elementwise pass over "
             f"{copy_mib} MiB reads and writes {copy_mib} MiB); durations are those of the counter runs "
             "(dispatches serialised by the profiler). GRBM_GUI_ACTIVE counts the GPU's busy cycles over "
             "the counter window, which for a dispatch of a few microseconds includes its launch and "
             "drain: MFMA busy and clock are shown for dispatches above 100 us only.", "",
             "| kernel | dispatches | avg us | MFMA busy | clock GHz | HBM read MB | HBM write MB | GB/s |",
             "|---|---|---|---|---|---|---|---|"]
    for name, r in rows.items():
        dur_m = avg(r["dur_m"])
        gui = avg(r["GRBM_GUI_ACTIVE"])
        busy = avg(r["SQ_VALU_MFMA_BUSY_CYCLES"])
        long = r["GRBM_GUI_ACTIVE"] and dur_m > 100e3
        util = busy / (gui / xcds * simds) if long else float("nan")
        clk = gui / xcds / dur_m if long else float("nan")
        rd = avg(r["FETCH_SIZE"]) * fs * 1024 / 1e6
        wr = avg(r["WRITE_SIZE"]) * ws * 1024 / 1e6
        dur_fw = avg(r["dur_f"] + r["dur_w"])
        gbs = (rd + wr) * 1e6 / (dur_fw * 1e-9) / 1e9 if dur_fw > 0 else float("nan")
        ut = f"{util:.1%}" if util == util else "-"
        ck = f"{clk:.2f}" if clk == clk else "-"
        lines.append(f"| {name} | {len(r['dur_m']) or len(r['dur_f'])} | {dur_m / 1e3:.2f} | {ut} | {ck} | "
                     f"{rd:.1f} | {wr:.1f} | {gbs:.0f} |")
    return "\n".join(lines) + "\n"


def dense_compare(T: int, d: int, H: int, reps: int, only: str = "", calibrate_copy_mib: int = 0) -> str:
    """The library's expert GEMMs on a single expert that takes every token (a dense SwiGLU
    FFN: gate-up T x 2H x d, down T x d x H) beside torch.matmul (the ROCm BLAS library) on
    the same two products, inputs N(0, 1) tokens and N(0, 0.02) weights in bfloat16, each
    timed with HIP events over `reps` calls after a warm-up. torch's gate-up writes all 2H
    columns; the library's writes the H SwiGLU outputs. `only` restricts the torch products to
    one of them (for counter runs, where both use the same library kernel); a calibration
    copy of N MiB, if asked for, ends the run (the counter scale, as in bench.py)."""
    import torch

    from . import ec2moe as E
    dev = torch.device("cuda", 0)
    g = torch.Generator(device=dev).manual_seed(0)
    bf = torch.bfloat16
    x = torch.randn(T, d, device=dev, generator=g).to(bf)
    w_gu = (torch.randn(1, 2 * H, d, device=dev, generator=g) * 0.02).to(bf)
    w_dn = (torch.randn(1, d, H, device=dev, generator=g) * 0.02).to(bf)
    seg = torch.tensor([0, T], dtype=torch.int32, device=dev)
    src = torch.arange(T, dtype=torch.int32, device=dev)
    ws = E.workspace(E.moe_workspace_size(E.moe_desc(T, 1, 1, d, H, 1, bf)), dev)
    for _ in range(2):
        E.expert_ffn(x, seg, src, w_gu, w_dn, 1, ws=ws)
    torch.cuda.synchronize()
    E.profile_select(None)
    E.profile_enable(True)
    for _ in range(reps):
        E.expert_ffn(x, seg, src, w_gu, w_dn, 1, ws=ws)
    torch.cuda.synchronize()
    st = E.profile_collect()
    E.profile_enable(False)
    # per call: the launch and its split-K reduction, if the tile count left a partial round
    lib = {k: sum(st[n][1] for n in (k, k + "_tail") if n in st) / reps * 1e3 for k in ("expert_gate_up", "expert_down")}

    a = torch.randn(T, H, device=dev, generator=g).to(bf)
    wgt, wdt = w_gu[0].t(), w_dn[0].t()
    blas = {}
    for name, (lhs, rhs) in (("expert_gate_up", (x, wgt)), ("expert_down", (a, wdt))):
        if only and name != "expert_" + only:
            blas[name] = float("nan")
            continue
        for _ in range(2):
            torch.matmul(lhs, rhs)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            torch.matmul(lhs, rhs)
        e1.record()
        torch.cuda.synchronize()
        blas[name] = e0.elapsed_time(e1) / reps * 1e3
    if calibrate_copy_mib:
        n = calibrate_copy_mib * (1 << 20) // 4
        c0 = torch.ones(n, dtype=torch.float32, device=dev)
        c1 = torch.empty_like(c0)
        torch.cuda.synchronize()
        torch.mul(c0, 1.0, out=c1)  # one elementwise kernel: reads and writes N MiB
        torch.cuda.synchronize()
        del c0, c1
    flops = {"expert_gate_up": 4.0 * T * d * H, "expert_down": 2.0 * T * d * H}
    lib_name = str(torch.backends.cuda.preferred_blas_library()).split(".")[-1]
    out = [f"dense SwiGLU expert, T = {T}, d = {d}, H = {H}, bf16, {reps} calls each "
           f"(torch {torch.__version__}, BLAS backend {lib_name})", "",
           "| product | shape (M x N x K) | library us | library PFLOP/s | torch.matmul us | torch PFLOP/s | ratio |",
           "|---|---|---|---|---|---|---|"]
    shapes = {"expert_gate_up": f"{T} x {2 * H} x {d}", "expert_down": f"{T} x {d} x {H}"}
    for k in ("expert_gate_up", "expert_down"):
        lu, bu = lib.get(k, float("nan")), blas[k]
        out.append(f"| {k} | {shapes[k]} | {lu:.1f} | {flops[k] / lu / 1e9:.3f} | {bu:.1f} | "
                   f"{flops[k] / bu / 1e9:.3f} | {bu / lu:.3f} |")
    return "\n".join(out) + "\n"


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    s.add_argument("--command", required=True)
    s.add_argument("--bench-json", help="the bench.py JSON line of the same run: its HIP-event "
                                        "averages are listed beside the profiler's")
    s.add_argument("-o", "--out")
    c = sub.add_parser("counters")
    c.add_argument("--mfma", required=True, help="csv of a run with GRBM_GUI_ACTIVE and SQ_VALU_MFMA_BUSY_CYCLES")
    c.add_argument("--fetch", required=True)
    c.add_argument("--write", required=True)
    c.add_argument("--copy-mib", type=int, required=True)
    c.add_argument("--command", required=True)
    c.add_argument("-o", "--out")
    t = sub.add_parser("traffic")
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--kernel", required=True, help="substring of the kernel name")
    t.add_argument("--name", required=True, help="profiler name of the kernel (e.g. expert_gate_up)")
    t.add_argument("--sources", nargs="+", required=True, help="csrc files the kernel is built from")
    t.add_argument("--copy-mib", type=int, required=True)
    t.add_argument("--workload", required=True)
    t.add_argument("--command", required=True)
    t.add_argument("-o", "--out")
    g = sub.add_parser("dense")
    g.add_argument("--tokens", type=int, default=8192)
    g.add_argument("--d-model", type=int, default=4096)
    g.add_argument("--hidden", type=int, default=14336)
    g.add_argument("--reps", type=int, default=20)
    g.add_argument("--only", choices=["gate_up", "down"], default="")
    g.add_argument("--calibrate-copy-mib", type=int, default=0)
    g.add_argument("-o", "--out")
    a = ap.parse_args(argv)
    if a.cmd == "dense":
        text = dense_compare(a.tokens, a.d_model, a.hidden, a.reps, a.only, a.calibrate_copy_mib)
    elif a.cmd == "counters":
        text = counters_summary(a.mfma, a.fetch, a.write, a.copy_mib, a.command)
    elif a.cmd == "stats":
        text = stats_summary(a.csv, a.command)
        if a.bench_json:
            rec = json.loads(open(a.bench_json).read().strip().splitlines()[-1])
            text += ("\nThe same run's bench.py line (library HIP events on the launch stream, timed "
                     "region only):\n\n| library kernel name | launches per step | avg us |\n|---|---|---|\n")
            for name, k in rec.get("kernels", {}).items():
                if not name.startswith("stage:"):
                    text += f"| {name} | {k['launches_per_step']:g} | {k['avg_us']} |\n"
            text += (f"\nbench: {rec['value']} {rec['unit']}, {rec['ms_per_step']} ms/step; roofline kernel "
                     f"{rec['roofline']['kernel']}: {rec['roofline']['achieved']} {rec['roofline']['unit']} "
                     f"({rec['roofline']['frac']:.1%} of peak)\n")
    else:
        rec = traffic(a.fetch, a.write, a.kernel, a.copy_mib)
        rec.update({"kernel": a.name, "workload": a.workload, "command": a.command, "sources": a.sources,
                    "source_digest": R.source_digest(*a.sources), "date": datetime.date.today().isoformat()})
        text = json.dumps(rec, indent=1) + "\n"
    if a.out:
        with open(a.out, "w") as f:
            f.write(text)
    else:
        sys.stdout.write(text)


if __name__ == "__main__":
    main()
