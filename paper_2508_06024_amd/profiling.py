"""Summaries of rocprofv3 output (kernel statistics and HBM counters) as short text.

    python -m paper_2508_06024_amd.profiling stats <run_kernel_stats.csv> --command "<cmd>" [-o out.md]
    python -m paper_2508_06024_amd.profiling traffic --fetch <fetch counter csv> --write <write counter csv>
        --kernel <substring> --copy-mib N --workload NAME --command "<cmd>" [-o out.json]
    python -m paper_2508_06024_amd.profiling counters --mfma <csv> --fetch <csv> --write <csv>
        --copy-mib N --command "<cmd>" [-o out.md]

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
    SIMD's matrix core busy for 32 of them."""
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
    a = ap.parse_args(argv)
    if a.cmd == "counters":
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
