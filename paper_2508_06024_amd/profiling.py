"""Summaries of rocprofv3 output (kernel statistics and HBM counters) as short text.

    python -m paper_2508_06024_amd.profiling stats <run_kernel_stats.csv> --command "<cmd>" [-o out.md]
    python -m paper_2508_06024_amd.profiling traffic --fetch <fetch counter csv> --write <write counter csv>
        --kernel <substring> --copy-mib N --workload NAME --command "<cmd>" [-o out.json]

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

_SHORT = [
    (r"gemm_kernel<ec2moe::bf16_t, ec2moe::bf16_t, (\d+), (\d+), \d, \d, true>", r"gemm swiglu bf16 \1x\2"),
    (r"gemm_kernel<ec2moe::bf16_t, ec2moe::bf16_t, (\d+), (\d+), \d, \d, false>", r"gemm store bf16 \1x\2"),
    (r"gemm_kernel<ec2moe::bf16_t, float, (\d+), (\d+), \d, \d, false>", r"gemm store bf16->f32 \1x\2"),
    (r"gemm_kernel<float, float, (\d+), (\d+), \d, \d, (true|false)>", r"gemm f32 \1x\2 \3"),
]


def short_name(n: str) -> str:
    n = n.replace("(anonymous namespace)::", "")
    for pat, rep in _SHORT:
        m = re.search(pat, n)
        if m:
            return m.expand(rep)
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


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    s.add_argument("--command", required=True)
    s.add_argument("--bench-json", help="the bench.py JSON line of the same run: its HIP-event "
                                        "averages are listed beside the profiler's")
    s.add_argument("-o", "--out")
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
    if a.cmd == "stats":
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
