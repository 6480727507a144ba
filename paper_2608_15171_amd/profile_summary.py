"""Turn rocprofv3 CSV output for one bench workload into the committed summary.

Inputs (one directory per workload, as written by the commands in the summary):
  <dir>/trace/run_kernel_stats.csv                       rocprofv3 --kernel-trace --stats
  <dir>/FETCH_SIZE/run_counter_collection.csv            rocprofv3 --pmc FETCH_SIZE
  <dir>/WRITE_SIZE/run_counter_collection.csv            rocprofv3 --pmc WRITE_SIZE
  <calib>/{FETCH_SIZE,WRITE_SIZE}/run_counter_collection.csv   the same counters for calibrate.py
  <dir>/trace_bench.json                                 bench.py's JSON line of the traced run

Writes profiles/<kernel>.<workload>.md and .traffic.json. The byte counters
are scaled by what they read for a plain copy of known size; the record carries
a hash of the kernel's sources (for the attention kernel, with the planner's) so
bench.py reports the traffic only while those sources are unchanged.

Usage: python -m paper_2608_15171_amd.profile_summary <workload> <dir> <calib_dir> [kernel]
       (kernel: attn_step_kernel, the default, or rope_append_kernel)
"""
from __future__ import annotations

import csv
import hashlib
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SOURCES = {
    "attn_step_kernel": ["paper_2608_15171_amd/csrc/attn_step.hip", "paper_2608_15171_amd/csrc/plan.cpp",
                         "paper_2608_15171_amd/csrc/plan.h"],
    "rope_append_kernel": ["paper_2608_15171_amd/csrc/rope_append.hip"],
}
DESCRIPTION = {
    "attn_step_kernel": "One packed attention launch of the mixed step on one MI355X (gfx950); bf16 inputs, fp32 "
                        "accumulation.",
    "rope_append_kernel": "The rotary embedding of a step's new rows fused with their page write, one launch on one "
                          "MI355X (gfx950); bf16 in and out, fp32 rotation.",
}
ALGORITHMIC = {
    "attn_step_kernel": "algorithmic bytes (visible K/V once + Q + O)",
    "rope_append_kernel": "algorithmic bytes (Q read and written, new K/V read and written, once each)",
}


def sources_hash(sources) -> str:
    h = hashlib.sha256()
    for src in sources:
        h.update(open(os.path.join(ROOT, src), "rb").read())
    return h.hexdigest()


def counter_per_dispatch(path: str, name_part: str, counter: str):
    """Mean over dispatches of the counter summed per dispatch, for kernels whose name contains name_part."""
    per = {}
    for r in csv.DictReader(open(path)):
        if name_part in r["Kernel_Name"] and r["Counter_Name"] == counter:
            per[r["Dispatch_Id"]] = per.get(r["Dispatch_Id"], 0.0) + float(r["Counter_Value"])
    if not per:
        raise ValueError(f"no {counter} records for {name_part} in {path}")
    return sum(per.values()) / len(per), len(per)


def main(workload: str, d: str, calib: str, kernel: str = "attn_step_kernel"):
    stats = list(csv.DictReader(open(os.path.join(d, "trace", "run_kernel_stats.csv"))))
    bench = json.loads(open(os.path.join(d, "trace_bench.json")).read().strip().splitlines()[-1])
    wl_name = bench["config"]["workload"]
    attn = [r for r in stats if kernel in r["Name"]]
    total = sum(float(r["TotalDurationNs"]) for r in stats)
    fetch_kib, nf = counter_per_dispatch(os.path.join(d, "FETCH_SIZE", "run_counter_collection.csv"), kernel, "FETCH_SIZE")
    write_kib, nw = counter_per_dispatch(os.path.join(d, "WRITE_SIZE", "run_counter_collection.csv"), kernel, "WRITE_SIZE")
    mib = 1024
    copy_bytes = mib * 1024 * 1024
    cf, _ = counter_per_dispatch(os.path.join(calib, "FETCH_SIZE", "run_counter_collection.csv"), "UnaryFunctor", "FETCH_SIZE")
    cw, _ = counter_per_dispatch(os.path.join(calib, "WRITE_SIZE", "run_counter_collection.csv"), "UnaryFunctor", "WRITE_SIZE")
    ffac = copy_bytes / (cf * 1024)
    wfac = copy_bytes / (cw * 1024)
    fetch_b = fetch_kib * 1024 * ffac
    write_b = write_kib * 1024 * wfac
    alg = bench["roofline"]["per_launch"]["bytes"]
    rec = {"kernel": kernel, "workload": wl_name, "kernel_sources_sha256": sources_hash(SOURCES[kernel]),
           "sources": SOURCES[kernel],
           "fetch_bytes_per_launch": fetch_b, "write_bytes_per_launch": write_b, "fetch_factor": ffac,
           "write_factor": wfac, "fetch_kib": fetch_kib, "write_kib": write_kib}
    out = os.path.join(ROOT, "profiles", f"{kernel}.{workload}")
    json.dump(rec, open(out + ".traffic.json", "w"), indent=1)
    cmd = f"bench.py --workload {workload} --no-cpu-baseline"
    lines = [f"# {kernel} -- workload {wl_name} ({workload})", "",
             DESCRIPTION[kernel], "",
             "## Kernel trace (rocprofv3 --kernel-trace --stats)", "", "Command:", "",
             f"    cd /tmp && TMPDIR=/tmp rocprofv3 --kernel-trace --stats --output-format csv -d <out> -o run -- "
             f"python3 <repo>/{cmd}", "",
             "| kernel | calls | average (us) | min (us) | share of GPU time |", "|---|---|---|---|---|"]
    for r in sorted(stats, key=lambda r: -float(r["TotalDurationNs"]))[:6]:
        lines.append(f"| {r['Name'][:60]} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {100 * float(r['TotalDurationNs']) / total:.1f}% |")
    a = attn[0]
    ev_us, tr_us = float(bench['roofline']['kernel_us']), float(a['AverageNs']) / 1e3
    lines += ["", f"bench.py in the same run, HIP events recorded by the launch: {ev_us:.2f} us per "
                  f"launch over its {bench['steps']} timed steps (rocprofv3 average {tr_us:.2f} us "
                  f"over {a['Calls']} launches including warm-up)."]
    if abs(ev_us - tr_us) > 0.1 * tr_us:
        lines.append(f"The two differ by {ev_us - tr_us:+.1f} us: under the profiler its own per-dispatch work "
                     "falls between the two events recorded by the launch, which shows for a kernel this short; "
                     "the trace's duration is the kernel's.")
    lines += ["", "## HBM traffic (rocprofv3 --pmc, one counter per run)", "", "Commands:", ""]
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        lines.append(f"    cd /tmp && TMPDIR=/tmp rocprofv3 --pmc {c} --output-format csv -d <out> -o run -- "
                     f"python3 <repo>/{cmd} --steps 3 --warmup 1")
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        lines.append(f"    cd /tmp && TMPDIR=/tmp rocprofv3 --pmc {c} --output-format csv -d <out> -o run -- "
                     f"python3 <repo>/paper_2608_15171_amd/calibrate.py --mib {mib}")
    lines += ["", f"Calibration: a plain copy that reads and writes {mib} MiB per launch reads FETCH_SIZE = {cf:.0f} KiB "
                  f"and WRITE_SIZE = {cw:.0f} KiB, so bytes = FETCH_SIZE x 1024 x {ffac:.3f} and WRITE_SIZE x 1024 x {wfac:.3f}.",
              "", "| per launch | value |", "|---|---|",
              f"| FETCH_SIZE (KiB, mean of {nf} launches) | {fetch_kib:.0f} |",
              f"| WRITE_SIZE (KiB, mean of {nw} launches) | {write_kib:.0f} |",
              f"| bytes read from memory | {fetch_b / 1e6:.1f} MB |",
              f"| bytes written | {write_b / 1e6:.1f} MB |",
              f"| {ALGORITHMIC[kernel]} | {alg / 1e6:.1f} MB |",
              f"| measured / algorithmic | {(fetch_b + write_b) / alg:.2f} |", ""]
    open(out + ".md", "w").write("\n".join(lines))
    print(out + ".md")


if __name__ == "__main__":
    main(*sys.argv[1:5])
