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
       (kernel: attn_step_kernel, the default, rope_append_kernel or gateup_kernel)
       python -m paper_2608_15171_amd.profile_summary --mfma <workload> <dir>
       (matrix-core utilisation from one counter pass: profiles/<kernel>.<workload>.mfma.md)
       python -m paper_2608_15171_amd.profile_summary --cache <workload> <dir>
       (L2 hit rate of the gate-up kernel from one counter pass: profiles/gateup_kernel.<workload>.cache.md)
       python -m paper_2608_15171_amd.profile_summary --read <dir> <calib_dir>
       (the streaming read that sets the measured HBM ceiling: profiles/stream_read_kernel.read-2GiB.md)
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
    "gateup_kernel": ["paper_2608_15171_amd/csrc/gateup.hip"],
}
DESCRIPTION = {
    "attn_step_kernel": "One packed attention launch of the mixed step on one MI355X (gfx950); bf16 inputs, fp32 "
                        "accumulation.",
    "rope_append_kernel": "The rotary embedding of a step's new rows fused with their page write, one launch on one "
                          "MI355X (gfx950); bf16 in and out, fp32 rotation.",
    "gateup_kernel": "The MLP's fused gate-up projection Y = X W^T (hidden 2048, 22016 stacked gate/up rows), one "
                     "launch on one MI355X (gfx950); bf16 inputs, fp32 accumulation.",
}
DESCRIPTION_ACT = ("The MLP's gate-up projection with the gated activation in its epilogue, Z = silu(X W_gate^T) * "
                   "(X W_up^T) (hidden 2048, 11008 features), one launch on one MI355X (gfx950); bf16 inputs, fp32 "
                   "accumulation and activation.")


def describe(kernel: str, workload: str) -> str:
    return DESCRIPTION_ACT if workload.startswith("gateup-act") else DESCRIPTION[kernel]


ALGORITHMIC = {
    "attn_step_kernel": "algorithmic bytes (visible K/V once + Q + O)",
    "rope_append_kernel": "algorithmic bytes (Q read and written, new K/V read and written, once each)",
    "gateup_kernel": "algorithmic bytes (X and W read once, the output written once)",
}


def _sec(kernel: str) -> str:
    """The attention workloads were profiled without the bench's secondary record."""
    return " --secondary none" if kernel == "attn_step_kernel" else ""


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
    cmd = f"bench.py --workload {workload}{_sec(kernel)} --no-cpu-baseline --no-attainable"
    lines = [f"# {kernel} -- workload {wl_name} ({workload})", "",
             describe(kernel, workload), "",
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


MFMA_COUNTERS = ["GRBM_GUI_ACTIVE", "SQ_WAVE_CYCLES", "SQ_BUSY_CYCLES", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_MFMA",
                 "SQ_INSTS_VALU", "SQ_INSTS_LDS", "SQ_LDS_IDX_ACTIVE", "SQ_LDS_BANK_CONFLICT"]


def mfma_summary(workload: str, d: str, kernel: str = "", simds: int = 1024, xcds: int = 8):
    """Matrix-core utilisation of the kernel from one rocprofv3 --pmc pass of MFMA_COUNTERS
    (<d>/MFMA/run_counter_collection.csv, <d>/MFMA_bench.json). SQ counters are summed over
    the chip, GRBM_GUI_ACTIVE over the XCDs; means over the pass's last two dispatches."""
    kernel = kernel or ("gateup_kernel" if workload.startswith("gateup") else "attn_step_kernel")
    rows = list(csv.DictReader(open(os.path.join(d, "MFMA", "run_counter_collection.csv"))))
    per, dur = {}, {}
    for r in rows:
        if kernel not in r["Kernel_Name"]:
            continue
        c = per.setdefault(r["Dispatch_Id"], {})
        c[r["Counter_Name"]] = c.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
        dur[r["Dispatch_Id"]] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
    ids = sorted(per, key=int)[-2:]
    m = {k: sum(per[i][k] for i in ids) / len(ids) for k in MFMA_COUNTERS}
    us = sum(dur[i] for i in ids) / len(ids)
    bench = json.loads(open(os.path.join(d, "MFMA_bench.json")).read().strip().splitlines()[-1])
    flop = bench["roofline"]["per_launch"]["flop"]
    cycles = m["GRBM_GUI_ACTIVE"] / xcds
    clock = cycles / us / 1e3
    busy = m["SQ_VALU_MFMA_BUSY_CYCLES"] / (simds * cycles)
    mfma_flop = m["SQ_INSTS_MFMA"] * 32768       # the 32x32x16 bf16 and 16x16x32 bf16 MFMAs both do 2*16384 FLOP
    cmd = (f"cd /tmp && TMPDIR=/tmp rocprofv3 --pmc {' '.join(MFMA_COUNTERS)} --output-format csv -d <out> -o run "
           f"-- python3 <repo>/bench.py --workload {workload}{_sec(kernel)} --no-cpu-baseline --no-attainable --steps 3 --warmup-seconds 0.5")
    lines = [f"# {kernel} -- matrix-core utilisation, workload {bench['config']['workload']} ({workload})", "",
             describe(kernel, workload), "", "Command (one counter pass):", "", "    " + cmd, "",
             "| quantity | value | how it is read |", "|---|---|---|",
             f"| kernel time under the profiler | {us:.1f} us | dispatch timestamps, mean of the pass's last two launches |",
             f"| engine clock | {clock:.2f} GHz | GRBM_GUI_ACTIVE / {xcds} XCDs / kernel time |",
             f"| MFMA pipe busy | {100 * busy:.1f} % of SIMD cycles | SQ_VALU_MFMA_BUSY_CYCLES / ({simds} SIMDs x cycles) |",
             f"| MFMA instructions x 32,768 FLOP | {mfma_flop / 1e9:.1f} GFLOP | SQ_INSTS_MFMA; algorithmic FLOP {flop / 1e9:.1f} G "
             f"(masked keys of diagonal blocks and padded decode heads are executed too) |",
             f"| MFMA rate at the run's clock | {mfma_flop / (us * 1e-6) / 1e12:.0f} TFLOP/s | executed MFMA FLOP / kernel time |",
             f"| algorithmic rate | {flop / (us * 1e-6) / 1e12:.0f} TFLOP/s = {100 * flop / (us * 1e-6) / 2.5e15:.1f} % of the 2.5 PFLOP/s bf16 peak | |",
             f"| VALU instructions per MFMA | {m['SQ_INSTS_VALU'] / m['SQ_INSTS_MFMA']:.2f} | SQ_INSTS_VALU / SQ_INSTS_MFMA (MFMAs included) |",
             f"| LDS instructions per MFMA | {m['SQ_INSTS_LDS'] / m['SQ_INSTS_MFMA']:.2f} | SQ_INSTS_LDS / SQ_INSTS_MFMA |",
             f"| LDS busy | {100 * m['SQ_LDS_IDX_ACTIVE'] / (cycles * simds / 4):.1f} % of CU cycles | SQ_LDS_IDX_ACTIVE / (CUs x cycles) |",
             f"| LDS bank conflict cycles | {m['SQ_LDS_BANK_CONFLICT']:.0f} | SQ_LDS_BANK_CONFLICT |", ""]
    out = os.path.join(ROOT, "profiles", f"{kernel}.{workload}.mfma.md")
    open(out, "w").write("\n".join(lines))
    print(out)


STALL_COUNTERS = ["GRBM_GUI_ACTIVE", "SQ_WAVE_CYCLES", "SQ_BUSY_CYCLES", "SQ_WAIT_ANY", "SQ_WAIT_INST_ANY",
                  "SQ_ACTIVE_INST_ANY", "SQ_ACTIVE_INST_LDS", "SQ_WAIT_INST_LDS", "SQ_ACTIVE_INST_VALU"]


def stall_summary(workload: str, d: str, kernel: str = "", cus: int = 256, xcds: int = 8):
    """Where the kernel's waves spend their time, from one rocprofv3 --pmc pass of
    STALL_COUNTERS (<d>/STALL/run_counter_collection.csv, <d>/STALL_bench.json). The SQ
    wave counters are wave-cycles in units of 4 cycles, summed over the chip; means over
    the pass's last two dispatches."""
    kernel = kernel or ("gateup_kernel" if workload.startswith("gateup") else "attn_step_kernel")
    rows = list(csv.DictReader(open(os.path.join(d, "STALL", "run_counter_collection.csv"))))
    per, dur = {}, {}
    for r in rows:
        if kernel not in r["Kernel_Name"]:
            continue
        c = per.setdefault(r["Dispatch_Id"], {})
        c[r["Counter_Name"]] = c.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
        dur[r["Dispatch_Id"]] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
    ids = sorted(per, key=int)[-2:]
    m = {k: sum(per[i][k] for i in ids) / len(ids) for k in STALL_COUNTERS}
    us = sum(dur[i] for i in ids) / len(ids)
    bench = json.loads(open(os.path.join(d, "STALL_bench.json")).read().strip().splitlines()[-1])
    cycles = m["GRBM_GUI_ACTIVE"] / xcds
    wave = m["SQ_WAVE_CYCLES"]
    cmd = (f"cd /tmp && TMPDIR=/tmp rocprofv3 --pmc {' '.join(STALL_COUNTERS)} --output-format csv -d <out> -o run "
           f"-- python3 <repo>/bench.py --workload {workload}{_sec(kernel)} --no-cpu-baseline --no-attainable --steps 3 --warmup-seconds 0.5")
    share = lambda k: f"{100 * m[k] / wave:.1f} % of wave time"
    lines = [f"# {kernel} -- where the waves spend their time, workload {bench['config']['workload']} ({workload})", "",
             describe(kernel, workload), "", "Command (one counter pass):", "", "    " + cmd, "",
             "| quantity | value | how it is read |", "|---|---|---|",
             f"| kernel time under the profiler | {us:.1f} us | dispatch timestamps, mean of the pass's last two launches |",
             f"| engine clock | {cycles / us / 1e3:.2f} GHz | GRBM_GUI_ACTIVE / {xcds} XCDs / kernel time |",
             f"| resident waves per CU | {4 * wave / (cycles * cus):.2f} | 4 x SQ_WAVE_CYCLES / (CUs x cycles) |",
             f"| issuing or executing | {share('SQ_ACTIVE_INST_ANY')} | SQ_ACTIVE_INST_ANY / SQ_WAVE_CYCLES |",
             f"| of which vector ALU (MFMA included) | {share('SQ_ACTIVE_INST_VALU')} | SQ_ACTIVE_INST_VALU / SQ_WAVE_CYCLES |",
             f"| of which LDS | {share('SQ_ACTIVE_INST_LDS')} | SQ_ACTIVE_INST_LDS / SQ_WAVE_CYCLES |",
             f"| waiting for its next instruction to issue | {share('SQ_WAIT_INST_ANY')} | SQ_WAIT_INST_ANY / SQ_WAVE_CYCLES |",
             f"| of which an LDS instruction | {share('SQ_WAIT_INST_LDS')} | SQ_WAIT_INST_LDS / SQ_WAVE_CYCLES |",
             f"| waiting for anything else (wait counts, barrier) | {share('SQ_WAIT_ANY')} | SQ_WAIT_ANY / SQ_WAVE_CYCLES |", ""]
    out = os.path.join(ROOT, "profiles", f"{kernel}.{workload}.stalls.md")
    open(out, "w").write("\n".join(lines))
    print(out)


CACHE_COUNTERS = ["GRBM_GUI_ACTIVE", "TCC_HIT_sum", "TCC_MISS_sum"]


def cache_summary(workload: str, d: str, kernel: str = "gateup_kernel", xcds: int = 8):
    """L2 (TCC) hit rate of the kernel from one rocprofv3 --pmc pass of CACHE_COUNTERS
    (<d>/CACHE/run_counter_collection.csv, <d>/CACHE_bench.json), with the matrix-core
    busy share and DRAM traffic of the other passes when present: the three quantities
    of the paper's Table 6 (SM throughput, L2 hit rate, DRAM throughput) read on this GPU."""
    rows = list(csv.DictReader(open(os.path.join(d, "CACHE", "run_counter_collection.csv"))))
    per, dur = {}, {}
    for r in rows:
        if kernel not in r["Kernel_Name"]:
            continue
        c = per.setdefault(r["Dispatch_Id"], {})
        c[r["Counter_Name"]] = c.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
        dur[r["Dispatch_Id"]] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
    ids = sorted(per, key=int)[-2:]
    m = {k: sum(per[i][k] for i in ids) / len(ids) for k in CACHE_COUNTERS}
    us = sum(dur[i] for i in ids) / len(ids)
    bench = json.loads(open(os.path.join(d, "CACHE_bench.json")).read().strip().splitlines()[-1])
    hit = m["TCC_HIT_sum"] / max(1.0, m["TCC_HIT_sum"] + m["TCC_MISS_sum"])
    cmd = (f"cd /tmp && TMPDIR=/tmp rocprofv3 --pmc {' '.join(CACHE_COUNTERS)} --output-format csv -d <out> -o run "
           f"-- python3 <repo>/bench.py --workload {workload} --no-cpu-baseline --no-attainable --steps 3 --warmup-seconds 0.5")
    lines = [f"# {kernel} -- L2 hit rate, workload {bench['config']['workload']} ({workload})", "",
             describe(kernel, workload), "", "Command (one counter pass):", "", "    " + cmd, "",
             "| quantity | value | how it is read |", "|---|---|---|",
             f"| kernel time under the profiler | {us:.1f} us | dispatch timestamps, mean of the pass's last two launches |",
             f"| engine clock | {m['GRBM_GUI_ACTIVE'] / xcds / us / 1e3:.2f} GHz | GRBM_GUI_ACTIVE / {xcds} XCDs / kernel time |",
             f"| L2 requests | {(m['TCC_HIT_sum'] + m['TCC_MISS_sum']) / 1e6:.1f} M | TCC_HIT_sum + TCC_MISS_sum |",
             f"| L2 hit rate | {100 * hit:.1f} % | TCC_HIT_sum / (TCC_HIT_sum + TCC_MISS_sum) |", ""]
    out = os.path.join(ROOT, "profiles", f"{kernel}.{workload}.cache.md")
    open(out, "w").write("\n".join(lines))
    print(out)


def read_summary(d: str, calib: str, workload: str = "mixed512"):
    """The streaming read that sets the measured HBM ceiling (stream_read_kernel, 2 GiB per
    launch, run by bench.py after its timed steps): its kernel-trace average and its
    FETCH_SIZE / WRITE_SIZE per launch, scaled like every traffic figure, which also
    checks that scaling on a kernel whose bytes are known exactly."""
    kernel = "stream_read_kernel"
    stats = list(csv.DictReader(open(os.path.join(d, "trace", "run_kernel_stats.csv"))))
    bench = json.loads(open(os.path.join(d, "trace_bench.json")).read().strip().splitlines()[-1])
    row = [r for r in stats if kernel in r["Name"]][0]
    fetch_kib, nf = counter_per_dispatch(os.path.join(d, "FETCH_SIZE", "run_counter_collection.csv"), kernel, "FETCH_SIZE")
    write_kib, nw = counter_per_dispatch(os.path.join(d, "WRITE_SIZE", "run_counter_collection.csv"), kernel, "WRITE_SIZE")
    mib = 1024
    copy_bytes = mib * 1024 * 1024
    cf, _ = counter_per_dispatch(os.path.join(calib, "FETCH_SIZE", "run_counter_collection.csv"), "UnaryFunctor", "FETCH_SIZE")
    cw, _ = counter_per_dispatch(os.path.join(calib, "WRITE_SIZE", "run_counter_collection.csv"), "UnaryFunctor", "WRITE_SIZE")
    ffac, wfac = copy_bytes / (cf * 1024), copy_bytes / (cw * 1024)
    nbytes = 2 << 30
    tr_us = float(row["AverageNs"]) / 1e3
    att = bench["attainable"]
    cmd = f"bench.py --workload {workload} --secondary none --no-cpu-baseline"
    lines = [f"# {kernel} -- the measured HBM read ceiling (2 GiB per launch)", "",
             "A plain streaming read of a 2 GiB device buffer (ppas_stream_read; each wave reads contiguous 8 KB runs "
             "with nontemporal 16-byte loads, one 256-thread workgroup per CU) on one MI355X (gfx950), launched by "
             "bench.py after its timed steps, alternating between two buffers.", "",
             "## Kernel trace (rocprofv3 --kernel-trace --stats)", "", "Command:", "",
             f"    cd /tmp && TMPDIR=/tmp rocprofv3 --kernel-trace --stats --output-format csv -d <out> -o run -- "
             f"python3 <repo>/{cmd}", "",
             "| kernel | calls | average (us) | min (us) | read rate at the average |", "|---|---|---|---|---|",
             f"| {kernel} | {row['Calls']} | {tr_us:.2f} | {float(row['MinNs']) / 1e3:.2f} | "
             f"{nbytes / (tr_us * 1e-6) / 1e12:.2f} TB/s |", "",
             f"bench.py in the same run, HIP events recorded by the launch: {att['hbm_read_gbps'] / 1e3:.2f} TB/s "
             f"(median of its 20 timed launches), {100 * att['hbm_read_frac_of_spec']:.1f} % of the 8 TB/s spec peak.",
             "", "## HBM traffic (rocprofv3 --pmc, one counter per run)", "", "Commands:", ""]
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        lines.append(f"    cd /tmp && TMPDIR=/tmp rocprofv3 --pmc {c} --output-format csv -d <out> -o run -- "
                     f"python3 <repo>/{cmd} --steps 3 --warmup 1")
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        lines.append(f"    cd /tmp && TMPDIR=/tmp rocprofv3 --pmc {c} --output-format csv -d <out> -o run -- "
                     f"python3 <repo>/paper_2608_15171_amd/calibrate.py --mib {mib}")
    lines += ["", f"Calibration as for the other kernels: bytes = FETCH_SIZE x 1024 x {ffac:.3f} and WRITE_SIZE x 1024 x "
                  f"{wfac:.3f} (a plain copy of {mib} MiB).", "", "| per launch | value |", "|---|---|",
              f"| FETCH_SIZE (KiB, mean of {nf} launches) | {fetch_kib:.0f} |",
              f"| WRITE_SIZE (KiB, mean of {nw} launches) | {write_kib:.0f} |",
              f"| bytes read from memory, scaled | {fetch_kib * 1024 * ffac / 1e9:.3f} GB |",
              f"| bytes the kernel reads | {nbytes / 1e9:.3f} GB |",
              f"| scaled / known | {fetch_kib * 1024 * ffac / nbytes:.3f} |", ""]
    out = os.path.join(ROOT, "profiles", f"{kernel}.read-2GiB.md")
    open(out, "w").write("\n".join(lines))
    print(out)


if __name__ == "__main__":
    if sys.argv[1] == "--read":
        read_summary(*sys.argv[2:4])
    elif sys.argv[1] == "--mfma":
        mfma_summary(*sys.argv[2:4])
    elif sys.argv[1] == "--stalls":
        stall_summary(*sys.argv[2:4])
    elif sys.argv[1] == "--cache":
        cache_summary(*sys.argv[2:4])
    else:
        main(*sys.argv[1:5])
