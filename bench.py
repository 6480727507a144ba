#!/usr/bin/env python3
"""Benchmark of one mixed scheduler step's attention over a paged KV cache on one MI355X.

A step is the whole hot path on one batch: the host plan, ppas_kv_append of the
step's new K/V, and ppas_attn_step (packed attention launch + split merge). Inputs
are seeded synthetic bf16 N(0,1) values at the Qwen2.5-3B attention shape
(16 query heads, 2 KV heads, head_dim 128, pages of 16 tokens, permuted block
table); they are resident in HBM before timing starts. The KV pools rotate over
several device copies so that no timed step finds its keys in the 256 MB
Infinity Cache from the previous step.

Prints ONE JSON line. By default the line is the 16,384-token chunk (the
MBT=16384 step, where prefill work peaks) with the decode-heavy pressure step as
a `secondary` record timed in the same run. `value` is the algorithmic
attention TFLOP/s of the whole step (FLOP = 4 * head_dim * n_q_heads * visible
(row, key) pairs, softmax not counted). `roofline` describes the packed
attention kernel, timed with the HIP events its launch records on its own
stream. `cpu_baseline` times the CPU oracle on a bounded sample of the same
step's rows, with the BLAS pools set to the cores the process may use.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

WORKLOADS = {"mixed512": 1, "mbt2048": 2, "mbt16384": 3, "pressure": 4,
             # diagnostics: parts of the pressure step alone
             "pressure-decode": "pressure-decode", "pressure-prefill": "pressure-prefill",
             # one GPU's shard of the MBT=2048 and pressure steps split two ways by KV head
             "mbt2048-tp2shard": "mbt2048-tp2shard", "pressure-tp2shard": "pressure-tp2shard",
             # 36-layer P-PAS serving trace (64 requests)
             "trace": None,
             # one prompt prefilled as several chunks vs as one chunk
             "chunks": None,
             # rotary embedding fused with the page write, on the new rows of a full-size step
             "rope-mbt2048": ("rope", 2), "rope-mbt16384": ("rope", 3),
             # the trace under P-PAS and under fixed 16k / 2k budgets: request latencies from
             # the measured attention time of every iteration
             "trace-latency": None,
             # the fused gate-up projection of the MLP (hidden 2048 -> 2 x 11008) on a chunk
             # of 16,384 or 2,048 tokens, and one 16k prompt as 8 x 2k chunks vs 1 x 16k
             "gateup-16384": ("gateup", 16384), "gateup-2048": ("gateup", 2048), "gateup-chunks": ("gateup", 0),
             "gateup-act-16384": ("gateup-act", 16384), "gateup-act-2048": ("gateup-act", 2048),
             # request latencies of the paper's bursty trace (seconds-based, steady 0.2 req/s and
             # swept burst rates) under P-PAS and fixed 16k / 2k budgets, every iteration's
             # cost measured on the GPU (one full decoder layer, times 36)
             "serving-sim": None}
METRIC = "mixed-step attn time; prefill TFLOP/s vs MFMA peak; decode KV GB/s vs HBM"
PEAK_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_GBPS = 8000.0     # MI355X HBM3E


KERNEL_SOURCES = ["paper_2608_15171_amd/csrc/attn_step.hip", "paper_2608_15171_amd/csrc/plan.cpp",
                  "paper_2608_15171_amd/csrc/plan.h"]


def measured_traffic(workload: str, kernel: str = "attn_step_kernel"):
    """HBM bytes per launch of a kernel from the committed rocprofv3 byte counters
    (calibrated against a plain copy), or None when no record exists or the kernel
    sources changed since the counters were taken."""
    import hashlib
    root = os.path.dirname(os.path.abspath(__file__))
    path = os.path.join(root, "profiles", f"{kernel}.{workload}.traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    h = hashlib.sha256()
    for src in rec.get("sources", KERNEL_SOURCES):
        h.update(open(os.path.join(root, src), "rb").read())
    if rec.get("kernel_sources_sha256") != h.hexdigest():
        return None
    return rec["fetch_bytes_per_launch"] + rec["write_bytes_per_launch"]


def host_cores() -> int:
    """Cores this process may run on (its affinity mask), not the machine's count."""
    return len(os.sched_getaffinity(0))


def cpu_baseline(data, scale, budget_s: float):
    """Time the oracle on a bounded sample of the step's rows, with the BLAS thread
    pools set to the cores this process may use; returns the JSON object."""
    from threadpoolctl import threadpool_info, threadpool_limits

    cores = host_cores()
    with threadpool_limits(limits=cores, user_api="blas"):
        rec, rows, ref = _cpu_baseline(data, scale, budget_s)
    threads = max([p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"] or [1])
    rec["cores"] = cores
    rec["blas_threads_default"] = int(threads)
    return rec, rows, ref


def _cpu_baseline(data, scale, budget_s: float):
    import oracle.attention as OA
    spec = data.spec
    desc = data.desc

    def sample(frac_rows):
        rows = []
        for s, (qs, n, c) in enumerate(desc.tolist()):
            if n == 1:
                rows.append(qs)
            else:
                k = max(1, int(round(n * frac_rows)))
                rows += list(range(qs + n - k, qs + n))      # the chunk's last rows: the longest ones
        return rows

    def flop(rows):
        pos = {}
        for s, (qs, n, c) in enumerate(desc.tolist()):
            for i in range(n):
                pos[qs + i] = c + i
        return sum(4.0 * spec.head_dim * spec.n_q_heads * (pos[r] + 1) for r in rows)

    frac = 1.0 / 256
    while True:
        rows = sample(frac)
        t0 = time.perf_counter()
        ref = OA.step_attention_from_data(data, scale, rows=rows)
        dt = time.perf_counter() - t0
        if dt >= budget_s / 4 or frac >= 1.0:
            break
        frac = min(1.0, frac * max(2.0, budget_s / 2 / max(dt, 1e-3)))
    f = flop(rows)
    rec = {"value": f / dt / 1e12, "unit": "TFLOP/s", "cores": 0, "kind": "oracle",
           "sample": f"{len(rows)} of {spec.n_rows} query rows (every decode row and the last "
                     f"{frac:.2%} of each prefill chunk), all 16 heads, fp64 NumPy; {f:.3e} FLOP in {dt:.1f} s"}
    return rec, rows, ref


def warm_up(step, args):
    """Untimed warm-up. With --warmup N >= 0, exactly N steps; by default, steps until
    --warmup-seconds of wall time have passed (at least 5 steps). The GPU raises its
    clocks over the first ~50 ms of sustained work after idling, so a warm-up of a few
    short steps would time that ramp instead of the kernel. Returns the step count."""
    import torch
    if args.warmup >= 0:
        for i in range(args.warmup):
            step(i)
        torch.cuda.synchronize()
        return args.warmup
    n, t0 = 0, time.perf_counter()
    while True:
        for _ in range(5):
            step(n)
            n += 1
        torch.cuda.synchronize()
        if time.perf_counter() - t0 >= args.warmup_seconds:
            return n


def attainable_peaks(args):
    """Ceilings measured on this device, beside the spec peaks: the HBM read rate of a plain
    streaming read (ppas_stream_read over two 2 GiB buffers in turn, far past the 256 MB
    Infinity Cache; kernel time from its launch's events) and hipBLASLt's dense bf16 GEMM
    (torch.matmul, 16384 x 16384 x 16384). Medians of the timed calls after a warm-up of
    --warmup-seconds each."""
    import numpy as np
    import torch

    from paper_2608_15171_amd import ppas
    from paper_2608_15171_amd.hip_events import HipEvents

    hip = HipEvents()
    nbytes = 2 << 30
    bufs = [torch.full((nbytes,), i + 1, dtype=torch.uint8, device="cuda") for i in range(2)]
    sink = torch.zeros(4, dtype=torch.int32, device="cuda")
    warm = argparse.Namespace(warmup=-1, warmup_seconds=args.warmup_seconds)
    warm_up(lambda i: ppas.stream_read(bufs[i % 2], sink), warm)
    ev = [(hip.create(), hip.create()) for _ in range(20)]
    for i, (a, b) in enumerate(ev):
        ppas.stream_read(bufs[i % 2], sink, ppas.events(a, b))
    torch.cuda.synchronize()
    read_us = float(np.median([hip.elapsed_ms(a, b) * 1e3 for a, b in ev]))
    for a, b in ev:
        hip.destroy(a)
        hip.destroy(b)
    del bufs, sink
    n = 16384
    g = torch.Generator(device="cuda").manual_seed(0)
    A = torch.randn((n, n), device="cuda", dtype=torch.bfloat16, generator=g)
    B = torch.randn((n, n), device="cuda", dtype=torch.bfloat16, generator=g)
    C = torch.empty((n, n), device="cuda", dtype=torch.bfloat16)
    warm_up(lambda i: torch.matmul(A, B, out=C), warm)
    tev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(10)]
    for a, b in tev:
        a.record()
        torch.matmul(A, B, out=C)
        b.record()
    torch.cuda.synchronize()
    gemm_us = float(np.median([a.elapsed_time(b) * 1e3 for a, b in tev]))
    del A, B, C
    torch.cuda.empty_cache()
    gbps = nbytes / (read_us * 1e-6) / 1e9
    tflops = 2.0 * n ** 3 / (gemm_us * 1e-6) / 1e12
    return {"hbm_read_gbps": round(gbps, 1), "hbm_read_frac_of_spec": round(gbps / PEAK_GBPS, 4),
            "mfma_gemm_tflops": round(tflops, 1), "mfma_gemm_frac_of_spec": round(tflops / PEAK_TFLOPS, 4),
            "read": "ppas_stream_read: 2 GiB contiguous, 16-byte nontemporal loads, two buffers in turn; "
                    f"median of 20 launches, {read_us:.1f} us each",
            "gemm": f"torch.matmul (hipBLASLt) bf16 {n}x{n}x{n}; median of 10 calls, {gemm_us:.0f} us each"}


def measured_ceilings(args):
    """attainable_peaks, or the error that stopped it: the line is printed either way."""
    import torch
    try:
        return attainable_peaks(args)
    except Exception as e:            # a missing library or memory on this device, reported in the line
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        return {"error": f"{type(e).__name__}: {e}"[:300]}


def with_attainable(rec, att):
    """Adds the fraction of the measured ceiling of the record's bound to its roofline."""
    if att is None or "error" in att or "roofline" not in rec:
        return rec
    r = rec["roofline"]
    ceil = att["hbm_read_gbps"] if r["bound"] == "hbm" else att["mfma_gemm_tflops"]
    r["attainable"] = ceil
    r["frac_of_attainable"] = round(r["achieved"] / ceil, 4)
    return rec


def parity_summary(out, ref, rows):
    """Max and mean |GPU - oracle| over the oracle's sample rows of the timed step."""
    import numpy as np
    err = np.abs(out[rows] - ref[rows])
    return {"rows": len(rows), "max_abs": float(err.max()), "mean_abs": float(err.mean()),
            "gate": {"max_abs": 1e-2, "mean_abs": 1e-3}}


def run_trace_workload(args):
    """The 36-layer serving trace: total attention time over every step and layer."""
    import numpy as np
    import torch

    from paper_2608_15171_amd import trace_run as TR

    setup = TR.make_setup(args.seed, mode=args.trace_mode, mbt=args.trace_mbt, layers=args.layers)
    banks = TR.make_banks(args.seed, setup.bank_rows)
    big = max(range(len(setup.steps)), key=lambda i: setup.steps[i].spec.n_rows)
    print(f"trace: {len(setup.steps)} steps x {args.layers} layers, {len(setup.requests)} requests",
          file=sys.stderr, flush=True)
    res = TR.run(setup, banks, args.layers, check=[(big, 0)],
                 progress=lambda i, n: print(f"step {i}/{n}", file=sys.stderr, flush=True))
    t_attn = res["attn_ms_total"] * 1e-3
    rec = {
        "metric": METRIC,
        "value": round(res["flops"] / t_attn / 1e12, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": len(setup.steps),
        "warmup": 0,
        "ms_per_step": round(res["wall_ms"] / len(setup.steps), 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"trace-{len(setup.requests)}req-{args.layers}layers-{args.trace_mode}"
                               + ("" if args.trace_mode == "ppas" else f"{args.trace_mbt}"),
                   "layers": args.layers, "requests": len(setup.requests), "scheduler_steps": len(setup.steps),
                   "prefill_tokens": int(sum(s.prefill_tokens for s in setup.steps)),
                   "decode_rows": int(sum(s.decode_rows for s in setup.steps)),
                   "heads": "16q/2kv", "head_dim": 128, "page_size": 16},
        "trace": {"attention_ms_total": round(res["attn_ms_total"], 3),
                  "kv_append_ms_total": round(res["kv_append_ms_total"], 3),
                  "input_gather_ms_total": round(res["gather_ms_total"], 3),
                  "wall_ms": round(res["wall_ms"], 1), "host_enqueue_ms": round(res["host_enqueue_ms"], 1),
                  "attn_launches": res["launches"],
                  "flop_total": res["flops"], "decode_kv_bytes_total": res["decode_kv_bytes"],
                  "roofline_ms": round(max(res["flops"] / (PEAK_TFLOPS * 1e12),
                                           res["decode_kv_bytes"] / (PEAK_GBPS * 1e9)) * 1e3, 3),
                  "largest_step_rows": setup.steps[big].spec.n_rows},
        "roofline": {"bound": "mfma", "achieved": round(res["flops"] / t_attn / 1e12, 2), "peak": PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(res["flops"] / t_attn / 1e12 / PEAK_TFLOPS, 4),
                     "traffic": None, "kernel": "attn_step_kernel"},
    }
    if not args.no_cpu_baseline:
        data = TR.oracle_inputs(setup, banks, big, 0)
        cb, rows, ref = cpu_baseline(data, 1.0 / math.sqrt(128.0), args.cpu_seconds)
        cb["sample"] = "largest step of the trace, layer 0: " + cb["sample"]
        rec["cpu_baseline"] = cb
        rec["parity"] = parity_summary(res["checks"][(big, 0)].astype(np.float64), ref, rows)
        rec["parity"]["step"] = big
    print(json.dumps(rec), flush=True)


def run_rope_workload(args, cfg):
    """ppas_rope_kv_append on the new rows of a full-size step (rotate Q in place, rotated K
    and plain V into the pages), timed beside ppas_kv_append of the same rows; kernel
    time from events its launch records. HBM-bound: the algorithmic bytes are Q read and
    written once plus the new K/V read once and written once."""
    import numpy as np
    import torch

    from paper_2608_15171_amd import inputs as I
    from paper_2608_15171_amd import ppas
    from paper_2608_15171_amd.hip_events import HipEvents
    from paper_2608_15171_amd.step import DeviceStep, bits_of

    spec = I.CONFIGS[cfg](args.seed)
    data = I.make_step_data(spec, args.seed, with_history=False)
    bt, npages = I.make_block_table(spec, args.seed, permute=True)
    ds = DeviceStep(data, bt, npages)
    theta = args.rope_theta
    # one call on the original rows, kept for the parity sample
    ds.rope_append(theta)
    torch.cuda.synchronize()
    q_rot = bits_of(ds.q)
    hip = HipEvents()
    K = args.steps

    def timed(fn):
        ev = [(hip.create(), hip.create()) for _ in range(K)]
        for i in range(K):
            fn(i, ppas.events(*ev[i]))
        torch.cuda.synchronize()
        t = [hip.elapsed_ms(a, b) * 1e3 for a, b in ev]
        for a, b in ev:
            hip.destroy(a)
            hip.destroy(b)
        return t

    plan = ds.plan(validate=False)
    # (rotates q again each call: norms are kept)
    rope = lambda i, ev=None: plan.rope_kv_append(theta, ds.q, ds.k_pages, ds.v_pages, ds.k_new, ds.v_new,  # noqa: E731
                                                  ds.bt, ev)
    plain = lambda i, ev=None: plan.kv_append(ds.k_pages, ds.v_pages, ds.k_new, ds.v_new, ds.bt, ev)  # noqa: E731
    W = warm_up(rope, args)
    t_rope = timed(rope)
    warm_up(plain, args)
    t_plain = timed(plain)
    plan.close()
    us, us_plain = float(np.median(t_rope)), float(np.median(t_plain))
    T, D = spec.n_rows, spec.head_dim
    B = float(T * (2 * spec.n_q_heads * D * 2 + 2 * 2 * spec.n_kv_heads * D * 2))
    B_plain = float(T * 2 * 2 * spec.n_kv_heads * D * 2)
    gbps = B / (us * 1e-6) / 1e9
    rec = {
        "metric": METRIC,
        "value": round(gbps, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(us * 1e-3, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"rope-append-{spec.name}", "new_rows": T, "rope_theta": theta,
                   "heads": f"{spec.n_q_heads}q/{spec.n_kv_heads}kv", "head_dim": D, "page_size": 16,
                   "block_table": "seeded permutation"},
        "roofline": {"bound": "hbm", "achieved": round(gbps, 2), "peak": PEAK_GBPS, "unit": "GB/s",
                     "frac": round(gbps / PEAK_GBPS, 4), "traffic": measured_traffic(
                         f"rope-mbt{2048 if cfg == 2 else 16384}", kernel="rope_append_kernel"),
                     "kernel": "rope_append_kernel", "kernel_us": round(us, 2), "kernel_us_min": round(min(t_rope), 2),
                     "per_launch": {"bytes": B}},
        "plain_kv_append": {"kernel_us": round(us_plain, 2), "bytes": B_plain,
                            "gbps": round(B_plain / (us_plain * 1e-6) / 1e9, 2)},
    }
    if not args.no_cpu_baseline:
        import oracle.rope as R
        rows = np.arange(T)
        n = min(T, 64)
        t0 = time.perf_counter()
        reps = 0
        while True:
            sample = rows[(reps * n) % T:(reps * n) % T + n]
            R.rotate(R.bf16_bits_to_f64(data.q[sample]), R.row_positions(data.desc)[sample], theta)
            reps += 1
            if time.perf_counter() - t0 >= min(args.cpu_seconds, 5.0):
                break
        dt = time.perf_counter() - t0
        bytes_cpu = reps * n * spec.n_q_heads * D * 2 * 2
        rec["cpu_baseline"] = {"value": round(bytes_cpu / dt / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
                               "sample": f"{reps} x {n} query rows rotated by the fp64 NumPy oracle in {dt:.1f} s"}
        q_ref, _ = R.rope_step(data.q, data.k_new, data.desc, theta)
        x = R.bf16_bits_to_f64(data.q)
        pair = np.abs(x[..., :D // 2]) + np.abs(x[..., D // 2:])
        tol = 2.0 ** -8 * np.abs(q_ref) + 1e-6 * np.concatenate([pair, pair], axis=-1)
        err = np.abs(R.bf16_bits_to_f64(q_rot) - q_ref)
        rec["parity"] = {"rows": int(T), "max_abs": float(err.max()), "within_bound": bool((err <= tol).all()),
                         "bound": "2^-8 |exact| + 1e-6 (|x_i| + |x_(i+64)|) per element"}
    print(json.dumps(rec), flush=True)


def run_gateup_workload(args, T, act=False):
    """ppas_gateup_proj, the MLP's fused gate-up projection Y = X W^T (hidden 2048, 22016
    stacked gate/up rows: the Qwen2.5-3B sizes) on one chunk of T tokens; T = 0 runs one
    16,384-token prompt as eight 2,048-token chunks and as one chunk (Section 6.1,
    Fig. 4b). Weights rotate over four device copies (344 MB, more than the 256 MB
    Infinity Cache), as a layer's weights would be evicted by the other layers' between
    two of its launches. Kernel time from events recorded by the launch. With act, the
    same projection with the gated activation applied in its epilogue (ppas_gateup_act,
    output [T, 11008]); its FLOP count is the projection's."""
    import numpy as np
    import torch

    from paper_2608_15171_amd import inputs as I
    from paper_2608_15171_amd import ppas
    from paper_2608_15171_amd.hip_events import HipEvents
    from paper_2608_15171_amd.step import to_device_bf16

    H, N = I.GATEUP_HIDDEN, 2 * I.GATEUP_INTER
    Tmax = 16384 if T == 0 else T
    xb = I.gateup_tokens(args.seed, Tmax)
    wb = I.gateup_weight(args.seed)
    x = to_device_bf16(xb)
    w0 = to_device_bf16(wb)
    copies = 4
    ws = [w0] + [w0.clone() for _ in range(copies - 1)]
    NO = N // 2 if act else N                     # output columns
    y = torch.empty((Tmax, NO), dtype=torch.bfloat16, device="cuda")
    hip = HipEvents()
    K = args.steps

    wsb = max(ppas.gateup_workspace_bytes(Tmax, H, N), ppas.gateup_workspace_bytes(2048, H, N))
    work = torch.empty(max(wsb, 4), dtype=torch.uint8, device="cuda") if wsb else None
    call = ppas.gateup_act if act else ppas.gateup_proj

    def launch(i, rows=None, ev=None):
        lo, n = (0, Tmax) if rows is None else rows
        call(x[lo:lo + n], ws[i % copies], y[lo:lo + n], work, ev)

    def timed(chunks):
        """Median over K rounds of the summed kernel time of the chunks (us each round)."""
        ev = [[(hip.create(), hip.create()) for _ in chunks] for _ in range(K)]
        for i in range(K):
            for j, c in enumerate(chunks):
                launch(i * len(chunks) + j, c, ppas.events(*ev[i][j]))
        torch.cuda.synchronize()
        per = [[hip.elapsed_ms(a, b) * 1e3 for a, b in e] for e in ev]
        for e in ev:
            for a, b in e:
                hip.destroy(a)
                hip.destroy(b)
        return per

    whole = [(0, Tmax)]
    W = warm_up(lambda i: launch(i), args)
    t_whole = timed(whole)
    us = float(np.median([sum(p) for p in t_whole]))
    F = 2.0 * Tmax * H * N
    B = 2.0 * (Tmax * H + N * H + Tmax * NO)
    tflops = F / (us * 1e-6) / 1e12
    name = "gateup-act" if act else "gateup"
    wl = f"{name}-{Tmax}x{H}x{N}" if T else f"gateup-prompt16384-8x2048-vs-1x16384-{H}x{N}"
    rec = {
        "metric": METRIC, "value": round(tflops, 3), "unit": "TFLOP/s", "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": round(us * 1e-3, 5), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": wl, "tokens": Tmax, "hidden": H, "gate_up_rows": N,
                   "weight_copies_rotated": copies, "activation": "silu(gate) * up" if act else None},
        "roofline": {"bound": "mfma", "achieved": round(tflops, 2), "peak": PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(tflops / PEAK_TFLOPS, 4),
                     "traffic": measured_traffic(f"{name}-{Tmax}", kernel="gateup_kernel"),
                     "kernel": "gateup_kernel", "kernel_us": round(us, 2),
                     "kernel_us_min": round(min(sum(p) for p in t_whole), 2),
                     "per_launch": {"flop": F, "bytes": B}},
    }
    if not args.no_attainable:
        # hipBLASLt on the same projection (the activation, if any, not applied), the same
        # rotated weight copies and the same warm-up, into a buffer of its own
        try:
            yb = torch.empty((Tmax, N), dtype=torch.bfloat16, device="cuda")

            def blas(i):
                torch.matmul(x, ws[i % copies].t(), out=yb)

            warm_up(blas, args)
            tev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
            for i, (a, b) in enumerate(tev):
                a.record()
                blas(i)
                b.record()
            torch.cuda.synchronize()
            blas_us = float(np.median([a.elapsed_time(b) * 1e3 for a, b in tev]))
            del yb
            rec["hipblaslt_same_shape"] = {
                "us": round(blas_us, 2), "tflops": round(F / (blas_us * 1e-6) / 1e12, 2),
                "ours_time_over_hipblaslt": round(us / blas_us, 4),
                "call": f"torch.matmul(x, w.t()) bf16 [{Tmax}, {H}] x [{H}, {N}]" + (", projection only" if act else "")}
        except Exception as e:        # reported in the line; the projection's own figures stand
            torch.cuda.synchronize()
            torch.cuda.empty_cache()
            rec["hipblaslt_same_shape"] = {"error": f"{type(e).__name__}: {e}"[:300]}
        att = measured_ceilings(args)
        rec["attainable"] = att
        with_attainable(rec, att)
    if T == 0:
        chunks = [(2048 * c, 2048) for c in range(8)]
        warm_up(lambda i: launch(i, chunks[i % 8]), args)
        t_ch = timed(chunks)
        per_chunk = np.median(np.array(t_ch), axis=0)
        rec["chunks"] = {"one_16384_us": round(us, 2), "eight_2048_us": round(float(per_chunk.sum()), 2),
                         "ratio_8x2k_over_1x16k": round(float(per_chunk.sum()) / us, 4),
                         "per_chunk_us": [round(float(v), 2) for v in per_chunk],
                         "paper_rtx5090_ms": {"eight_2k": 7.16, "one_16k": 6.66, "ratio": round(7.16 / 6.66, 4),
                                              "note": "one Qwen2.5-3B decoder block on the paper's GPU; context"}}
    if not args.no_cpu_baseline:
        import oracle.gemm as OG
        from threadpoolctl import threadpool_limits
        cores = host_cores()
        n = 16
        with threadpool_limits(limits=cores, user_api="blas"):
            while True:
                rows = np.linspace(0, Tmax - 1, n).astype(np.int64)
                t0 = time.perf_counter()
                if act:
                    ref, gate, up, ag, au = OG.gate_up_act(xb, wb, rows=rows, with_terms=True)
                else:
                    ref, absv = OG.gate_up(xb, wb, rows=rows, with_abs=True)
                dt = time.perf_counter() - t0
                if dt >= args.cpu_seconds / 4 or n >= Tmax:
                    break
                n = min(Tmax, n * max(2, int(args.cpu_seconds / 2 / max(dt, 1e-3))))
        f = 2.0 * len(rows) * H * N
        rec["cpu_baseline"] = {"value": f / dt / 1e12, "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
                               "sample": f"{len(rows)} of {Tmax} token rows, every output column, fp64 NumPy "
                                         f"(operands converted in the timed call); {f:.3e} FLOP in {dt:.1f} s"}
        # parity of the timed launch's output on the same rows
        launch(0)
        torch.cuda.synchronize()
        g = y[torch.from_numpy(rows).cuda()].float().cpu().numpy().astype(np.float64)
        err = np.abs(g - ref)
        if act:
            dg = (1 + 2.0 ** -8) * 2 * H * 2.0 ** -24 * ag
            du = (1 + 2.0 ** -8) * 2 * H * 2.0 ** -24 * au
            D = 1.1 * dg * (np.abs(up) + du) + np.abs(OG.silu(gate)) * du
            bound = (2.0 ** -8 * np.abs(ref) + D + 2.0 ** -24 * (np.abs(gate) + 4) * np.abs(ref)) / (1 - 2.0 ** -8)
            btxt = "(2^-8 |z| + 1.1 d_g (|u| + d_u) + |silu(g)| d_u + 2^-24 (|g| + 4) |z|) / (1 - 2^-8)"
        else:
            bound = 2.0 ** -8 * np.abs(ref) + (1 + 2.0 ** -8) * 2 * H * 2.0 ** -24 * absv
            btxt = "2^-8 |y| + (1 + 2^-8) 2 H 2^-24 sum_k |x_k w_k| per element"
        rec["parity"] = {"rows": int(len(rows)), "max_abs": float(err.max()), "mean_abs": float(err.mean()),
                         "max_err_over_bound": float((err / (bound + 1e-30)).max()), "bound": btxt}
    print(json.dumps(rec), flush=True)


def run_serving_sim_workload(args):
    """The paper's evaluation trace in seconds (Section 4.1, Fig. 2: five 10 s phases,
    steady 0.2 requests/s alternating with a swept burst rate, Poisson arrivals;
    25k-token prompts, 32 outputs) under P-PAS (16,384 / 2,048 by prefill pressure) and
    fixed budgets of 16,384 and 2,048 tokens and the paper's other static budgets (1k, 4k,
    8k; --extra-budgets). Each iteration's duration is measured on the GPU as it
    is scheduled: one decoder layer's kernels (QKV projection, rotary embedding + page
    write, attention, output, gate-up projection with its gated activation, down
    projection) times 36 layers
    (layer_cost.DecoderLayerCost). Reports mean and P95 end-to-end latency, TTFT and TPOT
    per rate and rule, and the paper's geometric-mean ratios of P-PAS to each fixed rule."""
    import numpy as np
    import torch

    from paper_2608_15171_amd import layer_cost as LC
    from paper_2608_15171_amd import serving_sim as S

    rates = [float(x) for x in args.burst_rates.split(",")]
    seeds = list(range(args.seed, args.seed + args.seeds))
    rules = {"ppas": ("ppas", 16384), "fixed16384": ("fixed", 16384), "fixed2048": ("fixed", 2048)}
    # the paper's other static budgets (its appendix table: MBT 1k, 4k, 8k)
    for b in (int(x) for x in args.extra_budgets.split(",") if x):
        rules[f"fixed{b}"] = ("fixed", b)
    # P-PAS with other (B_max, B_cap) pairs under the same global budget: the paper's
    # values define its evaluated configuration, not the policy (Section 3)
    for pair in (x for x in args.ppas_budgets.split(",") if x):
        bm, bc = (int(v) for v in pair.split(":"))
        rules[f"ppas{bm}-{bc}"] = ("ppas", 16384, bm, bc)
    results, parts = {}, {}
    t_start = time.perf_counter()
    from paper_2608_15171_amd.inputs import Seq, StepSpec
    for rate in rates:
        per_seed = {name: [] for name in rules}
        parts[rate] = {}
        for seed in seeds:
            reqs = S.bursty_arrivals(seed, rate)
            cost = LC.DecoderLayerCost(reqs, seed=seed)
            # warm the clocks up on a large iteration before the timed runs
            warm = StepSpec("warm", [Seq(16384, 0, reqs[0].req_id)])
            t0 = time.perf_counter()
            while time.perf_counter() - t0 < args.warmup_seconds:
                cost.layer_ms(warm)
            cost.parts_ms = {k: 0.0 for k in cost.parts_ms}
            for name, (mode, mbt, *bb) in rules.items():
                kw = {"b_max": bb[0], "b_cap": bb[1]} if bb else {}
                res = S.simulate(reqs, cost, mode=mode, mbt=mbt, **kw)
                per_seed[name].append(S.summarize(res))
                print(f"serving-sim rate {rate} seed {seed} {name}: {len(res.iterations)} iterations, mean e2e "
                      f"{per_seed[name][-1]['e2e_s']['mean']:.3f} s ({time.perf_counter() - t_start:.0f} s)",
                      file=sys.stderr, flush=True)
            for k, v in cost.parts_ms.items():
                parts[rate][k] = round(parts[rate].get(k, 0.0) + v, 1)
            cost.close()
            del cost
            torch.cuda.empty_cache()
        # each statistic averaged over the seeds (the paper averages five)
        results[rate] = {}
        for name, runs in per_seed.items():
            avg = {"requests": float(np.mean([r["requests"] for r in runs])),
                   "iterations": float(np.mean([r["iterations"] for r in runs])),
                   "makespan_s": float(np.mean([r["makespan_s"] for r in runs]))}
            for key in ("e2e_s", "ttft_s", "tpot_s"):
                avg[key] = {st: float(np.mean([r[key][st] for r in runs])) for st in ("mean", "p95", "max")}
            results[rate][name] = avg

    def metric(name, key, stat):
        return [results[r][name][key][stat] for r in rates]

    ratios = {}
    for base in ("fixed16384", "fixed2048"):
        ratios[f"ppas_vs_{base}"] = {
            "avg_latency": round(S.geomean_ratio(metric("ppas", "e2e_s", "mean"), metric(base, "e2e_s", "mean")), 4),
            "p95_latency": round(S.geomean_ratio(metric("ppas", "e2e_s", "p95"), metric(base, "e2e_s", "p95")), 4),
            "avg_ttft": round(S.geomean_ratio(metric("ppas", "ttft_s", "mean"), metric(base, "ttft_s", "mean")), 4),
            "avg_tpot": round(S.geomean_ratio(metric("ppas", "tpot_s", "mean"), metric(base, "tpot_s", "mean")), 4)}
    e16, e2 = metric("fixed16384", "e2e_s", "mean"), metric("fixed2048", "e2e_s", "mean")
    better = ["16k" if a < b else "2k" for a, b in zip(e16, e2)]
    fixed = sorted((n for n in rules if n.startswith("fixed")), key=lambda n: rules[n][1])
    best_fixed = [min(fixed, key=lambda n: results[r][n]["e2e_s"]["mean"]) for r in rates]
    for name in rules:
        if name.startswith("ppas") and name != "ppas":
            for base in ("fixed16384", "fixed2048") + tuple(f for f in fixed if f not in ("fixed16384", "fixed2048")):
                ratios[f"{name}_vs_{base}"] = {
                    "avg_latency": round(S.geomean_ratio(metric(name, "e2e_s", "mean"), metric(base, "e2e_s", "mean")), 4),
                    "p95_latency": round(S.geomean_ratio(metric(name, "e2e_s", "p95"), metric(base, "e2e_s", "p95")), 4)}
    ppas_mean = metric("ppas", "e2e_s", "mean")
    rec = {
        "metric": "serving simulation: mean end-to-end request latency under P-PAS (geometric mean over burst rates)",
        "value": round(float(np.exp(np.mean(np.log(ppas_mean)))), 4), "unit": "s", "n_gpus": 1,
        "steps": len(rates), "warmup": 0, "ms_per_step": None, "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "serving-sim-bursty-50s", "phases_s": [10] * 5, "steady_rate": 0.2,
                   "burst_rates": rates, "prompt_tokens": 25000, "output_tokens": 32, "layers": 36,
                   "model_shape": "Qwen2.5-3B (hidden 2048, intermediate 11008, 16q/2kv heads, head_dim 128)",
                   "iteration_cost": "one decoder layer measured per iteration x 36: QKV, rope+page write, "
                                     "attention (+merge), o, gate-up with silu(gate)*up in its epilogue, "
                                     "down; norms, residuals, LM head not included", "seeds": seeds,
                   "budgets": {n: list(v) for n, v in rules.items()}},
        "results": {str(r): {k: {m: (None if v[m] is None else {s: round(x, 4) for s, x in v[m].items()})
                                 if isinstance(v[m], dict) or v[m] is None else v[m]
                                 for m in v} for k, v in results[r].items()} for r in rates},
        "lower_latency_fixed_rule_per_rate": dict(zip([str(r) for r in rates], better)),
        "lowest_latency_fixed_budget_per_rate": dict(zip([str(r) for r in rates], best_fixed)),
        "vs_best_fixed_per_rate": {name: {str(r): round(results[r][name]["e2e_s"]["mean"]
                                                        / results[r][b]["e2e_s"]["mean"], 4)
                                          for r, b in zip(rates, best_fixed)}
                                   for name in rules if name.startswith("ppas")},
        "crossover": better[0] == "16k" and "2k" in better,
        "ratios": ratios,
        "kernel_ms_per_layer_summed": {str(r): parts[r] for r in rates},
        "wall_s": round(time.perf_counter() - t_start, 1),
    }
    print(json.dumps(rec), flush=True)


def run_trace_latency_workload(args):
    """The 36-layer trace under three budget rules (P-PAS: 16,384 / 2,048 by prefill
    pressure; fixed 16,384; fixed 2,048), each run on the GPU. From the measured
    attention + page-write time of every iteration (summed over the layers): the
    total, and per request the time to first token and time per output token in an
    iterations-back-to-back time model (attention-only: no other decoder-block work)."""
    from paper_2608_15171_amd import latency as LT
    from paper_2608_15171_amd import trace_run as TR

    rules = [("ppas", 16384), ("fixed", 16384), ("fixed", 2048)]
    per_rule, flops_ppas, t_ppas = {}, None, None
    banks = None
    for mode, mbt in rules:
        setup = TR.make_setup(args.seed, mode=mode, mbt=mbt, layers=args.layers)
        if banks is None or banks[0].shape[0] < setup.bank_rows:
            banks = TR.make_banks(args.seed, setup.bank_rows)
        name = "ppas" if mode == "ppas" else f"fixed{mbt}"
        print(f"trace-latency: {name}: {len(setup.steps)} steps x {args.layers} layers", file=sys.stderr, flush=True)
        res = TR.run(setup, banks, args.layers)
        lat = LT.summarize(LT.request_latencies(setup.requests, setup.steps, res["step_ms"]))
        per_rule[name] = {"scheduler_steps": len(setup.steps), "attention_ms_total": round(res["attn_ms_total"], 2),
                          "kv_append_ms_total": round(res["kv_append_ms_total"], 2),
                          "attention_tflops": round(res["flops"] / (res["attn_ms_total"] * 1e-3) / 1e12, 2), **lat}
        if mode == "ppas":
            flops_ppas, t_ppas = res["flops"], res["attn_ms_total"]
    achieved = flops_ppas / (t_ppas * 1e-3) / 1e12
    rec = {
        "metric": METRIC,
        "value": round(achieved, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": per_rule["ppas"]["scheduler_steps"],
        "warmup": 0,
        "ms_per_step": round(t_ppas / per_rule["ppas"]["scheduler_steps"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"trace-latency-64req-{args.layers}layers", "layers": args.layers,
                   "budget_rules": [n for n in per_rule], "heads": "16q/2kv", "head_dim": 128, "page_size": 16},
        "latency_attention_only": per_rule,
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_TFLOPS, 4), "traffic": None, "kernel": "attn_step_kernel"},
    }
    print(json.dumps(rec), flush=True)


def run_chunks_workload(args):
    """One prompt prefilled in chunks of --chunk tokens and as a single chunk: the
    attention time of each schedule (kernel time from HIP events, medians)."""
    import numpy as np

    from paper_2608_15171_amd import chunk_replay as CR
    from paper_2608_15171_amd import inputs as I

    P, C = args.prompt, args.chunk
    rp = CR.Replay(P, args.seed)
    n_chunks = P // C
    print(f"chunks: prompt {P} as {n_chunks} x {C} and as 1 x {P}", file=sys.stderr, flush=True)
    def pair(_):
        rp.run(C)
        rp.run(P)
    n_warm = warm_up(pair, args)
    chunked, single = [], []
    for _ in range(args.steps):
        chunked.append(rp.run(C))
        single.append(rp.run(P)[0])
    per_chunk = np.median(np.array(chunked), axis=0)
    t_single = float(np.median(single))
    t_chunked = float(np.median(np.array(chunked).sum(axis=1)))
    F = CR.flops(P)
    achieved = F / (t_single * 1e-3) / 1e12
    rec = {
        "metric": METRIC,
        "value": round(achieved, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": n_warm,
        "ms_per_step": round(t_single, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"prompt{P}-chunk{C}", "prompt_tokens": P, "chunk_tokens": C, "layers": 1,
                   "heads": "16q/2kv", "head_dim": 128, "page_size": 16, "block_table": "seeded permutation"},
        "chunking": {
            "per_chunk_ms": [round(float(x), 4) for x in per_chunk],
            "chunked_total_ms": round(t_chunked, 4),
            "single_chunk_ms": round(t_single, 4),
            "chunked_over_single": round(t_chunked / t_single, 4),
            "chunked_tflops": round(F / (t_chunked * 1e-3) / 1e12, 2),
            "paper_fig4a_ms": {"eight_2k": 7.21, "one_16k": 5.83, "ratio": round(7.21 / 5.83, 4),
                               "note": "FlashAttention of one Qwen2.5-3B decoder block on the paper's GPU; "
                                       "context, not a target"},
        },
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_TFLOPS, 4), "traffic": None, "kernel": "attn_step_kernel",
                     "kernel_us": round(t_single * 1e3, 2), "per_launch": {"flop": F}},
    }
    if not args.no_cpu_baseline:
        q, desc, ks, vs = rp.oracle_inputs()
        spec = I.StepSpec(f"prompt{P}", [I.Seq(P, 0, 0)])
        empty = np.zeros((0, I.HKV, I.HEAD_DIM), dtype=np.uint16)
        data = I.StepData(spec, desc, q, ks[0], vs[0], [empty], [empty])
        rec["cpu_baseline"], rows, ref = cpu_baseline(data, rp.shape.scale, args.cpu_seconds)
        rec["parity"] = parity_summary(rp.out_f64(), ref, rows)
    print(json.dumps(rec), flush=True)


def measure_step(args, workload: str, with_cpu: bool):
    """One single-step workload: K timed whole steps (plan + page write + attention +
    merge), the kernels' own times from the events their launches record, the oracle
    on a bounded sample beside it. Returns the JSON record."""
    import numpy as np
    import torch

    from paper_2608_15171_amd import inputs as I
    from paper_2608_15171_amd import metrics as M
    from paper_2608_15171_amd import ppas
    from paper_2608_15171_amd.hip_events import HipEvents
    from paper_2608_15171_amd.step import DeviceStep

    key = WORKLOADS[workload]
    spec = (I.CONFIGS[key] if isinstance(key, int) else I.DIAGNOSTICS[key])(args.seed)
    print(f"bench: {workload} ({spec.name}, {spec.n_rows} rows)", file=sys.stderr, flush=True)
    data = I.make_step_data(spec, args.seed)
    bt, npages = I.make_block_table(spec, args.seed, permute=True)
    ds = DeviceStep(data, bt, npages)
    ds.fill_history()
    pool_bytes = ds.k_pages.numel() * 2 * 2
    copies = max(2, min(8, math.ceil(1.0e9 / pool_bytes) + 1))
    pools = [(ds.k_pages, ds.v_pages)] + [(ds.k_pages.clone(), ds.v_pages.clone()) for _ in range(copies - 1)]
    probe = ds.plan()
    has_merge = probe.info.n_merge > 0
    tile = int(probe.info.tile_positions)
    n_items = int(probe.info.n_items)
    probe.close()
    torch.cuda.synchronize()

    hip = HipEvents()
    K = args.steps
    ev = [tuple(hip.create() for _ in range(4 if has_merge else 2)) for _ in range(K)]
    ea = [(hip.create(), hip.create()) for _ in range(K)]

    # A step: plan (validation, work list, page-write list), the page write, the
    # attention launch and the split merge. In the timed steps only the attention
    # and merge launches record events (their durations feed the roofline); the
    # page write is timed in a pass of its own afterwards, because every extra
    # event also adds to the step's wall time.
    def one_step(i, events=None, app_events=None):
        ds.k_pages, ds.v_pages = pools[i % copies]
        plan = ds.plan()
        ds.append(plan=plan, events=app_events)
        ds.attend(plan=plan, events=events)
        plan.close()

    W = warm_up(lambda i: one_step(i), args)
    t0 = time.perf_counter()
    for i in range(K):
        one_step(i, events=ppas.events(*ev[i]))
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for i in range(K):
        one_step(i, app_events=ppas.events(*ea[i]))
    torch.cuda.synchronize()

    ms_step = (t1 - t0) / K * 1e3
    attn_ms = [hip.elapsed_ms(e[0], e[1]) for e in ev]
    merge_ms = [hip.elapsed_ms(e[2], e[3]) for e in ev] if has_merge else [0.0] * K
    span_ms = [hip.elapsed_ms(e[0], e[3]) for e in ev] if has_merge else attn_ms
    app_ms = [hip.elapsed_ms(a, b) for a, b in ea]
    for e in ev + ea:
        for x in e:
            hip.destroy(x)
    k_ms = float(np.mean(attn_ms))
    span = float(np.mean(span_ms))

    F = M.flops(spec)
    B = M.attn_bytes(spec)
    t_flop, t_byte = F / (PEAK_TFLOPS * 1e12), B / (PEAK_GBPS * 1e9)
    bound = "mfma" if t_flop >= t_byte else "hbm"
    if bound == "mfma":
        achieved, peak, unit = F / (k_ms * 1e-3) / 1e12, PEAK_TFLOPS, "TFLOP/s"
        step_attn = F / (span * 1e-3) / 1e12
    else:
        achieved, peak, unit = B / (k_ms * 1e-3) / 1e9, PEAK_GBPS, "GB/s"
        step_attn = B / (span * 1e-3) / 1e9

    rec = {
        "metric": METRIC,
        "value": round(F / (ms_step * 1e-3) / 1e12, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": spec.name,
            "layers": 1,
            "requests": [[s.n_query, s.cached_len] for s in spec.seqs] if len(spec.seqs) <= 12 else
                        f"{sum(1 for s in spec.seqs if s.n_query == 1)} decode rows + "
                        f"{[(s.n_query, s.cached_len) for s in spec.seqs if s.n_query > 1]} (n_query, cached_len) chunks",
            "query_rows": spec.n_rows,
            "kv_tokens": int(spec.kv_lens().sum()),
            "heads": f"{spec.n_q_heads}q/{spec.n_kv_heads}kv", "head_dim": 128, "page_size": 16,
            "block_table": "seeded permutation", "kv_pool_copies_rotated": copies,
            "tile_positions": tile, "workgroups": n_items,
        },
        "roofline": {
            "bound": bound, "achieved": round(achieved, 2), "peak": peak, "unit": unit,
            "frac": round(achieved / peak, 4), "traffic": measured_traffic(workload),
            "kernel": "attn_step_kernel", "kernel_us": round(k_ms * 1e3, 2),
            "per_launch": {"flop": F, "bytes": B},
        },
        "breakdown": {
            "attn_kernel_us": round(k_ms * 1e3, 2),
            "attn_kernel_us_min": round(float(np.min(attn_ms)) * 1e3, 2),
            "merge_kernel_us": round(float(np.mean(merge_ms)) * 1e3, 2),
            # from the attention launch's start to the merge launch's end: the whole
            # attention of the step, dispatch gap included
            "attn_with_merge_us": round(span * 1e3, 2),
            "attn_with_merge_frac": round(step_attn / peak, 4),
            "attn_kernel_us_median": round(float(np.median(attn_ms)) * 1e3, 2),
            "kv_append_us": round(float(np.mean(app_ms)) * 1e3, 2),
            "tflops_in_kernel": round(F / (k_ms * 1e-3) / 1e12, 2),
            "mfma_frac": round(F / (k_ms * 1e-3) / 1e12 / PEAK_TFLOPS, 4),
            "kv_gbps_in_kernel": round(M.kv_bytes(spec) / (k_ms * 1e-3) / 1e9, 2),
            "hbm_frac": round(M.kv_bytes(spec) / (k_ms * 1e-3) / 1e9 / PEAK_GBPS, 4),
            "prefill_tflops_in_kernel": round(M.flops(spec, "prefill") / (k_ms * 1e-3) / 1e12, 2),
            "decode_kv_gbps_in_kernel": round(M.kv_bytes(spec, "decode") / (k_ms * 1e-3) / 1e9, 2),
            "step_roofline_us": round(max(t_flop, t_byte) * 1e6, 2),
            # max(F / F_peak, B / B_peak) over the kernel's time: the roofline fraction
            "roofline_frac": round(max(t_flop, t_byte) / (k_ms * 1e-3), 4),
        },
    }
    if with_cpu:
        rec["cpu_baseline"], rows, ref = cpu_baseline(data, ds.shape.scale, args.cpu_seconds)
        rec["parity"] = parity_summary(ds.out_f64(), ref, rows)
    return rec


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=-1,
                    help="untimed warm-up steps; default: as many as fill --warmup-seconds")
    ap.add_argument("--warmup-seconds", type=float, default=0.25)
    ap.add_argument("--workload", choices=sorted(WORKLOADS), default="mbt16384")
    ap.add_argument("--secondary", choices=sorted(k for k, v in WORKLOADS.items() if v is not None
                                                  and not isinstance(v, tuple)) + ["none"], default="pressure",
                    help="a second single-step workload timed in the same run and reported in the same line")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-attainable", action="store_true",
                    help="skip measuring this device's HBM read and bf16 GEMM ceilings")
    ap.add_argument("--layers", type=int, default=36, help="trace workload: layers")
    ap.add_argument("--trace-mode", choices=["ppas", "fixed"], default="ppas", help="trace workload: budget policy")
    ap.add_argument("--trace-mbt", type=int, default=16384, help="trace workload: global token budget")
    ap.add_argument("--prompt", type=int, default=16384, help="chunks workload: prompt tokens")
    ap.add_argument("--chunk", type=int, default=2048, help="chunks workload: tokens per chunk")
    ap.add_argument("--rope-theta", type=float, default=1e6, help="rope workloads: rotary base")
    ap.add_argument("--burst-rates", default="1,2,3,4,5",
                    help="serving-sim workload: burst-phase arrival rates (requests/s)")
    ap.add_argument("--seeds", type=int, default=3, help="serving-sim workload: traces per rate (seeds 0..n-1)")
    ap.add_argument("--extra-budgets", default="1024,4096,8192",
                    help="serving-sim workload: further fixed token budgets beside 2,048 and 16,384")
    ap.add_argument("--ppas-budgets", default="8192:4096,8192:2048,16384:4096",
                    help="serving-sim workload: further P-PAS (B_max:B_cap) pairs beside 16384:2048")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}): the mixed-step attention path has no "
              "multi-GPU mode (a step shards by request or by KV head with no exchange, which is not built)",
              file=sys.stderr)
        sys.exit(2)

    import torch

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.workload == "trace":
        return run_trace_workload(args)
    if args.workload == "chunks":
        return run_chunks_workload(args)
    if args.workload == "trace-latency":
        return run_trace_latency_workload(args)
    if args.workload == "serving-sim":
        return run_serving_sim_workload(args)
    if isinstance(WORKLOADS[args.workload], tuple) and WORKLOADS[args.workload][0] in ("gateup", "gateup-act"):
        return run_gateup_workload(args, WORKLOADS[args.workload][1], act=WORKLOADS[args.workload][0] == "gateup-act")
    if isinstance(WORKLOADS[args.workload], tuple):
        return run_rope_workload(args, WORKLOADS[args.workload][1])
    rec = measure_step(args, args.workload, not args.no_cpu_baseline)
    if args.secondary != "none" and args.secondary != args.workload:
        sec = measure_step(args, args.secondary, not args.no_cpu_baseline)
        rec["secondary"] = {k: sec[k] for k in ("config", "value", "unit", "ms_per_step", "steps", "warmup",
                                                 "roofline", "breakdown", "cpu_baseline", "parity") if k in sec}
    if not args.no_attainable:
        att = measured_ceilings(args)
        rec["attainable"] = att
        with_attainable(rec, att)
        if "secondary" in rec:
            with_attainable(rec["secondary"], att)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
