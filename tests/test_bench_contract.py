"""bench.py's command-line contract: one JSON line with the agreed fields (GPU), and
a clear refusal of more than one GPU (CPU)."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run_bench(*args, timeout=300):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                          timeout=timeout, cwd=ROOT)


def test_more_than_one_gpu_is_refused():
    r = run_bench("--gpus", "2", timeout=60)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


@pytest.mark.gpu
@pytest.mark.parametrize("workload", ["mbt2048", "rope-mbt16384"])
def test_json_line_fields(workload):
    r = run_bench("--workload", workload, "--steps", "3", "--warmup", "3", "--no-cpu-baseline")
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip().startswith("{")]
    assert len(lines) == 1, r.stdout
    rec = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline"):
        assert key in rec, key
    assert rec["n_gpus"] == 1 and rec["steps"] == 3 and rec["warmup"] == 3
    assert rec["value"] > 0 and rec["ms_per_step"] > 0 and rec["higher_is_better"] is True
    assert rec["dtype"] == "bf16" and rec["data"] == "synthetic" and "workload" in rec["config"]
    roof = rec["roofline"]
    for key in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert key in roof, key
    assert roof["bound"] in ("hbm", "mfma") and 0 < roof["frac"] < 1
    assert abs(roof["frac"] - roof["achieved"] / roof["peak"]) < 1e-3


@pytest.mark.gpu
def test_default_line_is_the_16k_chunk_with_the_pressure_step_beside_it():
    """With no workload flags the line is the 16,384-token chunk (where the prefill
    target is quoted) and carries the decode-heavy pressure step as `secondary`, each
    with its own roofline against its own bound."""
    r = run_bench("--steps", "3", "--warmup", "3", "--no-cpu-baseline")
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip().startswith("{")]
    assert len(lines) == 1, r.stdout
    rec = json.loads(lines[0])
    assert rec["config"]["workload"] == "mbt16384-chunk8616"
    assert rec["roofline"]["bound"] == "mfma"
    sec = rec["secondary"]
    assert sec["config"]["workload"] == "pressure-2x1024+48dec"
    assert sec["roofline"]["bound"] == "hbm" and 0 < sec["roofline"]["frac"] < 1
    assert "merge_kernel_us" in sec["breakdown"] and "attn_with_merge_us" in sec["breakdown"]
    # the ceilings measured on the same device, and each record's share of its own
    att = rec["attainable"]
    assert 2000 < att["hbm_read_gbps"] < 8000 and 300 < att["mfma_gemm_tflops"] < 2500
    for r, ceil in ((rec, att["mfma_gemm_tflops"]), (sec, att["hbm_read_gbps"])):
        assert r["roofline"]["attainable"] == ceil
        assert abs(r["roofline"]["frac_of_attainable"] - r["roofline"]["achieved"] / ceil) < 1e-3
        b = r["breakdown"]
        assert b["attn_kernel_us_min"] <= b["attn_kernel_us_median"]
        assert abs(b["roofline_frac"] - b["step_roofline_us"] / b["attn_kernel_us"]) < 2e-3


def _bench_module():
    import importlib.util
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_fraction_of_the_measured_ceiling_follows_the_bound():
    """Each record's roofline gains its achieved rate over the measured ceiling of its own
    bound (the GEMM ceiling for MFMA-bound kernels, the streaming read for HBM-bound ones);
    a ceiling that failed to measure leaves the record as it was."""
    b = _bench_module()
    att = {"hbm_read_gbps": 7200.0, "mfma_gemm_tflops": 1350.0}
    mf = {"roofline": {"bound": "mfma", "achieved": 1147.5}}
    hb = {"roofline": {"bound": "hbm", "achieved": 4500.0}}
    b.with_attainable(mf, att)
    b.with_attainable(hb, att)
    assert mf["roofline"]["attainable"] == 1350.0 and mf["roofline"]["frac_of_attainable"] == 0.85
    assert hb["roofline"]["attainable"] == 7200.0 and hb["roofline"]["frac_of_attainable"] == 0.625
    failed = {"roofline": {"bound": "mfma", "achieved": 1000.0}}
    b.with_attainable(failed, {"error": "RuntimeError: no library"})
    assert failed == {"roofline": {"bound": "mfma", "achieved": 1000.0}}
    assert b.with_attainable({"value": 1}, att) == {"value": 1}
