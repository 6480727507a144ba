"""Request latencies of a bursty serving run in seconds, from per-iteration costs.

The paper evaluates P-PAS on 50 s traces of five 10 s phases that alternate a
steady Poisson arrival rate of 0.2 requests/s with burst phases whose Poisson
rate is swept (Section 4.1, Fig. 2); requests have 25k-token prompts and 32
output tokens in the primary configuration. It reports end-to-end latency
(arrival to the last output token), time to first token (TTFT), time per output
token (TPOT), their means and 95th percentiles, and the makespan (Section 4.4),
for fixed budgets of 2k and 16k tokens and for P-PAS (N_th = 2, 16k / 2k), and
summarises P-PAS against a baseline by the geometric mean over burst rates of
the per-rate ratio of a metric (Section 5.1).

Time model: one engine runs scheduler iterations back to back. At the start of
an iteration, every request whose arrival time has passed joins the scheduler
(first-come first-served by arrival); the iteration's composition follows the
scheduler of ppas_trace (decode rows first, prefill chunks under the budget of
the chosen rule); its duration is cost(spec), the measured time of one full
iteration, and the clock advances by it. With nothing to run, the clock jumps
to the next arrival. A request's first token appears at the end of the iteration
that processes its last prompt chunk, each later token at the end of the
iteration holding its decode row; it completes with its last token. TPOT of a
request with O > 1 outputs is (completion - first token) / (O - 1).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import ppas_trace as PT
from .inputs import StepSpec, rng

PHASE_S, N_PHASES, STEADY_RATE = 10.0, 5, 0.2


@dataclass(frozen=True)
class TimedRequest:
    req_id: int
    prompt_len: int
    output_len: int
    arrival_s: float


def bursty_arrivals(seed: int, burst_rate: float, steady_rate: float = STEADY_RATE, phase_s: float = PHASE_S,
                    n_phases: int = N_PHASES, prompt_len: int = 25000, output_len: int = 32,
                    prompt_range=None, output_range=None) -> list[TimedRequest]:
    """Arrival times of a trace of n_phases phases of phase_s seconds, steady and burst
    phases alternating (steady first); within a phase arrivals are a Poisson process of
    that phase's rate. Prompt and output lengths are fixed, or uniform integers over the
    given ranges."""
    g = rng(seed, 12, int(round(burst_rate * 1000)))
    out, rid = [], 0
    for k in range(n_phases):
        rate = steady_rate if k % 2 == 0 else burst_rate
        t, end = k * phase_s, (k + 1) * phase_s
        while rate > 0:
            t += float(g.exponential(1.0 / rate))
            if t >= end:
                break
            L = int(g.integers(prompt_range[0], prompt_range[1], endpoint=True)) if prompt_range else prompt_len
            O = int(g.integers(output_range[0], output_range[1], endpoint=True)) if output_range else output_len
            out.append(TimedRequest(rid, L, O, t))
            rid += 1
    return out


@dataclass
class SimIteration:
    start_s: float
    duration_s: float
    prefill_tokens: int
    decode_rows: int
    budget: int
    n_prefill: int
    n_decode: int


@dataclass
class SimResult:
    requests: list
    arrival: dict
    first_token: dict
    finish: dict
    iterations: list = field(default_factory=list)


def simulate(requests: list[TimedRequest], cost, mode: str = "ppas", mbt: int = 16384, n_th: int = PT.N_TH,
             b_max: int = PT.B_MAX, b_cap: int = PT.B_CAP, max_iters: int = 1_000_000) -> SimResult:
    """Run the trace; cost(spec) gives the duration in seconds of an iteration whose
    descriptors are spec (a StepSpec with one Seq per request in the iteration)."""
    order = sorted(requests, key=lambda r: (r.arrival_s, r.req_id))
    state = {r.req_id: PT.Request(r.req_id, r.prompt_len, r.output_len, 0) for r in order}
    arrival = {r.req_id: r.arrival_s for r in order}
    res = SimResult(list(order), arrival, {}, {})
    arrived: list = []
    nxt, clock = 0, 0.0
    for _ in range(max_iters):
        while nxt < len(order) and order[nxt].arrival_s <= clock:
            arrived.append(state[order[nxt].req_id])
            nxt += 1
        live = [r for r in arrived if not r.finished]
        if not live:
            if nxt >= len(order):
                return res
            clock = order[nxt].arrival_s
            continue
        seqs, chunks, decodes, budget, n_p, n_d = PT.compose_iteration(live, mode, mbt, n_th, b_max, b_cap)
        spec = StepSpec(f"sim-iter{len(res.iterations)}", seqs)
        dt = float(cost(spec))
        if not (dt > 0.0):
            raise ValueError(f"iteration cost must be positive, got {dt}")
        first, done = PT.apply_iteration(chunks, decodes)
        res.iterations.append(SimIteration(clock, dt, sum(k for _, k in chunks), len(decodes), budget, n_p, n_d))
        clock += dt
        for rid in first:
            res.first_token[rid] = clock
        for rid in done:
            res.finish[rid] = clock
    raise RuntimeError("simulation did not finish within max_iters iterations")


def _stats(x) -> dict | None:
    x = np.asarray(x, dtype=np.float64)
    if x.size == 0:
        return None
    return {"mean": float(x.mean()), "p95": float(np.percentile(x, 95)), "max": float(x.max())}


def summarize(res: SimResult) -> dict:
    """Means and 95th percentiles (seconds) of end-to-end latency, TTFT and TPOT over the
    requests, the makespan (first arrival to last completion) and the iteration count."""
    e2e, ttft, tpot = [], [], []
    for r in res.requests:
        a, f, d = res.arrival[r.req_id], res.first_token[r.req_id], res.finish[r.req_id]
        e2e.append(d - a)
        ttft.append(f - a)
        if r.output_len > 1:
            tpot.append((d - f) / (r.output_len - 1))
    first = min(res.arrival.values())
    return {"requests": len(res.requests), "iterations": len(res.iterations),
            "makespan_s": float(max(res.finish.values()) - first),
            "e2e_s": _stats(e2e), "ttft_s": _stats(ttft), "tpot_s": _stats(tpot)}


def geomean_ratio(ours, base) -> float:
    """The paper's summary of a metric over K burst rates: (prod_k m_ours,k / m_base,k)^(1/K)."""
    a, b = np.asarray(ours, dtype=np.float64), np.asarray(base, dtype=np.float64)
    return float(np.exp(np.mean(np.log(a / b))))
