"""Step compositions of a multi-request serving trace under P-PAS or a fixed token budget.

This is host logic only: it decides which requests contribute which tokens to each
scheduler iteration, and emits one StepSpec (the (n_query, cached_len) descriptors)
per iteration for the attention path to run.

Policy (Section 3, Algorithm 1): at every iteration, N_p counts the running plus
waiting prefills and N_d the running decode requests; when N_p >= N_th and N_d > 0
the aggregate prefill tokens are limited to B_cap, otherwise to B_max. The engine's
global per-iteration token budget stays as configured. The evaluated setting is
N_th = 2, B_max = 16384, B_cap = 2048. Fixed-budget baselines (Section 4.3) use
the same machinery with one budget.

Scheduling rules the paper leaves to the engine, as read here:
  * decode first: every running decode request gets one token in each iteration,
    and prefill chunks fill what remains of the budget (stall-free batching of
    the related work in Section 7);
  * prefill chunks are handed out first-come first-served, running prefills before
    waiting ones, several requests per iteration if the budget allows;
  * a request whose last prompt chunk runs in an iteration produces its first
    output token there; each later output token takes one decode iteration, so a
    request with O output tokens needs O - 1 decode iterations;
  * arrivals are given as iteration indices; iterations with nothing to run are
    skipped (they launch nothing).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from .inputs import Seq, StepSpec, rng

N_TH, B_MAX, B_CAP = 2, 16384, 2048


@dataclass
class Request:
    req_id: int
    prompt_len: int
    output_len: int
    arrival_step: int
    prefilled: int = 0          # prompt tokens already processed
    generated: int = 0          # output tokens produced so far

    @property
    def in_prefill(self) -> bool:
        return self.prefilled < self.prompt_len

    @property
    def finished(self) -> bool:
        return not self.in_prefill and self.generated >= self.output_len


@dataclass
class TraceStep:
    index: int                  # scheduler iteration index
    spec: StepSpec
    n_prefill: int              # N_p seen by the policy
    n_decode: int               # N_d seen by the policy
    prefill_budget: int
    prefill_tokens: int = 0
    decode_rows: int = 0
    completed: list = field(default_factory=list)


def ppas_budget(n_p: int, n_d: int, n_th: int = N_TH, b_max: int = B_MAX, b_cap: int = B_CAP) -> int:
    """Algorithm 1: the small cap under prefill pressure with active decodes, else the large budget."""
    under_pressure = (n_p >= n_th) and (n_d > 0)
    return b_cap if under_pressure else b_max


def bursty_requests(seed: int, n_bursts: int = 16, burst_size: int = 4, mean_gap: float = 160.0,
                    prompt_range=(20000, 30000), output_range=(16, 64)) -> list[Request]:
    """Requests arriving in bursts at iteration indices; burst gaps are ceil(Exp(mean_gap)),
    the first burst at iteration 0. Prompt and output lengths are uniform integers."""
    g = rng(seed, 11)
    reqs, t, rid = [], 0, 0
    for b in range(n_bursts):
        if b > 0:
            t += int(np.ceil(g.exponential(mean_gap)))
        for _ in range(burst_size):
            L = int(g.integers(prompt_range[0], prompt_range[1], endpoint=True))
            O = int(g.integers(output_range[0], output_range[1], endpoint=True))
            reqs.append(Request(rid, L, O, t))
            rid += 1
    return reqs


def compose_iteration(live: list[Request], mode: str = "ppas", mbt: int = 16384, n_th: int = N_TH,
                      b_max: int = B_MAX, b_cap: int = B_CAP):
    """One scheduler iteration over the live (arrived, unfinished) requests, in arrival
    order: returns (seqs, chunks, decodes, budget, n_p, n_d) with seqs the iteration's
    descriptors (decode rows first), chunks the (request, tokens) prefill pieces and
    decodes the requests given one decode token. Does not change the requests.

    mode "ppas": prefill budget from Algorithm 1 under a global budget of mbt tokens.
    mode "fixed": prefill budget is simply what mbt leaves after the decode tokens."""
    prefills = [r for r in live if r.in_prefill]
    decodes = [r for r in live if not r.in_prefill]
    n_p, n_d = len(prefills), len(decodes)
    if mode == "ppas":
        budget = ppas_budget(n_p, n_d, n_th, b_max, b_cap)
    elif mode == "fixed":
        budget = mbt
    else:
        raise ValueError(mode)
    seqs: list[Seq] = []
    for r in decodes:
        # the token generated last iteration is fed back at position L + g - 1
        seqs.append(Seq(1, r.prompt_len + r.generated - 1, r.req_id))
    room = min(budget, mbt - len(decodes))
    # running prefills (already started) before waiting ones, each first-come first-served
    order = [r for r in prefills if r.prefilled > 0] + [r for r in prefills if r.prefilled == 0]
    chunks = []
    for r in order:
        if room <= 0:
            break
        take = min(r.prompt_len - r.prefilled, room)
        chunks.append((r, take))
        room -= take
    for r, take in chunks:
        seqs.append(Seq(take, r.prefilled, r.req_id))
    return seqs, chunks, decodes, budget, n_p, n_d


def apply_iteration(chunks, decodes) -> tuple[list, list]:
    """Advance the requests by one executed iteration. Returns (first_token, completed):
    the ids of requests that produced their first output token (last prompt chunk) and
    of those that finished, in this iteration."""
    first, completed = [], []
    for r in decodes:
        r.generated += 1
        if r.finished:
            completed.append(r.req_id)
    for r, take in chunks:
        r.prefilled += take
        if not r.in_prefill:
            r.generated = 1
            first.append(r.req_id)
            if r.finished:
                completed.append(r.req_id)
    return first, completed


def run_trace(requests: list[Request], mode: str = "ppas", mbt: int = 16384,
              n_th: int = N_TH, b_max: int = B_MAX, b_cap: int = B_CAP,
              max_steps: int = 10_000_000) -> list[TraceStep]:
    """Simulate the scheduler over iteration-indexed arrivals and return the non-empty
    iterations in order (modes as in compose_iteration)."""
    reqs = sorted((Request(r.req_id, r.prompt_len, r.output_len, r.arrival_step) for r in requests),
                  key=lambda r: (r.arrival_step, r.req_id))
    arrived: list[Request] = []
    nxt = 0
    steps: list[TraceStep] = []
    t = 0
    while (nxt < len(reqs) or any(not r.finished for r in arrived)) and t < max_steps:
        while nxt < len(reqs) and reqs[nxt].arrival_step <= t:
            arrived.append(reqs[nxt])
            nxt += 1
        live = [r for r in arrived if not r.finished]
        if not live:
            t = reqs[nxt].arrival_step
            continue
        seqs, chunks, decodes, budget, n_p, n_d = compose_iteration(live, mode, mbt, n_th, b_max, b_cap)
        step = TraceStep(t, StepSpec(f"trace-step{t}", seqs), n_p, n_d, budget,
                         prefill_tokens=sum(k for _, k in chunks), decode_rows=len(decodes))
        _, step.completed = apply_iteration(chunks, decodes)
        steps.append(step)
        t += 1
    return steps
