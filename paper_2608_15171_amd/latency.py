"""Request latencies of a serving trace from measured step times (attention-only view).

P-PAS chooses each iteration's prefill budget so that decoding requests are not held
behind long prefill chunks under prefill pressure (Section 3, Algorithm 1); the paper
reports the effect as time to first token and time per output token of whole-model
serving. This module derives both from the scheduler iterations of a trace and one
measured time per iteration. Here that time is the iteration's attention work
(packed attention launch + page writes, summed over the layers), so the figures are
an attention-only view: the other operators of a decoder block are not in them.

Time model: iterations run back to back; an iteration that launches nothing takes
no time. A request that arrives at iteration a gets its first token at the end of
the iteration that processes its last prompt chunk; each later token comes at the
end of the iteration that holds its decode row, so its time per output token is
the time of that iteration.
"""
from __future__ import annotations

import numpy as np


def request_latencies(requests, steps, step_ms) -> dict:
    """Per-request time to first token and per-token decode latencies.

    requests: objects with req_id, prompt_len, arrival_step; steps: the launched
    iterations in order (index, spec.seqs with req_id, n_query, cached_len); step_ms:
    the measured time of each launched iteration. Returns {req_id: (ttft_ms,
    [token_ms, ...])} for every request whose first token was produced."""
    assert len(steps) == len(step_ms)
    prompt = {r.req_id: r.prompt_len for r in requests}
    arrival = {r.req_id: r.arrival_step for r in requests}
    index = np.array([st.index for st in steps], dtype=np.int64)
    start = np.concatenate([[0.0], np.cumsum(np.asarray(step_ms, dtype=np.float64))])   # start of launched step k
    prefilled = {rid: 0 for rid in prompt}
    out = {}
    for k, st in enumerate(steps):
        end = start[k + 1]
        for s in st.spec.seqs:
            rid = s.req_id
            if s.cached_len >= prompt[rid]:
                # a decode row: one more output token at the end of this iteration
                out[rid][1].append(float(step_ms[k]))
                continue
            prefilled[rid] += s.n_query
            if prefilled[rid] == prompt[rid]:
                # the first launched iteration at or after the arrival starts the clock
                first = int(np.searchsorted(index, arrival[rid]))
                out[rid] = (float(end - start[first]), [])
    return out


def summarize(lat: dict) -> dict:
    """Mean, median and 99th percentile of time to first token (over requests), of
    each request's mean time per output token, and of all token latencies."""
    def stats(x):
        x = np.asarray(x, dtype=np.float64)
        if x.size == 0:
            return None
        return {"mean": round(float(x.mean()), 3), "p50": round(float(np.percentile(x, 50)), 3),
                "p99": round(float(np.percentile(x, 99)), 3)}
    ttft = [v[0] for v in lat.values()]
    tpot = [float(np.mean(v[1])) for v in lat.values() if v[1]]
    tokens = [t for v in lat.values() for t in v[1]]
    return {"requests": len(lat), "ttft_ms": stats(ttft), "tpot_ms": stats(tpot), "token_ms": stats(tokens)}
