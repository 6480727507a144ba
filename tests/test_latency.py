"""The latency bookkeeping over a trace (CPU): with every launched iteration taking one
time unit, time to first token counts the launched iterations from arrival through the
last prompt chunk, and every output token after the first takes one unit; a hand-traced
two-request schedule gives the same figures worked out on paper."""
import numpy as np

from paper_2608_15171_amd import latency as LT
from paper_2608_15171_amd import ppas_trace as PT
from paper_2608_15171_amd.inputs import Seq, StepSpec


def test_unit_step_times_count_iterations():
    reqs = PT.bursty_requests(3, n_bursts=3, burst_size=3, mean_gap=5, prompt_range=(300, 900),
                              output_range=(3, 7))
    steps = PT.run_trace(reqs, mode="ppas", mbt=512, b_max=512, b_cap=128)
    lat = LT.request_latencies(reqs, steps, np.ones(len(steps)))
    assert set(lat) == {r.req_id for r in reqs}
    index = [st.index for st in steps]
    for r in reqs:
        ttft, toks = lat[r.req_id]
        last_chunk = max(k for k, st in enumerate(steps)
                         for s in st.spec.seqs if s.req_id == r.req_id and s.cached_len < r.prompt_len)
        first = next(k for k, i in enumerate(index) if i >= r.arrival_step)
        assert ttft == last_chunk - first + 1
        assert toks == [1.0] * (r.output_len - 1)          # the first token comes with the last chunk


def test_hand_traced_schedule():
    """Request 0 (prompt 5, arrives at 0) and request 1 (prompt 3, arrives at 1); a
    budget of 4 prompt tokens per iteration after the decode rows, decodes first.
    Iteration times 2, 3, 5, 7 ms:
      it0: r0 prompt 0..3                     (2 ms)
      it1: r0 prompt 4 (first token), r1 0..2 (first token)   (3 ms)
      it2: r0 decode, r1 decode               (5 ms)
      it3: r1 decode                          (7 ms)
    r0: TTFT 2 + 3 = 5, tokens [5]; r1: TTFT 3 (arrived at it1), tokens [5, 7]."""
    class R:
        def __init__(self, i, p, a):
            self.req_id, self.prompt_len, self.arrival_step = i, p, a

    class S:
        def __init__(self, i, seqs):
            self.index, self.spec = i, StepSpec(f"s{i}", seqs)

    reqs = [R(0, 5, 0), R(1, 3, 1)]
    steps = [S(0, [Seq(4, 0, 0)]), S(1, [Seq(1, 4, 0), Seq(3, 0, 1)]), S(2, [Seq(1, 5, 0), Seq(1, 3, 1)]),
             S(3, [Seq(1, 4, 1)])]
    lat = LT.request_latencies(reqs, steps, [2.0, 3.0, 5.0, 7.0])
    assert lat[0] == (5.0, [5.0]) and lat[1] == (3.0, [5.0, 7.0])
    s = LT.summarize(lat)
    assert s["requests"] == 2 and s["ttft_ms"]["mean"] == 4.0 and s["token_ms"]["p50"] == 5.0
