"""The seconds-based serving simulator (serving_sim): arrival process, time model and
latency bookkeeping, checked with synthetic iteration costs against hand-traced
cases, closed forms and conservation laws (no GPU)."""
import math

import numpy as np
import pytest

from paper_2608_15171_amd import ppas_trace as PT
from paper_2608_15171_amd import serving_sim as S


def test_arrivals_follow_the_phase_structure():
    reqs = S.bursty_arrivals(0, burst_rate=2.0)
    t = np.array([r.arrival_s for r in reqs])
    assert (np.diff(t) >= 0).all() and t.min() >= 0 and t.max() < 50.0
    assert all(r.prompt_len == 25000 and r.output_len == 32 for r in reqs)
    assert [r.req_id for r in reqs] == list(range(len(reqs)))


@pytest.mark.parametrize("seed", range(3))
def test_arrival_counts_match_the_phase_rates(seed):
    # long phases: counts are Poisson with mean rate x phase length; allow 5 sigma
    reqs = S.bursty_arrivals(seed, burst_rate=1.0, steady_rate=0.2, phase_s=1000.0)
    t = np.array([r.arrival_s for r in reqs])
    for k in range(5):
        n = int(((t >= 1000.0 * k) & (t < 1000.0 * (k + 1))).sum())
        mean = 1000.0 * (0.2 if k % 2 == 0 else 1.0)
        assert abs(n - mean) <= 5 * math.sqrt(mean), (k, n, mean)


def test_length_ranges():
    reqs = S.bursty_arrivals(1, 3.0, prompt_range=(20000, 30000), output_range=(16, 64))
    assert all(20000 <= r.prompt_len <= 30000 and 16 <= r.output_len <= 64 for r in reqs)


def test_single_request_constant_cost():
    # 5000-token prompt at a fixed 2,048-token budget: 3 prefill iterations, then
    # O - 1 = 3 decode iterations, each of cost c, starting at the arrival time
    c = 0.01
    r = S.TimedRequest(0, 5000, 4, 1.0)
    res = S.simulate([r], lambda spec: c, mode="fixed", mbt=2048)
    assert len(res.iterations) == 6 and res.iterations[0].start_s == 1.0
    assert res.first_token[0] == pytest.approx(1.0 + 3 * c)
    assert res.finish[0] == pytest.approx(1.0 + 6 * c)
    s = S.summarize(res)
    assert s["ttft_s"]["mean"] == pytest.approx(3 * c)
    assert s["e2e_s"]["mean"] == pytest.approx(6 * c)
    assert s["tpot_s"]["mean"] == pytest.approx(c)


def cost_model(spec):
    pre = sum(q.n_query for q in spec.seqs if q.n_query > 1 or q.cached_len == 0)
    dec = len(spec.seqs) - sum(1 for q in spec.seqs if q.n_query > 1 or q.cached_len == 0)
    return 0.001 + 1e-6 * pre + 1e-4 * dec


def test_hand_traced_two_requests_under_ppas():
    """A (20,000 prompt, 3 outputs) at 0 and B (3,000, 2) at 5 ms, cost 1 ms + 1 us per
    prefill token + 0.1 ms per decode row:
      it1 @0:        A alone, no decode -> budget 16,384: A 16,384      -> 17.384 ms
      it2 @17.384:   A, B prefills, no decode -> 16,384: A 3,616, B 3,000 -> 25.000 ms
                     (A and B first tokens)
      it3 @25.000:   two decode rows                                      -> 26.200 ms (B done)
      it4 @26.200:   one decode row                                       -> 27.300 ms (A done)"""
    reqs = [S.TimedRequest(0, 20000, 3, 0.0), S.TimedRequest(1, 3000, 2, 0.005)]
    res = S.simulate(reqs, cost_model, mode="ppas")
    assert [(it.prefill_tokens, it.decode_rows) for it in res.iterations] == [(16384, 0), (6616, 0), (0, 2), (0, 1)]
    assert res.first_token[0] == pytest.approx(0.025) and res.first_token[1] == pytest.approx(0.025)
    assert res.finish[1] == pytest.approx(0.0262) and res.finish[0] == pytest.approx(0.0273)
    s = S.summarize(res)
    assert s["e2e_s"]["mean"] == pytest.approx((0.0273 + 0.0212) / 2)
    assert s["tpot_s"]["mean"] == pytest.approx((0.00115 + 0.0012) / 2)
    assert s["makespan_s"] == pytest.approx(0.0273)


def test_pressure_caps_the_prefill_budget():
    """A decoding request and two waiting prefills: Algorithm 1 caps prefill at 2,048."""
    reqs = [S.TimedRequest(0, 1000, 10, 0.0), S.TimedRequest(1, 9000, 2, 0.0005),
            S.TimedRequest(2, 9000, 2, 0.0006)]
    res = S.simulate(reqs, lambda spec: 0.001, mode="ppas")
    it = res.iterations[1]      # A decodes, B and C wait
    assert (it.n_prefill, it.n_decode, it.budget, it.prefill_tokens) == (2, 1, 2048, 2048)
    res16 = S.simulate(reqs, lambda spec: 0.001, mode="fixed", mbt=16384)
    assert res16.iterations[1].prefill_tokens == 16384 - 1


def test_idle_gap_jumps_to_the_next_arrival():
    reqs = [S.TimedRequest(0, 100, 2, 0.0), S.TimedRequest(1, 100, 2, 7.5)]
    res = S.simulate(reqs, lambda spec: 0.01, mode="ppas")
    starts = [it.start_s for it in res.iterations]
    assert starts == pytest.approx([0.0, 0.01, 7.5, 7.51])


@pytest.mark.parametrize("mode,mbt", [("ppas", 16384), ("fixed", 2048), ("fixed", 16384)])
def test_conservation_and_monotone_clock(mode, mbt):
    reqs = S.bursty_arrivals(4, burst_rate=3.0, prompt_range=(2000, 9000), output_range=(2, 12))
    res = S.simulate(reqs, cost_model, mode=mode, mbt=mbt)
    assert set(res.finish) == {r.req_id for r in reqs}
    assert sum(it.prefill_tokens for it in res.iterations) == sum(r.prompt_len for r in reqs)
    assert sum(it.decode_rows for it in res.iterations) == sum(r.output_len - 1 for r in reqs)
    for a, b in zip(res.iterations, res.iterations[1:]):
        assert b.start_s >= a.start_s + a.duration_s - 1e-12
    for r in reqs:
        assert res.arrival[r.req_id] <= res.first_token[r.req_id] <= res.finish[r.req_id]
    for it in res.iterations:
        assert it.prefill_tokens + it.decode_rows <= mbt
        if mode == "ppas" and it.n_prefill >= PT.N_TH and it.n_decode > 0:
            assert it.prefill_tokens <= PT.B_CAP


def test_geomean_ratio():
    assert S.geomean_ratio([1, 4], [2, 2]) == pytest.approx(1.0)
    assert S.geomean_ratio([1, 1, 1], [2, 2, 2]) == pytest.approx(0.5)


def test_mbt_crossover_with_a_chunk_efficiency_cost_model():
    """A cost model with the two effects of Section 2 (a large chunk processes prompt
    tokens more efficiently; an iteration holds its decode rows until it ends): at a low
    burst rate the 16k budget gives lower mean latency than 2k, at a high rate 2k wins,
    and P-PAS is never worse than the worse fixed budget."""
    def cost(spec):
        # prompt tokens cost ~10 % more per token in a 2k iteration than in a 16k one
        # (the kernel-level gap of Section 6.1); a fixed per-iteration cost; cheap decode rows
        P = sum(q.n_query for q in spec.seqs if q.n_query > 1)
        dec = sum(1 for q in spec.seqs if q.n_query == 1)
        return 0.003 + 8e-6 * P * (1.0 + 256.0 / (P + 256.0)) + 2e-5 * dec
    out = {}
    for rate in (0.3, 5.0):
        reqs = S.bursty_arrivals(0, rate)
        out[rate] = {k: S.summarize(S.simulate(reqs, cost, mode=m, mbt=b))["e2e_s"]["mean"]
                     for k, (m, b) in {"16k": ("fixed", 16384), "2k": ("fixed", 2048), "ppas": ("ppas", 16384)}.items()}
    assert out[0.3]["16k"] < out[0.3]["2k"]
    assert out[5.0]["2k"] < out[5.0]["16k"]
    for rate in out:
        assert out[rate]["ppas"] <= max(out[rate]["16k"], out[rate]["2k"]) + 1e-9


@pytest.mark.parametrize("b_max,b_cap", [(8192, 4096), (16384, 4096), (8192, 2048)])
def test_other_budget_pairs_bound_every_iteration(b_max, b_cap):
    """P-PAS with other (B_max, B_cap) pairs under the 16,384-token global budget: no
    iteration schedules more prefill tokens than B_max, and under pressure (at least
    N_th prefills and a decode) none more than B_cap; both budgets are used."""
    reqs = S.bursty_arrivals(2, burst_rate=20.0, prompt_range=(4000, 12000), output_range=(2, 12))
    res = S.simulate(reqs, lambda spec: 5 * cost_model(spec), mode="ppas", mbt=16384, b_max=b_max, b_cap=b_cap)
    assert set(res.finish) == {r.req_id for r in reqs}
    for it in res.iterations:
        assert it.prefill_tokens <= b_max
        if it.n_prefill >= PT.N_TH and it.n_decode > 0:
            assert it.budget == b_cap and it.prefill_tokens <= b_cap
        else:
            assert it.budget == b_max
    assert {it.budget for it in res.iterations} == {b_max, b_cap}
