"""The P-PAS prefill budget and the step-composition generator (CPU only).

Pins: Algorithm 1's truth table and parameters as printed in Section 3 (fixture in
tests/golden), re-evaluation every iteration, conservation of prompt and output
tokens over a trace, and a hand-traced two-request example."""
import json
import os

import pytest

import oracle.policy as OP
from paper_2608_15171_amd import ppas_trace as PT

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "ppas_algorithm1.json")))


def test_parameters_match_paper():
    p = GOLD["parameters"]
    assert (OP.N_TH, OP.B_MAX, OP.B_CAP) == (p["N_th"], p["B_max"], p["B_cap"])
    assert (PT.N_TH, PT.B_MAX, PT.B_CAP) == (p["N_th"], p["B_max"], p["B_cap"])


@pytest.mark.parametrize("row", GOLD["truth_table"])
def test_truth_table(row):
    want = row["B_prefill"]
    assert OP.prefill_budget(row["prefill_running"], row["prefill_waiting"], row["decode_running"]) == want
    assert PT.ppas_budget(row["prefill_running"] + row["prefill_waiting"], row["decode_running"]) == want


def test_generator_budget_agrees_with_oracle_on_grid():
    for n_p in range(0, 6):
        for n_d in range(0, 6):
            assert PT.ppas_budget(n_p, n_d) == OP.prefill_budget(n_p, 0, n_d)


def replay_check(reqs, steps, mbt):
    """Recompute N_p/N_d from the emitted steps alone and check every budget and bound."""
    state = {r.req_id: dict(L=r.prompt_len, O=r.output_len, arr=r.arrival_step, pre=0, gen=0) for r in reqs}
    for st in steps:
        live = [k for k, v in state.items() if v["arr"] <= st.index and not (v["pre"] >= v["L"] and v["gen"] >= v["O"])]
        n_p = sum(1 for k in live if state[k]["pre"] < state[k]["L"])
        n_d = sum(1 for k in live if state[k]["pre"] >= state[k]["L"])
        assert (st.n_prefill, st.n_decode) == (n_p, n_d)
        assert st.prefill_budget == OP.prefill_budget(n_p, 0, n_d)
        pre = sum(s.n_query for s in st.spec.seqs if not (state[s.req_id]["pre"] >= state[s.req_id]["L"]))
        assert pre <= st.prefill_budget
        assert st.spec.n_rows <= mbt
        for s in st.spec.seqs:
            v = state[s.req_id]
            if v["pre"] < v["L"]:
                assert s.cached_len == v["pre"]
                v["pre"] += s.n_query
                if v["pre"] >= v["L"]:
                    v["gen"] = 1
            else:
                assert s.n_query == 1 and s.cached_len == v["L"] + v["gen"] - 1
                v["gen"] += 1
    for v in state.values():
        assert v["pre"] == v["L"] and v["gen"] == v["O"]


def test_trace_conservation_and_budgets():
    reqs = PT.bursty_requests(5, n_bursts=4, burst_size=4, mean_gap=40)
    steps = PT.run_trace(reqs, mode="ppas")
    replay_check(reqs, steps, 16384)
    dec_rows = {}
    for st in steps:
        for s in st.spec.seqs:
            if s.n_query == 1 and s.cached_len >= next(r.prompt_len for r in reqs if r.req_id == s.req_id):
                dec_rows[s.req_id] = dec_rows.get(s.req_id, 0) + 1
    for r in reqs:
        assert dec_rows.get(r.req_id, 0) == r.output_len - 1
    assert any(st.prefill_budget == 2048 for st in steps) and any(st.prefill_budget == 16384 for st in steps)


@pytest.mark.parametrize("mbt", [2048, 16384])
def test_fixed_budget_trace(mbt):
    reqs = PT.bursty_requests(6, n_bursts=3, burst_size=4, mean_gap=30)
    steps = PT.run_trace(reqs, mode="fixed", mbt=mbt)
    for st in steps:
        assert st.spec.n_rows <= mbt


def test_hand_traced_two_requests():
    # A: 20000-token prompt, 3 outputs, arrives at 0. B: 5000-token prompt, 2 outputs, arrives at 1.
    reqs = [PT.Request(0, 20000, 3, 0), PT.Request(1, 5000, 2, 1)]
    steps = PT.run_trace(reqs, mode="ppas")
    got = [(st.index, [(s.req_id, s.n_query, s.cached_len) for s in st.spec.seqs], st.prefill_budget) for st in steps]
    assert got == [
        (0, [(0, 16384, 0)], 16384),                       # N_p=1, N_d=0
        (1, [(0, 3616, 16384), (1, 5000, 0)], 16384),      # N_p=2 but no decode yet: large budget; A and B finish prefill
        (2, [(0, 1, 20000), (1, 1, 5000)], 16384),         # both decode; B is done after this
        (3, [(0, 1, 20001)], 16384),
    ]


def test_pressure_caps_prefill():
    # A decoding while two prefills wait -> cap applies
    reqs = [PT.Request(0, 100, 50, 0), PT.Request(1, 30000, 2, 2), PT.Request(2, 30000, 2, 2)]
    steps = PT.run_trace(reqs, mode="ppas")
    st = next(s for s in steps if s.index == 2)
    assert st.n_prefill == 2 and st.n_decode == 1 and st.prefill_budget == 2048
    assert [(s.req_id, s.n_query) for s in st.spec.seqs] == [(0, 1), (1, 2048)]


# ---------------------------------------------------------------- mutation test
# Plausible misreadings of Algorithm 1 planted in a copy of the oracle; the printed
# truth table must reject each one.

MUTANTS = {
    "strict_threshold": ("return prefills_pending >= n_th and", "return prefills_pending > n_th and"),
    "waiting_prefills_ignored": ("pending = n_prefill_running + n_prefill_waiting", "pending = n_prefill_running"),
    "decodes_ignored": ("prefills_pending >= n_th and decodes_active > 0", "prefills_pending >= n_th"),
    "either_condition": ("prefills_pending >= n_th and decodes_active > 0", "prefills_pending >= n_th or decodes_active > 0"),
    "budgets_swapped": ("return b_cap if under_pressure", "return b_max if under_pressure"),
}


def policy_mutant(name):
    import types
    src = open(OP.__file__).read()
    a, b = MUTANTS[name]
    assert src.count(a) == 1, name
    mod = types.ModuleType("policy_mutant_" + name)
    exec(compile(src.replace(a, b), "<mutant>", "exec"), mod.__dict__)
    return mod


def table_passes(mod) -> bool:
    return all(mod.prefill_budget(r["prefill_running"], r["prefill_waiting"], r["decode_running"]) == r["B_prefill"]
               for r in GOLD["truth_table"])


def test_truth_table_accepts_the_oracle():
    assert table_passes(OP)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_truth_table_rejects_planted_mistake(name):
    assert not table_passes(policy_mutant(name)), f"mutant {name} survived the truth table"
