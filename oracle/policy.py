"""The P-PAS prefill budget (Section 3, Algorithm 1).

TEST INFRASTRUCTURE (see the package docstring): the product's step-composition
generator is a separate implementation checked against this one.

Per scheduler iteration: N_p is the number of running plus waiting prefills and
N_d the number of running decode requests. Prefill pressure is N_p >= N_th while
at least one decode is active; then the aggregate prefill tokens of the
iteration are limited to B_cap, otherwise to B_max. The global token budget of
the engine is not changed, and the decision is taken afresh every iteration.
The evaluated configuration is N_th = 2, B_max = 16384, B_cap = 2048 (Section 3,
Section 4.3).
"""
from __future__ import annotations

N_TH, B_MAX, B_CAP = 2, 16384, 2048


def prefill_budget(n_prefill_running: int, n_prefill_waiting: int, n_decode_running: int,
                   n_th: int = N_TH, b_max: int = B_MAX, b_cap: int = B_CAP) -> int:
    n_p = n_prefill_running + n_prefill_waiting
    n_d = n_decode_running
    if n_p >= n_th and n_d > 0:
        return b_cap
    return b_max
