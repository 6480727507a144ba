"""The P-PAS prefill budget (Section 3, Algorithm 1).

TEST INFRASTRUCTURE (see the package docstring): the product's step-composition
generator is a separate implementation checked against this one.

Restated: one predicate over the scheduler state decides each iteration. The
state is under prefill pressure when the requests that still have prompt tokens
to process, counted whether their prefill has started or is still queued, are at
least N_th in number, and at the same time some request is generating tokens.
Under pressure the iteration may schedule at most B_cap prefill tokens in total,
otherwise at most B_max. The engine's own per-iteration token budget is a
separate limit that P-PAS leaves as it is, and since the predicate is evaluated
again at every iteration the large budget returns as soon as pressure ends. The
paper evaluates N_th = 2, B_max = 16384, B_cap = 2048 (Section 3; Section 4.3).
"""
from __future__ import annotations

N_TH, B_MAX, B_CAP = 2, 16384, 2048


def under_pressure(prefills_pending: int, decodes_active: int, n_th: int = N_TH) -> bool:
    """The pressure predicate: enough pending prefills while decoding is under way."""
    return prefills_pending >= n_th and decodes_active > 0


def prefill_budget(n_prefill_running: int, n_prefill_waiting: int, n_decode_running: int,
                   n_th: int = N_TH, b_max: int = B_MAX, b_cap: int = B_CAP) -> int:
    """Aggregate prefill-token limit of one iteration."""
    pending = n_prefill_running + n_prefill_waiting
    return b_cap if under_pressure(pending, n_decode_running, n_th) else b_max
