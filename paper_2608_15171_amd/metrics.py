"""Algorithmic work of one mixed step, for roofline accounting.

A row at position p attends to keys 0..p (causal within its chunk, full over the
cached prefix), so a request with n new tokens after c cached ones contributes
n*c + n(n+1)/2 (query row, key) pairs per query head. Each pair costs 2*D FLOP
for QK^T and 2*D for PV (the FlashAttention counting convention; softmax
exponentials are not counted). Bytes count every visible K and V element once
plus Q in and O out, all bf16.
"""
from __future__ import annotations

from .inputs import StepSpec

# MI355X published peaks
PEAK_BF16_FLOPS = 2.5e15      # dense MFMA bf16
PEAK_HBM_BPS = 8.0e12         # HBM3E


def visible_pairs(spec: StepSpec, only=None) -> int:
    tot = 0
    for s in spec.seqs:
        if only == "prefill" and s.n_query == 1:
            continue
        if only == "decode" and s.n_query != 1:
            continue
        tot += s.n_query * s.cached_len + s.n_query * (s.n_query + 1) // 2
    return int(tot)


def flops(spec: StepSpec, only=None) -> float:
    return 4.0 * spec.head_dim * spec.n_q_heads * visible_pairs(spec, only)


def kv_bytes(spec: StepSpec, only=None) -> float:
    toks = 0
    for s in spec.seqs:
        if only == "prefill" and s.n_query == 1:
            continue
        if only == "decode" and s.n_query != 1:
            continue
        toks += s.cached_len + s.n_query
    return float(toks * spec.n_kv_heads * spec.head_dim * 2 * 2)


def attn_bytes(spec: StepSpec) -> float:
    return kv_bytes(spec) + float(2 * spec.n_rows * spec.n_q_heads * spec.head_dim * 2)


def append_bytes(spec: StepSpec) -> float:
    """kv_append traffic: each new K and V row read once and written once."""
    return float(spec.n_rows * spec.n_kv_heads * spec.head_dim * 2 * 2 * 2)


def roofline_time(spec: StepSpec) -> float:
    return max(flops(spec) / PEAK_BF16_FLOPS, attn_bytes(spec) / PEAK_HBM_BPS)
