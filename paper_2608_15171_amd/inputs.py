"""Seeded synthetic inputs for one mixed scheduler step.

This module draws random numbers and integer structure only: bf16 bit
patterns for Q and K/V, the per-request descriptors (query_start, n_query,
cached_len) and physical-page block tables. It holds none of the attention
arithmetic and none of the page-scatter rules; the GPU path and the CPU oracle
both consume what it returns.

Value recipe: every tensor is float32 standard normal from NumPy's PCG64,
rounded to bf16 by round-to-nearest-even on the bit pattern, so both sides see
identical bf16 bits. Every stream is keyed by (seed, kind, request id), so a
request's data does not depend on which other requests share the step or on
the order of the descriptors.

Workload shapes follow the paper's long-context setting (prompts of 20k-30k
tokens, short outputs; Sections 4.1-4.2) at the attention shape of a
Qwen2.5-3B layer: 16 query heads, 2 KV heads, head_dim 128, pages of 16
tokens.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

HQ, HKV, HEAD_DIM, PAGE = 16, 2, 128, 16

# stream kinds
_Q, _KH, _VH, _KN, _VN, _LEN, _PAGES = 1, 2, 3, 4, 5, 6, 7


def rng(seed: int, *key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(seed), *map(int, key)])))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even) and return the uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def normal_bf16(g: np.random.Generator, shape) -> np.ndarray:
    return f32_to_bf16_bits(g.standard_normal(size=shape, dtype=np.float32))


@dataclass(frozen=True)
class Seq:
    """One request's share of a step: n_query new tokens after cached_len cached ones."""
    n_query: int
    cached_len: int
    req_id: int


@dataclass
class StepSpec:
    name: str
    seqs: list[Seq]
    n_q_heads: int = HQ
    n_kv_heads: int = HKV
    head_dim: int = HEAD_DIM
    page_size: int = PAGE
    info: dict = field(default_factory=dict)

    @property
    def n_rows(self) -> int:
        return sum(s.n_query for s in self.seqs)

    def descriptors(self) -> np.ndarray:
        """int32 [S, 3] rows of (query_start, n_query, cached_len); query_start packs rows contiguously."""
        d = np.zeros((len(self.seqs), 3), dtype=np.int32)
        qs = 0
        for i, s in enumerate(self.seqs):
            d[i] = (qs, s.n_query, s.cached_len)
            qs += s.n_query
        return d

    def kv_lens(self) -> np.ndarray:
        return np.array([s.cached_len + s.n_query for s in self.seqs], dtype=np.int64)

    def pages_per_seq(self) -> np.ndarray:
        return (self.kv_lens() + self.page_size - 1) // self.page_size


# ---------------------------------------------------------------------------
# The four single-step workloads (one layer each). Decode rows come first in the
# descriptor array, prefill chunks after them; row order never changes a result.
# ---------------------------------------------------------------------------

def config_small(seed: int = 0) -> StepSpec:
    """512-token prefill chunk at cached_len 0 plus 4 decode rows at cached context 1024."""
    seqs = [Seq(1, 1024, i) for i in range(4)] + [Seq(512, 0, 4)]
    return StepSpec("mixed-512+4dec", seqs)


def config_small_budget(seed: int = 0) -> StepSpec:
    """MBT=2048 step: the 2048-token chunk at offset 22,528 of a 25,000-token prompt plus 8
    decode rows with cached contexts uniform in 25,000..25,032."""
    g = rng(seed, _LEN)
    ctx = g.integers(25000, 25032, size=8, endpoint=True)
    seqs = [Seq(1, int(c), i) for i, c in enumerate(ctx)] + [Seq(2048, 22528, 8)]
    return StepSpec("mbt2048-chunk22528+8dec", seqs)


def config_large_budget(seed: int = 0) -> StepSpec:
    """MBT=16384 low-pressure step: one 16,384-token chunk at offset 8,616 (ends at 25,000)."""
    return StepSpec("mbt16384-chunk8616", [Seq(16384, 8616, 0)])


def config_high_pressure(seed: int = 0) -> StepSpec:
    """2048-token budget under pressure: 2 chunks of 1,024 tokens at seeded offsets inside
    prompts of 20k..30k tokens, plus 48 decode rows with contexts uniform in 20,000..30,064."""
    g = rng(seed, _LEN)
    plen = g.integers(20000, 30000, size=2, endpoint=True)
    off = [int(g.integers(0, int(L) - 1024, endpoint=True)) for L in plen]
    ctx = g.integers(20000, 30064, size=48, endpoint=True)
    seqs = [Seq(1, int(c), i) for i, c in enumerate(ctx)]
    seqs += [Seq(1024, off[k], 48 + k) for k in range(2)]
    return StepSpec("pressure-2x1024+48dec", seqs, info={"prompt_lens": [int(x) for x in plen]})


def config_pressure_decode_only(seed: int = 0) -> StepSpec:
    """Diagnostic: only the 48 decode rows of the high-pressure step."""
    full = config_high_pressure(seed)
    return StepSpec("pressure-48dec-only", [s for s in full.seqs if s.n_query == 1])


def config_pressure_prefill_only(seed: int = 0) -> StepSpec:
    """Diagnostic: only the two 1,024-token chunks of the high-pressure step."""
    full = config_high_pressure(seed)
    return StepSpec("pressure-2x1024-only", [s for s in full.seqs if s.n_query > 1])


def tp2_shard(spec: StepSpec) -> StepSpec:
    """One GPU's half of a step split two ways by KV head: query heads 8k..8k+7 and
    KV head k (8 query heads, 1 KV head, the same requests and lengths)."""
    return StepSpec(spec.name + "-tp2shard", spec.seqs, n_q_heads=spec.n_q_heads // 2,
                    n_kv_heads=spec.n_kv_heads // 2, head_dim=spec.head_dim, page_size=spec.page_size,
                    info=dict(spec.info))


def config_small_budget_tp2(seed: int = 0) -> StepSpec:
    """Diagnostic: the KV-head-split shard of the MBT=2048 step."""
    return tp2_shard(config_small_budget(seed))


def config_high_pressure_tp2(seed: int = 0) -> StepSpec:
    """Diagnostic: the KV-head-split shard of the high-pressure step."""
    return tp2_shard(config_high_pressure(seed))


CONFIGS = {
    1: config_small,
    2: config_small_budget,
    3: config_large_budget,
    4: config_high_pressure,
}

DIAGNOSTICS = {
    "pressure-decode": config_pressure_decode_only,
    "pressure-prefill": config_pressure_prefill_only,
    "mbt2048-tp2shard": config_small_budget_tp2,
    "pressure-tp2shard": config_high_pressure_tp2,
}


# ---------------------------------------------------------------------------
# Tensors
# ---------------------------------------------------------------------------

@dataclass
class StepData:
    spec: StepSpec
    desc: np.ndarray          # int32 [S, 3]
    q: np.ndarray             # uint16 bf16 bits [T, Hq, D]
    k_new: np.ndarray         # uint16 [T, Hkv, D]
    v_new: np.ndarray         # uint16 [T, Hkv, D]
    k_hist: list              # per sequence uint16 [cached_len, Hkv, D]
    v_hist: list


def seq_history(seed: int, seq: Seq, n_kv_heads: int = HKV, head_dim: int = HEAD_DIM):
    """The request's cached K and V rows (positions 0..cached_len-1)."""
    shape = (seq.cached_len, n_kv_heads, head_dim)
    return normal_bf16(rng(seed, _KH, seq.req_id), shape), normal_bf16(rng(seed, _VH, seq.req_id), shape)


def seq_new(seed: int, seq: Seq, n_q_heads: int = HQ, n_kv_heads: int = HKV, head_dim: int = HEAD_DIM):
    """The step's Q rows and new K/V rows for one request (positions cached_len..cached_len+n-1)."""
    n = seq.n_query
    q = normal_bf16(rng(seed, _Q, seq.req_id), (n, n_q_heads, head_dim))
    k = normal_bf16(rng(seed, _KN, seq.req_id), (n, n_kv_heads, head_dim))
    v = normal_bf16(rng(seed, _VN, seq.req_id), (n, n_kv_heads, head_dim))
    return q, k, v


def make_step_data(spec: StepSpec, seed: int, with_history: bool = True) -> StepData:
    desc = spec.descriptors()
    T = spec.n_rows
    q = np.empty((T, spec.n_q_heads, spec.head_dim), dtype=np.uint16)
    kn = np.empty((T, spec.n_kv_heads, spec.head_dim), dtype=np.uint16)
    vn = np.empty_like(kn)
    kh, vh = [], []
    for i, s in enumerate(spec.seqs):
        qs, n = int(desc[i, 0]), int(desc[i, 1])
        q[qs:qs + n], kn[qs:qs + n], vn[qs:qs + n] = seq_new(seed, s, spec.n_q_heads, spec.n_kv_heads, spec.head_dim)
        if with_history:
            a, b = seq_history(seed, s, spec.n_kv_heads, spec.head_dim)
        else:
            a = b = None
        kh.append(a)
        vh.append(b)
    return StepData(spec, desc, q, kn, vn, kh, vh)


def make_block_table(spec: StepSpec, seed: int, permute: bool = True, spare_pages: int = 0):
    """Per-request logical page -> physical page table.

    The pool has sum(ceil(kv_len/16)) + spare_pages pages. With permute, one seeded
    permutation of the pool is cut into consecutive slices, one per request; without
    it, requests get consecutive pages in descriptor order. Unused entries are -1.
    Returns (table int32 [S, stride], num_pages).
    """
    need = spec.pages_per_seq()
    total = int(need.sum()) + int(spare_pages)
    order = rng(seed, _PAGES).permutation(total) if permute else np.arange(total)
    stride = max(1, int(need.max()) if len(need) else 1)
    bt = np.full((len(spec.seqs), stride), -1, dtype=np.int32)
    at = 0
    for i, k in enumerate(need):
        bt[i, :k] = order[at:at + k]
        at += int(k)
    return bt, total


def random_small_step(seed: int, max_seqs: int = 6, max_n: int = 70, max_c: int = 300,
                      n_q_heads: int = HQ, n_kv_heads: int = HKV) -> StepSpec:
    """A seeded small mixed step for fuzzing: a random mix of decode rows and prefill chunks
    whose lengths straddle tile and page boundaries."""
    g = rng(seed, 99)
    S = int(g.integers(1, max_seqs, endpoint=True))
    seqs = []
    for i in range(S):
        if g.random() < 0.4:
            seqs.append(Seq(1, int(g.integers(0, max_c, endpoint=True)), i))
        else:
            seqs.append(Seq(int(g.integers(1, max_n, endpoint=True)), int(g.integers(0, max_c, endpoint=True)), i))
    return StepSpec(f"fuzz{seed}", seqs, n_q_heads=n_q_heads, n_kv_heads=n_kv_heads)


# ---------------------------------------------------------------------------
# Fused gate-up projection of a decoder block's MLP (the paper's other profiled
# prefill operation, Section 6.1). Sizes of the published Qwen2.5-3B
# configuration: hidden 2048, intermediate 11008 (the stacked weight has 22016
# rows). Hidden states are N(0, 1) (the scale of normalised activations);
# weights are N(0, 0.02^2), the initialiser scale of this model family.
GATEUP_HIDDEN, GATEUP_INTER = 2048, 11008
GATEUP_W_STD = 0.02
_GX, _GW = 8, 9
_GX_BLOCK = 256   # token rows drawn per seeded block


def gateup_weight(seed: int, hidden: int = GATEUP_HIDDEN, inter: int = GATEUP_INTER) -> np.ndarray:
    """Stacked gate/up weight [2 * inter, hidden] as bf16 bit patterns (gate rows first)."""
    g = rng(seed, _GW, hidden, inter)
    return f32_to_bf16_bits(g.standard_normal(size=(2 * inter, hidden), dtype=np.float32) * np.float32(GATEUP_W_STD))


def gateup_tokens(seed: int, n_rows: int, first_row: int = 0, hidden: int = GATEUP_HIDDEN) -> np.ndarray:
    """Token rows first_row..first_row+n_rows-1 of a seeded prompt's hidden states [n, hidden]
    (bf16 bits). Rows come in seeded blocks of 256, so any chunking of the prompt sees the
    same rows as the whole prompt."""
    out = np.empty((n_rows, hidden), dtype=np.uint16)
    r = first_row
    while r < first_row + n_rows:
        b = r // _GX_BLOCK
        blk = normal_bf16(rng(seed, _GX, hidden, b), (_GX_BLOCK, hidden))
        lo = r - b * _GX_BLOCK
        take = min(_GX_BLOCK - lo, first_row + n_rows - r)
        out[r - first_row:r - first_row + take] = blk[lo:lo + take]
        r += take
    return out
