"""Float64 reference attention for one mixed scheduler step.

TEST INFRASTRUCTURE (see the package docstring): never called by the product path.

What is computed. A scheduler iteration batches prefill chunks and decode tokens
of different requests (Section 2, continuous batching with chunked prefill; the
mixed iterations of Section 6.2). Prefill stores each token's key and value in
the KV cache and decode generates one token per request per iteration
(Section 2). A request with n new tokens after c cached ones therefore owns
query rows at positions c..c+n-1; its new keys/values occupy the same positions
and are in the cache before attention runs. The row at position p attends to
keys 0..p: fully to the cached prefix and causally within its own chunk. A
decode row is the case n = 1.

The paper gives no attention formula, head grouping or scale; the readings used
here are: softmax(scale * q.k) weighted sum of values, scale = 1/sqrt(head_dim),
query head h reading KV head floor(h / (Hq/Hkv)), and an inclusive diagonal.
Paging (Section 7, PagedAttention) only changes where keys live, so this
reference reads the logical, unpaged keys of each request.

For each request s, KV head g, query head h in g's group and row i:
    l_j = scale * sum_d Q[qs+i, h, d] * K_s[j, g, d]      for j = 0..c+i
    O[qs+i, h, :] = sum_j exp(l_j - max l) V_s[j, g, :] / sum_j exp(l_j - max l)

On request, the same weights also give A[qs+i, h, :] = sum_j w_j |V_s[j, g, :]|
(w_j the normalised softmax weights): the weighted mean of the values' magnitudes,
which bounds how far rounding the weights can move O (a test bound, not part of
the attention).
"""
from __future__ import annotations

import numpy as np


def bf16_to_f64(bits) -> np.ndarray:
    """Exact bf16 -> float64: a bf16 pattern is the top half of a float32 pattern."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def logical_kv(hist_bits, new_bits) -> np.ndarray:
    """A request's keys (or values) at positions 0..c+n-1: the c cached rows followed by
    the step's n new rows, which the step writes to the cache before attending."""
    parts = [np.asarray(new_bits, dtype=np.uint16)]
    if hist_bits is not None and len(hist_bits):
        parts.insert(0, np.asarray(hist_bits, dtype=np.uint16))
    return np.concatenate(parts, axis=0)


def _attend(qf, kf, vf, pos, scale, with_abs=False):
    """qf [r, G, D]; kf, vf [nk, D]; pos [r] positions; returns [r, G, D] (and the
    weighted mean of |V| under the same weights when with_abs).
    Row i sees keys 0..pos[i]."""
    r, G, D = qf.shape
    logits = scale * (qf.reshape(r * G, D) @ kf.T).reshape(r, G, -1)
    hidden = np.arange(kf.shape[0])[None, :] > pos[:, None]          # [r, nk]
    logits[np.broadcast_to(hidden[:, None, :], logits.shape)] = -np.inf
    m = logits.max(axis=-1, keepdims=True)
    w = np.exp(logits - m)
    den = w.sum(axis=-1)[..., None]
    o = (w.reshape(r * G, -1) @ vf).reshape(r, G, D) / den
    if not with_abs:
        return o
    return o, (w.reshape(r * G, -1) @ np.abs(vf)).reshape(r, G, D) / den


def mixed_step_attention(q_bits, desc, k_seq, v_seq, scale: float, n_kv_heads: int,
                         rows=None, block_elems: int = 1 << 25, with_abs: bool = False):
    """Attention outputs of one mixed step.

    q_bits: uint16 bf16 [T, Hq, D]; desc: int [S, 3] of (query_start, n_query, cached_len);
    k_seq / v_seq: per request uint16 bf16 [cached_len + n_query, Hkv, D] (logical order).
    rows: optional iterable of row indices in [0, T); only those rows are computed and
    the others are NaN. Returns float64 [T, Hq, D]; with with_abs, the pair (O, A) of
    the outputs and the weighted means of |V| (module docstring).
    """
    q_bits = np.asarray(q_bits, dtype=np.uint16)
    T, Hq, D = q_bits.shape
    G = Hq // n_kv_heads
    out = np.full((T, Hq, D), np.nan)
    absv = np.full((T, Hq, D), np.nan) if with_abs else None
    want = None if rows is None else np.zeros(T, dtype=bool)
    if want is not None:
        want[np.asarray(list(rows), dtype=np.int64)] = True
    for s in range(len(desc)):
        qs, n, c = (int(x) for x in desc[s])
        local = np.arange(n)
        if want is not None:
            local = local[want[qs:qs + n]]
        if local.size == 0:
            continue
        K = bf16_to_f64(k_seq[s])
        V = bf16_to_f64(v_seq[s])
        assert K.shape[0] == c + n and V.shape[0] == c + n, "logical K/V must cover positions 0..c+n-1"
        for g in range(n_kv_heads):
            hs = slice(g * G, (g + 1) * G)
            start = 0
            while start < local.size:
                nk = c + int(local[start]) + 1
                rb = max(1, block_elems // (G * max(nk, 1)))
                blk = local[start:start + rb]
                nk = c + int(blk[-1]) + 1          # keys needed by the last row of the block
                qf = bf16_to_f64(q_bits[qs + blk, hs, :])
                res = _attend(qf, K[:nk, g, :], V[:nk, g, :], c + blk, scale, with_abs)
                if with_abs:
                    out[qs + blk, hs, :], absv[qs + blk, hs, :] = res
                else:
                    out[qs + blk, hs, :] = res
                start += blk.size
    return (out, absv) if with_abs else out


def step_attention_from_data(data, scale: float, rows=None, with_abs: bool = False):
    """The attention of a step given as a StepData-like object: q and the step's new
    rows k_new / v_new [T, Hkv, D] (row query_start + i of request s is its position
    cached_len + i), each request's cached history k_hist[s] / v_hist[s] (positions
    0..cached_len-1), and desc. Request s's logical keys are its history followed by
    its new rows qs..qs+n-1."""
    ks, vs = [], []
    for s in range(len(data.desc)):
        qs, n, _ = (int(x) for x in data.desc[s])
        ks.append(logical_kv(data.k_hist[s], data.k_new[qs:qs + n]))
        vs.append(logical_kv(data.v_hist[s], data.v_new[qs:qs + n]))
    return mixed_step_attention(data.q, data.desc, ks, vs, scale, data.k_new.shape[1], rows=rows,
                                with_abs=with_abs)
