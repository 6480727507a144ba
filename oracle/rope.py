"""Rotary position embedding of a step's new rows, and the page write that follows it.

TEST INFRASTRUCTURE (see the package docstring): never called by the product path.

The paper does not describe how positions enter attention. Its model is a
decoder block whose attention runs on the step's new query, key and value rows
(Section 6.1), and the models it serves rotate queries and keys by their
positions before attention. The reading used here is the standard rotary
position embedding (RoPE; Su et al., "RoFormer", 2021) in its rotate-half form
over the whole head: for a head vector x of even length D at position p, the
feature pairs (i, i + D/2), i < D/2, turn by the angle a_i = p * theta^(-2i/D):

    y_i       = x_i cos a_i - x_{i+D/2} sin a_i
    y_{i+D/2} = x_{i+D/2} cos a_i + x_i sin a_i

Query rows and new key rows are rotated at their own positions (cached_len + i
for row i of a request); values are not rotated. The rotated keys are then
written to the pages exactly as the plain append writes unrotated ones
(oracle.kv_cache). theta is a parameter (10^6 for the Qwen2.5 family whose
attention shape the workloads use; 10^4 in the original RoPE paper).

Everything is float64; inputs are bf16 bit patterns converted exactly.
"""
from __future__ import annotations

import numpy as np

from oracle import kv_cache


def bf16_bits_to_f64(x) -> np.ndarray:
    """bf16 bit patterns (uint16) to float64, exactly."""
    return (np.asarray(x, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def f64_to_bf16_bits(x) -> np.ndarray:
    """float64 values to bf16 bit patterns, rounded to nearest, ties to even, in one
    step: scale each value so its bf16 grid (8 significant bits) becomes the integers,
    round with numpy's round-half-even, scale back (all exact in float64; values stay
    in bf16's normal range here). The result is exactly representable in float32, whose
    top 16 bits are the bf16 pattern."""
    x = np.asarray(x, dtype=np.float64)
    out = np.zeros(x.shape, dtype=np.float64)
    nz = x != 0
    e = np.floor(np.log2(np.abs(x[nz])))
    u = np.exp2(e - 7)                                   # grid spacing of the value's binade
    out[nz] = np.rint(x[nz] / u) * u
    return (out.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)


def angles(positions, head_dim: int, theta: float) -> np.ndarray:
    """[n, D/2] rotation angles: position p times theta^(-2i/D) for pair i."""
    pos = np.asarray(positions, dtype=np.float64)
    i = np.arange(head_dim // 2, dtype=np.float64)
    freq = np.power(float(theta), -2.0 * i / head_dim)
    return pos[:, None] * freq[None, :]


def rotate(x, positions, theta: float) -> np.ndarray:
    """Rotate x [n, H, D] (float64 values) row r at positions[r]; returns float64 [n, H, D]."""
    x = np.asarray(x, dtype=np.float64)
    n, H, D = x.shape
    a = angles(positions, D, theta)[:, None, :]          # [n, 1, D/2]
    c, s = np.cos(a), np.sin(a)
    x1, x2 = x[:, :, :D // 2], x[:, :, D // 2:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=2)


def row_positions(desc) -> np.ndarray:
    """Position of every row of the step: cached_len + i for row query_start + i."""
    desc = np.asarray(desc)
    T = int(desc[:, 1].sum()) if len(desc) else 0
    pos = np.zeros(T, dtype=np.int64)
    for qs, n, c in desc.tolist():
        pos[qs:qs + n] = c + np.arange(n)
    return pos


def rope_step(q_bits, k_new_bits, desc, theta: float):
    """The rotated query rows [T, Hq, D] and new key rows [T, Hkv, D] of a step, float64."""
    pos = row_positions(desc)
    return rotate(bf16_bits_to_f64(q_bits), pos, theta), rotate(bf16_bits_to_f64(k_new_bits), pos, theta)


def rope_kv_append(k_pool, v_pool, q_bits, k_new_bits, v_new_bits, desc, block_table, page_size: int,
                   theta: float):
    """Rotated Q (float64), rotated new K (float64), and the V pool after the append
    (bit patterns; V is copied unrotated, so this part is exact)."""
    q_rot, k_rot = rope_step(q_bits, k_new_bits, desc, theta)
    _, vp = kv_cache.append(k_pool, v_pool, k_new_bits, v_new_bits, desc, block_table, page_size)
    return q_rot, k_rot, vp
