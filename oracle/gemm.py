"""Float64 reference of a decoder block's fused gate-up projection.

TEST INFRASTRUCTURE (see the package docstring): never called by the product path.

What is computed. Besides attention, the paper profiles the fused gate-up
projection as the other dominant operation of a prefill chunk in a Qwen2.5
decoder block (Section 6.1: cumulative time of eight 2k chunks against one 16k
chunk, Fig. 4b; SM throughput, L2 hit rate and DRAM throughput at MBT 2k and
16k, Table 6). In those models the MLP's gate and up projections read the same
input, the block's normalised hidden states, and run as one linear layer whose
weight holds the gate rows followed by the up rows. For a chunk of T tokens,
hidden size H and intermediate size I:

    Y[t, n] = sum_k X[t, k] * W[n, k]        t < T, n < 2I

with X [T, H] the hidden states and W [2I, H] the stacked weight (rows 0..I-1
gate, rows I..2I-1 up). The paper prints neither H nor I; they are parameters
(H = 2048, I = 11008 in the published Qwen2.5-3B configuration).

The activation that follows in those models' MLP (a gated SiLU unit) takes the
two halves of Y for each token and intermediate feature f < I:

    Z[t, f] = silu(Y[t, f]) * Y[t, I + f],     silu(g) = g / (1 + exp(-g))

gate_up_act computes Z from the exact Y; the paper profiles the projection
alone, and the library also offers the projection with this activation applied
on the way out (half the output bytes, no separate pass).

Inputs are bf16 bit patterns, converted exactly to float64; the sum is the
float64 matrix product (its rounding, ~1e-16 relative, is far below bf16's).
With with_abs the same product of magnitudes, A[t, n] = sum_k |X[t, k] W[n, k]|,
is returned too: it bounds how far a reordered fp32 accumulation can drift (a
test bound, not part of the projection).
"""
from __future__ import annotations

import numpy as np


def bf16_to_f64(bits) -> np.ndarray:
    """Exact bf16 -> float64: a bf16 pattern is the top half of a float32 pattern."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def gate_up(x_bits, w_bits, rows=None, with_abs: bool = False):
    """Y = X W^T in float64 for X [T, H] and W [2I, H] bf16 patterns; rows (optional)
    restricts the result to those token rows (returned in that order)."""
    x = np.asarray(x_bits, dtype=np.uint16)
    w = np.asarray(w_bits, dtype=np.uint16)
    assert x.ndim == 2 and w.ndim == 2 and x.shape[1] == w.shape[1], "X [T, H] and W [2I, H]"
    if rows is not None:
        x = x[np.asarray(rows)]
    X = bf16_to_f64(x)
    W = bf16_to_f64(w)
    Y = X @ W.T
    if with_abs:
        return Y, np.abs(X) @ np.abs(W).T
    return Y


def silu(g) -> np.ndarray:
    """g / (1 + exp(-g)) in float64, in a form that neither overflows nor loses
    the sign: for g < 0 it is g e^g / (1 + e^g)."""
    g = np.asarray(g, dtype=np.float64)
    e = np.exp(-np.abs(g))
    return np.where(g >= 0, g / (1.0 + e), g * e / (1.0 + e))


def gate_up_act(x_bits, w_bits, rows=None, with_terms: bool = False):
    """Z = silu(Y[:, :I]) * Y[:, I:] in float64, Y = X W^T (see the module docstring).
    With with_terms also the gate and up halves of Y and of the magnitude product
    (g, u, A_g, A_u), from which a test derives its bound."""
    y, a = gate_up(x_bits, w_bits, rows=rows, with_abs=True)
    n2 = y.shape[1]
    assert n2 % 2 == 0, "W stacks I gate rows over I up rows"
    i = n2 // 2
    g, u = y[:, :i], y[:, i:]
    z = silu(g) * u
    if with_terms:
        return z, g, u, a[:, :i], a[:, i:]
    return z
