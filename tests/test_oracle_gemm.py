"""Pins of the gate-up projection oracle (oracle/gemm.py) against what the
mathematics fixes, not against itself: a pure-Python fsum brute force with its own
bf16 decoding, closed forms (a permutation weight copies columns, all-ones inputs
give weight row sums, rank-one inputs factor), invariants (token rows are
independent, so any chunking of a prompt gives the same rows -- the property the
paper's 8 x 2k vs 1 x 16k comparison rests on; the gate and up halves are
independent projections; integer-valued inputs are exactly linear), and planted
mistakes that the pins must reject. The gated activation (gate_up_act) is pinned
by a brute force with math.exp, the identity silu(g) - silu(-g) = g, its limits,
and zero halves."""
import math
import struct
import types

import numpy as np
import pytest

import oracle.gemm as OG
from paper_2608_15171_amd import inputs as I


def bits(x):
    """float values exactly representable in bf16 -> bf16 patterns."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32)
    assert ((u & 0xFFFF) == 0).all(), "value not exactly representable in bf16"
    return (u >> 16).astype(np.uint16)


def decode(b):
    """bf16 pattern -> Python float, through struct (independent of the oracle's decoding)."""
    return struct.unpack("<f", struct.pack("<I", int(b) << 16))[0]


def brute_force(xb, wb, with_abs=False):
    T, H = xb.shape
    N = wb.shape[0]
    Y = np.zeros((T, N))
    A = np.zeros((T, N))
    for t in range(T):
        for n in range(N):
            terms = [decode(xb[t, k]) * decode(wb[n, k]) for k in range(H)]
            Y[t, n] = math.fsum(terms)
            A[t, n] = math.fsum(abs(v) for v in terms)
    return (Y, A) if with_abs else Y


def rand_bits(seed, shape, scale=1.0):
    g = np.random.default_rng(seed)
    return I.f32_to_bf16_bits((g.standard_normal(shape) * scale).astype(np.float32))


@pytest.mark.parametrize("seed", range(4))
def test_bruteforce_tiny(seed):
    T, H, N = 3 + seed, 8 + 3 * seed, 5 + 2 * seed
    xb, wb = rand_bits(seed, (T, H)), rand_bits(100 + seed, (N, H), 0.02)
    y, a = OG.gate_up(xb, wb, with_abs=True)
    by, ba = brute_force(xb, wb, with_abs=True)
    np.testing.assert_allclose(y, by, rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(a, ba, rtol=1e-13, atol=1e-15)


def test_permutation_weight_copies_columns_exactly():
    T, H = 7, 16
    xb = rand_bits(1, (T, H))
    perm = np.random.default_rng(2).permutation(H)
    w = np.zeros((H, H), dtype=np.float32)
    w[np.arange(H), perm] = 1.0
    y = OG.gate_up(xb, bits(w))
    assert np.array_equal(y, OG.bf16_to_f64(xb)[:, perm])


def test_ones_input_gives_weight_row_sums():
    H, N = 24, 9
    wb = rand_bits(3, (N, H), 0.02)
    y = OG.gate_up(bits(np.ones((2, H), np.float32)), wb)
    for n in range(N):
        s = math.fsum(decode(v) for v in wb[n])
        assert abs(y[0, n] - s) <= 1e-15 and y[1, n] == y[0, n]


def test_rank_one_factors():
    # X = a u^T, W = b v^T with small integers: Y = (a b^T) (u . v), exactly
    a, u = np.array([1, -2, 3], np.float32), np.array([2, 0, -1, 4, 1], np.float32)
    b, v = np.array([3, 1, -1, 2], np.float32), np.array([1, 1, 2, -3, 5], np.float32)
    y = OG.gate_up(bits(np.outer(a, u)), bits(np.outer(b, v)))
    assert np.array_equal(y, np.outer(a, b).astype(np.float64) * float(u @ v))


def test_integer_inputs_are_exactly_linear():
    g = np.random.default_rng(4)
    x1, x2 = g.integers(-8, 9, (5, 32)).astype(np.float32), g.integers(-8, 9, (5, 32)).astype(np.float32)
    w = g.integers(-8, 9, (6, 32)).astype(np.float32)
    y = OG.gate_up(bits(x1 + x2), bits(w))
    assert np.array_equal(y, OG.gate_up(bits(x1), bits(w)) + OG.gate_up(bits(x2), bits(w)))
    assert np.array_equal(y, (x1 + x2).astype(np.float64) @ w.T.astype(np.float64))


def test_chunked_rows_equal_whole_prompt():
    """Eight chunks of a prompt projected one after another give the rows of the whole
    prompt projected at once (rows are independent)."""
    H, N, T = 64, 48, 8 * 40
    wb = I.gateup_weight(0, hidden=H, inter=N // 2)
    whole = OG.gate_up(I.gateup_tokens(0, T, 0, hidden=H), wb)
    parts = [OG.gate_up(I.gateup_tokens(0, 40, 40 * c, hidden=H), wb) for c in range(8)]
    np.testing.assert_allclose(np.concatenate(parts), whole, rtol=1e-14, atol=1e-15)


def test_gate_and_up_halves_are_separate_projections():
    H, inter = 32, 12
    xb, wb = I.gateup_tokens(5, 9, 0, hidden=H), I.gateup_weight(5, hidden=H, inter=inter)
    y = OG.gate_up(xb, wb)
    np.testing.assert_allclose(y[:, :inter], OG.gate_up(xb, wb[:inter]), rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(y[:, inter:], OG.gate_up(xb, wb[inter:]), rtol=1e-14, atol=1e-15)


def test_rows_argument_selects_rows():
    xb, wb = rand_bits(6, (20, 16)), rand_bits(7, (10, 16))
    rows = np.array([19, 0, 7, 7])
    np.testing.assert_array_equal(OG.gate_up(xb, wb, rows=rows), OG.gate_up(xb, wb)[rows])


def test_abs_product_bounds_the_product():
    xb, wb = rand_bits(8, (6, 40)), rand_bits(9, (7, 40))
    y, a = OG.gate_up(xb, wb, with_abs=True)
    assert (a >= np.abs(y) - 1e-15).all()
    pos = bits(np.abs(OG.bf16_to_f64(xb)).astype(np.float32))
    y2, a2 = OG.gate_up(pos, bits(np.abs(OG.bf16_to_f64(wb)).astype(np.float32)), with_abs=True)
    np.testing.assert_allclose(y2, a2, rtol=1e-14, atol=0)


# ------------------------------------------------------------- gated activation

def silu_math(g):
    """g * sigmoid(g) with math.exp, written for both signs without overflow."""
    if g >= 0:
        return g / (1.0 + math.exp(-g))
    e = math.exp(g)
    return g * e / (1.0 + e)


def test_silu_closed_forms():
    assert OG.silu(0.0) == 0.0
    assert OG.silu(1.0) == pytest.approx(1.0 / (1.0 + math.exp(-1.0)), rel=1e-15)
    assert OG.silu(-1.0) == pytest.approx(-math.exp(-1.0) / (1.0 + math.exp(-1.0)), rel=1e-15)
    assert OG.silu(60.0) == pytest.approx(60.0, rel=1e-15)             # sigmoid -> 1
    assert -1e-20 < OG.silu(-60.0) < 0.0                                  # -> 0 from below
    assert OG.silu(-1e4) == 0.0 and OG.silu(1e4) == 1e4                 # no overflow either way


def test_silu_odd_part_is_identity():
    """silu(g) - silu(-g) = g sigmoid(g) + g (1 - sigmoid(g)) = g for every g."""
    g = np.random.default_rng(11).standard_normal(1000) * 6
    np.testing.assert_allclose(OG.silu(g) - OG.silu(-g), g, rtol=1e-14, atol=1e-14)


def brute_act(xb, wb):
    y = brute_force(xb, wb)
    i = wb.shape[0] // 2
    return np.array([[silu_math(y[t, f]) * y[t, i + f] for f in range(i)] for t in range(y.shape[0])])


@pytest.mark.parametrize("seed", range(3))
def test_act_bruteforce_tiny(seed):
    T, H, I2 = 3 + seed, 8 + 4 * seed, 2 * (3 + seed)
    xb, wb = rand_bits(20 + seed, (T, H)), rand_bits(30 + seed, (I2, H), 0.3)
    np.testing.assert_allclose(OG.gate_up_act(xb, wb), brute_act(xb, wb), rtol=1e-12, atol=1e-15)


def test_act_terms_are_the_halves():
    xb, wb = rand_bits(40, (5, 16)), rand_bits(41, (12, 16), 0.3)
    z, g, u, ag, au = OG.gate_up_act(xb, wb, with_terms=True)
    y, a = OG.gate_up(xb, wb, with_abs=True)
    assert np.array_equal(g, y[:, :6]) and np.array_equal(u, y[:, 6:])
    assert np.array_equal(ag, a[:, :6]) and np.array_equal(au, a[:, 6:])


def test_act_zero_halves():
    """A zero up half gives zero; a zero gate half gives silu(0) = 0."""
    xb = rand_bits(42, (4, 16))
    w = OG.bf16_to_f64(rand_bits(43, (10, 16), 0.3)).astype(np.float32)
    w_up0, w_gate0 = w.copy(), w.copy()
    w_up0[5:] = 0.0
    w_gate0[:5] = 0.0
    assert not np.any(OG.gate_up_act(xb, bits(w_up0)))
    assert not np.any(OG.gate_up_act(xb, bits(w_gate0)))


def test_act_large_gate_passes_up_through():
    """With the gate half a large positive multiple of an all-ones row, Z = g u."""
    H = 8
    x = np.ones((2, H), np.float32)
    w = np.zeros((4, H), np.float32)
    w[:2] = 8.0                                   # g = 64 for every token
    w[2, 0], w[3, :] = 0.5, -0.25                 # u = 0.5 and -2
    z = OG.gate_up_act(bits(x), bits(w))
    np.testing.assert_allclose(z, [[32.0, -128.0], [32.0, -128.0]], rtol=1e-15)


# ---------------------------------------------------------------- mutation test

MUTANTS = {
    "weight_not_transposed": ("Y = X @ W.T", "Y = X @ W"),
    "bf16_low_half": ("(b.astype(np.uint32) << 16)", "(b.astype(np.uint32) << 15)"),
    "rows_ignored": ("        x = x[np.asarray(rows)]\n", "        pass\n"),
    "last_feature_dropped": ("Y = X @ W.T", "Y = X[:, :-1] @ W[:, :-1].T"),
    "abs_of_signed_weight": ("np.abs(X) @ np.abs(W).T", "np.abs(X) @ W.T"),
    "rows_from_weight_order": ("Y = X @ W.T", "Y = X @ W[::-1].T"),
    "silu_sign": ("e = np.exp(-np.abs(g))", "e = np.exp(np.abs(g))"),
    "act_halves_swapped": ("z = silu(g) * u", "z = silu(u) * g"),
    "act_without_gate_weight": ("z = silu(g) * u", "z = g * u"),
    "act_gate_half_shifted": ("g, u = y[:, :i], y[:, i:]", "g, u = y[:, 1:i + 1], y[:, i:]"),
}


def mutant(name):
    src = open(OG.__file__).read()
    a, b = MUTANTS[name]
    assert src.count(a) == 1, name
    mod = types.ModuleType("oracle_gemm_mutant_" + name)
    exec(compile(src.replace(a, b), "<mutant>", "exec"), mod.__dict__)
    return mod


def pins_pass(mod) -> bool:
    try:
        for seed in range(2):
            T, H, N = 3, 8, 5
            xb, wb = rand_bits(seed, (T, H)), rand_bits(50 + seed, (N, H), 0.02)
            y, a = mod.gate_up(xb, wb, with_abs=True)
            by, ba = brute_force(xb, wb, with_abs=True)
            if not (np.allclose(y, by, rtol=1e-13, atol=1e-15) and np.allclose(a, ba, rtol=1e-13, atol=1e-15)):
                return False
        xb, wb = rand_bits(6, (20, 16)), rand_bits(7, (10, 16))
        rows = np.array([19, 0, 7])
        if not np.allclose(mod.gate_up(xb, wb, rows=rows), brute_force(xb[rows], wb), rtol=1e-13, atol=1e-15):
            return False
        xb, wb = rand_bits(8, (3, 12)), rand_bits(9, (8, 12), 0.3)
        if not np.allclose(mod.gate_up_act(xb, wb), brute_act(xb, wb), rtol=1e-12, atol=1e-15):
            return False
    except Exception:
        return False
    return True


def test_pins_accept_the_oracle():
    assert pins_pass(OG)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_planted_mistake(name):
    assert not pins_pass(mutant(name)), f"mutant {name} survived the pins"
