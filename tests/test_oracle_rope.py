"""Pins for the rotary-embedding oracle (CPU only). Each catches a different
plausible mistake: a scalar brute-force loop (pairing and index errors), a
rotation of basis vectors read back with atan2 (direction and frequency of every
pair, against closed-form frequencies such as theta^(-1/2) for the middle pair),
the complex-multiplication form of the same rotation, position 0 as the
identity, per-pair norm preservation, composition of rotations, the
relative-position property of rotated dot products, linearity, and the row
positions of a mixed step (cached_len + i)."""
import math

import numpy as np
import pytest

import oracle.rope as R
import oracle.kv_cache as OK
from paper_2608_15171_amd import inputs as I


def brute(x, positions, theta):
    """Pure-Python loops, math.cos / math.sin, rotate-half pairs (i, i + D/2)."""
    n, H, D = len(x), len(x[0]), len(x[0][0])
    out = [[[0.0] * D for _ in range(H)] for _ in range(n)]
    for r in range(n):
        for h in range(H):
            for i in range(D // 2):
                a = positions[r] * theta ** (-2.0 * i / D)
                x1, x2 = x[r][h][i], x[r][h][i + D // 2]
                out[r][h][i] = x1 * math.cos(a) - x2 * math.sin(a)
                out[r][h][i + D // 2] = x2 * math.cos(a) + x1 * math.sin(a)
    return np.array(out)


@pytest.mark.parametrize("D", [2, 4, 8, 16])
@pytest.mark.parametrize("theta", [10000.0, 1e6, 3.0])
def test_matches_brute_force(D, theta):
    g = np.random.default_rng(D)
    x = g.standard_normal((5, 3, D))
    pos = [0, 1, 7, 1000, 29999]
    assert np.allclose(R.rotate(x, pos, theta), brute(x.tolist(), pos, theta), rtol=0, atol=1e-12)


@pytest.mark.parametrize("theta", [10000.0, 1e6])
def test_basis_vectors_turn_by_closed_form_angles(theta):
    """e_i at position p comes out as (cos a, sin a) in slots (i, i + D/2) with a = p * theta^(-2i/D);
    pair 0 turns by p radians, pair D/4 by p / sqrt(theta), pair D/2 - 1 by p * theta^(-(D-2)/D)."""
    D = 128
    closed = {0: 1.0, D // 4: 1.0 / math.sqrt(theta), D // 2 - 1: theta ** (-(D - 2) / D)}
    for p in (1, 5, 123):
        for i, f in closed.items():
            x = np.zeros((1, 1, D))
            x[0, 0, i] = 1.0
            y = R.rotate(x, [p], theta)[0, 0]
            assert np.count_nonzero(np.abs(y) > 1e-15) <= 2
            a = math.atan2(y[i + D // 2], y[i])
            want = math.remainder(p * f, 2 * math.pi)
            assert abs(a - want) < 1e-9, (p, i, a, want)
            assert abs(math.hypot(y[i], y[i + D // 2]) - 1.0) < 1e-14


def test_complex_form():
    """Pair i as the complex number x_i + j x_{i+D/2}, multiplied by exp(j a_i)."""
    g = np.random.default_rng(1)
    D, theta = 128, 1e6
    x = g.standard_normal((7, 4, D))
    pos = np.array([0, 3, 16, 255, 4096, 25000, 30063])
    z = x[:, :, :D // 2] + 1j * x[:, :, D // 2:]
    w = z * np.exp(1j * pos[:, None, None] * theta ** (-np.arange(D // 2) / (D // 2)))[:, :, :]
    y = R.rotate(x, pos, theta)
    assert np.allclose(y[:, :, :D // 2], w.real, atol=1e-11) and np.allclose(y[:, :, D // 2:], w.imag, atol=1e-11)


def test_position_zero_is_identity_and_norms_are_kept():
    g = np.random.default_rng(2)
    x = g.standard_normal((4, 3, 128))
    assert np.array_equal(R.rotate(x, [0, 0, 0, 0], 1e6), x)
    y = R.rotate(x, [1, 77, 5000, 30000], 1e6)
    pair = lambda v: v[:, :, :64] ** 2 + v[:, :, 64:] ** 2
    assert np.allclose(pair(y), pair(x), rtol=1e-13, atol=1e-13)


def test_composition_and_inverse():
    g = np.random.default_rng(3)
    x = g.standard_normal((3, 2, 128))
    p1, p2 = np.array([5, 100, 20000]), np.array([7, 3000, 9000])
    both = R.rotate(R.rotate(x, p1, 1e6), p2, 1e6)
    assert np.allclose(both, R.rotate(x, p1 + p2, 1e6), atol=1e-9)
    assert np.allclose(R.rotate(R.rotate(x, p1, 1e6), -p1, 1e6), x, atol=1e-9)


def test_rotated_dot_products_depend_on_relative_position_only():
    g = np.random.default_rng(4)
    q, k = g.standard_normal((1, 1, 128)), g.standard_normal((1, 1, 128))
    for p1, p2, shift in [(10, 3, 1), (25000, 24990, 5000), (0, 0, 12345)]:
        a = float(np.sum(R.rotate(q, [p1], 1e6) * R.rotate(k, [p2], 1e6)))
        b = float(np.sum(R.rotate(q, [p1 + shift], 1e6) * R.rotate(k, [p2 + shift], 1e6)))
        assert abs(a - b) < 1e-9 * (1 + abs(a))


def test_linearity():
    g = np.random.default_rng(5)
    x, y = g.standard_normal((2, 3, 128)), g.standard_normal((2, 3, 128))
    pos = [9, 1234]
    assert np.allclose(R.rotate(2.5 * x - y, pos, 1e4), 2.5 * R.rotate(x, pos, 1e4) - R.rotate(y, pos, 1e4),
                       atol=1e-12)


def test_step_rows_rotate_at_cached_len_plus_offset():
    spec = I.StepSpec("mix", [I.Seq(1, 40, 0), I.Seq(5, 0, 1), I.Seq(3, 17, 2)])
    data = I.make_step_data(spec, 0, with_history=False)
    q, k = R.rope_step(data.q, data.k_new, data.desc, 1e6)
    pos = [40, 0, 1, 2, 3, 4, 17, 18, 19]
    assert list(R.row_positions(data.desc)) == pos
    for r, p in enumerate(pos):
        assert np.array_equal(q[r:r + 1], R.rotate(R.bf16_bits_to_f64(data.q[r:r + 1]), [p], 1e6))
        assert np.array_equal(k[r:r + 1], R.rotate(R.bf16_bits_to_f64(data.k_new[r:r + 1]), [p], 1e6))
    # row 1 is request 1's first token at position 0: unchanged
    assert np.array_equal(q[1], R.bf16_bits_to_f64(data.q[1]))


def test_append_after_rotation_copies_v_and_leaves_k_to_the_rotation():
    spec = I.random_small_step(3, max_seqs=3, max_n=20, max_c=40)
    data = I.make_step_data(spec, 3, with_history=False)
    bt, npages = I.make_block_table(spec, 3, permute=True, spare_pages=2)
    kp = np.full((npages, 2, 16, 16, 8), 0xFFFF, np.uint16)
    vp = np.full((npages, 2, 128, 16), 0xFFFF, np.uint16)
    q_rot, k_rot, vp2 = R.rope_kv_append(kp, vp, data.q, data.k_new, data.v_new, data.desc, bt, 16, 1e6)
    assert np.array_equal(vp2, OK.append(kp, vp, data.k_new, data.v_new, data.desc, bt, 16)[1])
    assert q_rot.shape == data.q.shape and k_rot.shape == data.k_new.shape


def test_f64_to_bf16_rounding():
    """Nearest-even on the 8-bit significand grid: exact values stay, halfway cases go to
    the even neighbour, everything else to the nearer one; the bit patterns decode back."""
    one_ulp = 2.0 ** -7
    cases = {1.0: 1.0, 1.0 + one_ulp / 2: 1.0, 1.0 + 3 * one_ulp / 2: 1.0 + 2 * one_ulp,
             1.0 + one_ulp * 0.51: 1.0 + one_ulp, -3.0: -3.0, 0.0: 0.0,
             2.0 - one_ulp / 4: 2.0, 255.5: 256.0, 1e-3: None}
    for x, want in cases.items():
        got = float(R.bf16_bits_to_f64(R.f64_to_bf16_bits([x]))[0])
        if want is None:
            assert abs(got - x) <= 2.0 ** -9 * abs(x)
        else:
            assert got == want, (x, got, want)
    g = np.random.default_rng(6)
    bits = g.integers(0, 1 << 16, size=4000, dtype=np.uint16)
    bits = bits[((bits >> 7) & 0xFF) != 0xFF]             # finite patterns only
    vals = R.bf16_bits_to_f64(bits)
    fin = np.isfinite(vals) & (np.abs(vals) > 1e-30) & (np.abs(vals) < 1e30)
    assert np.array_equal(R.f64_to_bf16_bits(vals[fin]), bits[fin])
