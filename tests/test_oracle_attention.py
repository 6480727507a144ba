"""Pins for the float64 attention oracle (CPU only).

The paper prints no attention values, so the oracle is pinned to things other
than itself: a scalar brute-force loop, PyTorch's float64 SDPA as a library
routine, closed forms (uniform weights, one visible key, planted keys, a
two-key softmax), and invariants of the problem (chunking, decode vs prefill,
grouped-query heads, batch and order independence). A mutation test then plants
plausible mistakes into a copy of the oracle and checks these pins catch each one.
"""
import math
import struct
import types

import numpy as np
import pytest
import torch

import oracle.attention as OA
from paper_2608_15171_amd import inputs as I

SCALE128 = 1.0 / math.sqrt(128.0)


def bits(x):
    return I.f32_to_bf16_bits(np.asarray(x, dtype=np.float32))


def f64(b):
    return (np.asarray(b, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def make(spec, seed):
    return I.make_step_data(spec, seed)


def run(data, scale, mod=OA, rows=None, with_abs=False):
    """The oracle's entry point for a step (the one the GPU tests, smoke() and the bench
    call), so every pin below also covers how it assembles each request's keys."""
    return mod.step_attention_from_data(data, scale, rows=rows, with_abs=with_abs)


# ---------------------------------------------------------------- brute force

def bf16_scalar(b) -> float:
    """Decode one bf16 pattern through its big-endian float32 bytes."""
    b = int(b)
    return struct.unpack(">f", bytes([b >> 8, b & 0xFF, 0, 0]))[0]


def brute_force(data, scale, with_abs=False):
    """Scalar loops with math.fsum; shares nothing with the oracle's NumPy code. With
    with_abs also the weighted mean of |V| under the same weights."""
    f64 = bf16_scalar
    T, Hq, D = data.q.shape
    Hkv = data.k_new.shape[1]
    G = Hq // Hkv
    out = np.zeros((T, Hq, D))
    absv = np.zeros((T, Hq, D))
    for s in range(len(data.desc)):
        qs, n, c = (int(x) for x in data.desc[s])
        K = [[[float(f64(data.k_hist[s][j, g, d])) for d in range(D)] for g in range(Hkv)] for j in range(c)]
        V = [[[float(f64(data.v_hist[s][j, g, d])) for d in range(D)] for g in range(Hkv)] for j in range(c)]
        for i in range(n):
            K.append([[float(f64(data.k_new[qs + i, g, d])) for d in range(D)] for g in range(Hkv)])
            V.append([[float(f64(data.v_new[qs + i, g, d])) for d in range(D)] for g in range(Hkv)])
        for i in range(n):
            p = c + i
            for h in range(Hq):
                g = h // G
                qv = [float(f64(data.q[qs + i, h, d])) for d in range(D)]
                lg = [scale * math.fsum(qv[d] * K[j][g][d] for d in range(D)) for j in range(p + 1)]
                mx = max(lg)
                w = [math.exp(x - mx) for x in lg]
                den = math.fsum(w)
                for d in range(D):
                    out[qs + i, h, d] = math.fsum(w[j] * V[j][g][d] for j in range(p + 1)) / den
                    absv[qs + i, h, d] = math.fsum(w[j] * abs(V[j][g][d]) for j in range(p + 1)) / den
    return (out, absv) if with_abs else out


def tiny_spec(seed):
    g = I.rng(seed, 123)
    S = int(g.integers(1, 3, endpoint=True))
    seqs = [I.Seq(int(g.integers(1, 5, endpoint=True)), int(g.integers(0, 7, endpoint=True)), k) for k in range(S)]
    return I.StepSpec("tiny", seqs, n_q_heads=4, n_kv_heads=2, head_dim=8)


@pytest.mark.parametrize("seed", range(6))
def test_bruteforce_tiny(seed):
    data = make(tiny_spec(seed), seed)
    o, a = run(data, 0.37, with_abs=True)
    bo, ba = brute_force(data, 0.37, with_abs=True)
    np.testing.assert_allclose(o, bo, rtol=0, atol=1e-12)
    np.testing.assert_allclose(a, ba, rtol=0, atol=1e-12)
    np.testing.assert_array_equal(run(data, 0.37), o)


def test_entry_point_with_history_and_new_rows():
    """step_attention_from_data on a step whose requests all have cached history and
    new rows (prefill chunks and decodes, query_start > 0 for all but the first):
    equal to the brute force, which reads history and new rows on its own."""
    spec = I.StepSpec("hist", [I.Seq(1, 6, 0), I.Seq(4, 3, 1), I.Seq(3, 5, 2), I.Seq(1, 2, 3)],
                      n_q_heads=4, n_kv_heads=2, head_dim=8)
    data = make(spec, 31)
    assert all(len(h) > 0 for h in data.k_hist)
    np.testing.assert_allclose(OA.step_attention_from_data(data, 0.41), brute_force(data, 0.41), rtol=0, atol=1e-12)


# ---------------------------------------------------------------- library pin

def sdpa_reference(data, scale):
    T, Hq, D = data.q.shape
    Hkv = data.k_new.shape[1]
    out = np.zeros((T, Hq, D))
    for s in range(len(data.desc)):
        qs, n, c = (int(x) for x in data.desc[s])
        K = np.concatenate([f64(data.k_hist[s]), f64(data.k_new[qs:qs + n])]) if c else f64(data.k_new[qs:qs + n])
        V = np.concatenate([f64(data.v_hist[s]), f64(data.v_new[qs:qs + n])]) if c else f64(data.v_new[qs:qs + n])
        q = torch.from_numpy(f64(data.q[qs:qs + n])).permute(1, 0, 2)             # [Hq, n, D]
        k = torch.from_numpy(K).permute(1, 0, 2).repeat_interleave(Hq // Hkv, 0)  # [Hq, L, D]
        v = torch.from_numpy(V).permute(1, 0, 2).repeat_interleave(Hq // Hkv, 0)
        allowed = torch.arange(c + n)[None, :] <= (c + torch.arange(n))[:, None]
        o = torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=allowed, scale=scale)
        out[qs:qs + n] = o.permute(1, 0, 2).numpy()
    return out


@pytest.mark.parametrize("seed", range(4))
def test_matches_torch_sdpa_fp64(seed):
    spec = I.random_small_step(seed, max_seqs=4, max_n=40, max_c=90)
    data = make(spec, seed)
    np.testing.assert_allclose(run(data, SCALE128), sdpa_reference(data, SCALE128), rtol=0, atol=1e-12)


# ---------------------------------------------------------------- closed forms

def test_zero_query_gives_prefix_mean():
    spec = I.StepSpec("z", [I.Seq(9, 5, 0), I.Seq(1, 11, 1)])
    data = make(spec, 3)
    data.q[:] = 0
    out, absv = run(data, SCALE128, with_abs=True)
    for s in range(2):
        qs, n, c = (int(x) for x in data.desc[s])
        V = np.concatenate([f64(data.v_hist[s]), f64(data.v_new[qs:qs + n])])
        csum = np.cumsum(V, axis=0)
        asum = np.cumsum(np.abs(V), axis=0)
        for i in range(n):
            p = c + i
            want = csum[p] / (p + 1)                              # [Hkv, D]
            np.testing.assert_allclose(out[qs + i], np.repeat(want, 8, axis=0), rtol=0, atol=1e-13)
            np.testing.assert_allclose(absv[qs + i], np.repeat(asum[p] / (p + 1), 8, axis=0), rtol=0, atol=1e-13)


def test_equal_keys_give_prefix_mean():
    spec = I.StepSpec("eq", [I.Seq(6, 3, 0)])
    data = make(spec, 4)
    data.k_hist[0][:] = data.k_hist[0][0]
    data.k_new[:] = data.k_hist[0][0]
    out = run(data, SCALE128)
    V = np.concatenate([f64(data.v_hist[0]), f64(data.v_new)])
    for i in range(6):
        want = V[:4 + i].mean(axis=0)
        np.testing.assert_allclose(out[i], np.repeat(want, 8, axis=0), rtol=0, atol=1e-13)


def test_single_visible_key_returns_its_value_exactly():
    spec = I.StepSpec("one", [I.Seq(3, 0, 0)])
    data = make(spec, 5)
    out, absv = run(data, SCALE128, with_abs=True)
    assert np.array_equal(out[0], np.repeat(f64(data.v_new[0]), 8, axis=0))
    assert np.array_equal(absv[0], np.abs(out[0]))


def test_two_key_softmax_closed_form():
    # one head, D=2; logits 0 and x at keys 0 and 1 -> weights 1/(1+e^x), e^x/(1+e^x)
    spec = I.StepSpec("two", [I.Seq(2, 0, 0)], n_q_heads=1, n_kv_heads=1, head_dim=2)
    data = make(spec, 0)
    data.q[:] = bits([[[1.0, 0.0]], [[1.0, 0.0]]])
    data.k_new[:] = bits([[[0.0, 5.0]], [[1.5, -2.0]]])
    data.v_new[:] = bits([[[2.0, -1.0]], [[-3.0, 0.5]]])
    out = run(data, 1.0)
    x = 1.5
    w1 = math.exp(x) / (1 + math.exp(x))
    np.testing.assert_allclose(out[0, 0], [2.0, -1.0], rtol=0, atol=0)
    np.testing.assert_allclose(out[1, 0], [(1 - w1) * 2.0 + w1 * -3.0, (1 - w1) * -1.0 + w1 * 0.5], rtol=0, atol=1e-15)


@pytest.mark.parametrize("where", ["at_p", "past_p", "prefix"])
def test_planted_key(where):
    """A key aligned with the query and scaled far up takes all the weight if visible and
    none if it lies one position past the row: catches off-by-one masks."""
    c, n = 20, 6
    spec = I.StepSpec("plant", [I.Seq(n, c, 0)], n_q_heads=8, n_kv_heads=1)
    data = make(spec, 7)
    i = 3                                   # row at position 23
    p = c + i
    j = {"at_p": p, "past_p": p + 1, "prefix": 5}[where]
    qrow = f64(data.q[i, 0])
    kplant = bits(qrow * 4.0)               # q.k ~ 4*|q|^2 ~ 512 -> dominant after scaling
    data.q[i, 1:] = data.q[i, 0]
    if j < c:
        data.k_hist[0][j, 0] = kplant
    else:
        data.k_new[j - c, 0] = kplant
    out = run(data, SCALE128)
    V = np.concatenate([f64(data.v_hist[0]), f64(data.v_new)])
    if where == "past_p":
        # the planted key is invisible: result equals attention without it
        data2 = make(spec, 7)
        data2.q[i, 1:] = data2.q[i, 0]
        ref = run(data2, SCALE128)
        np.testing.assert_allclose(out[i], ref[i], rtol=0, atol=1e-14)
        assert np.abs(out[i, 0] - V[j, 0]).max() > 0.05
    else:
        np.testing.assert_allclose(out[i, 0], V[j, 0], rtol=0, atol=1e-9)


# ---------------------------------------------------------------- invariants

def chunked_outputs(q, k, v, chunks, scale, Hkv):
    """Run a prefill of len(q) tokens as consecutive chunks (separate steps)."""
    outs, c = [], 0
    for m in chunks:
        desc = np.array([[0, m, c]], dtype=np.int32)
        o = OA.mixed_step_attention(q[c:c + m], desc, [k[:c + m]], [v[:c + m]], scale, Hkv)
        outs.append(o)
        c += m
    return np.concatenate(outs)


@pytest.mark.parametrize("mbt", [1, 7, 16, 64, 2048, 16384])
def test_chunking_invariance(mbt):
    L = 150
    g = I.rng(42, 1)
    q = I.normal_bf16(g, (L, 16, 128))
    k = I.normal_bf16(g, (L, 2, 128))
    v = I.normal_bf16(g, (L, 2, 128))
    full = chunked_outputs(q, k, v, [L], SCALE128, 2)
    sizes = []
    rem = L
    while rem:
        sizes.append(min(mbt, rem))
        rem -= sizes[-1]
    np.testing.assert_allclose(chunked_outputs(q, k, v, sizes, SCALE128, 2), full, rtol=0, atol=1e-13)


def test_decode_row_equals_last_prefill_row():
    g = I.rng(43, 1)
    c = 77
    q = I.normal_bf16(g, (c + 1, 16, 128))
    k = I.normal_bf16(g, (c + 1, 2, 128))
    v = I.normal_bf16(g, (c + 1, 2, 128))
    full = OA.mixed_step_attention(q, np.array([[0, c + 1, 0]]), [k], [v], SCALE128, 2)
    dec = OA.mixed_step_attention(q[c:], np.array([[0, 1, c]]), [k], [v], SCALE128, 2)
    np.testing.assert_allclose(dec[0], full[c], rtol=0, atol=1e-13)


def test_gqa_identical_queries_in_group_give_identical_outputs():
    spec = I.StepSpec("g", [I.Seq(5, 9, 0), I.Seq(1, 30, 1)])
    data = make(spec, 8)
    data.q[:, 0:8] = data.q[:, 3:4]
    data.q[:, 8:16] = data.q[:, 12:13]
    out = run(data, SCALE128)
    for h in range(8):
        assert np.array_equal(out[:, h], out[:, 0])
        assert np.array_equal(out[:, 8 + h], out[:, 8])
    assert not np.allclose(out[:, 0], out[:, 8])


def test_gqa_equals_mha_with_repeated_kv():
    spec = I.StepSpec("g", [I.Seq(4, 6, 0), I.Seq(1, 12, 1)])
    data = make(spec, 9)
    out = run(data, SCALE128)
    rep = I.StepData(data.spec, data.desc, data.q, np.repeat(data.k_new, 8, axis=1), np.repeat(data.v_new, 8, axis=1),
                     [np.repeat(x, 8, axis=1) for x in data.k_hist], [np.repeat(x, 8, axis=1) for x in data.v_hist])
    np.testing.assert_allclose(run(rep, SCALE128), out, rtol=0, atol=1e-14)


def test_swapping_kv_heads_permutes_query_head_groups():
    spec = I.StepSpec("g", [I.Seq(4, 6, 0)])
    data = make(spec, 10)
    out = run(data, SCALE128)
    sw = I.StepData(data.spec, data.desc, np.concatenate([data.q[:, 8:], data.q[:, :8]], axis=1),
                    data.k_new[:, ::-1].copy(), data.v_new[:, ::-1].copy(),
                    [x[:, ::-1].copy() for x in data.k_hist], [x[:, ::-1].copy() for x in data.v_hist])
    o2 = run(sw, SCALE128)
    np.testing.assert_allclose(o2[:, 8:], out[:, :8], rtol=0, atol=1e-14)
    np.testing.assert_allclose(o2[:, :8], out[:, 8:], rtol=0, atol=1e-14)


def test_batch_and_order_independence():
    spec = I.random_small_step(11, max_seqs=5, max_n=30, max_c=60)
    data = make(spec, 11)
    out = run(data, SCALE128)
    for s, sq in enumerate(spec.seqs):
        alone = make(I.StepSpec("a", [sq]), 11)
        qs, n, _ = (int(x) for x in data.desc[s])
        np.testing.assert_allclose(run(alone, SCALE128), out[qs:qs + n], rtol=0, atol=1e-14)
    rev = I.StepSpec("r", list(reversed(spec.seqs)))
    d2 = make(rev, 11)
    o2 = run(d2, SCALE128)
    for s in range(len(spec.seqs)):
        qs, n, _ = (int(x) for x in data.desc[s])
        r = len(spec.seqs) - 1 - s
        qs2 = int(d2.desc[r, 0])
        np.testing.assert_allclose(o2[qs2:qs2 + n], out[qs:qs + n], rtol=0, atol=1e-14)


def test_sampled_rows_equal_full_rows():
    spec = I.StepSpec("rows", [I.Seq(1, 40, 0), I.Seq(37, 20, 1)])
    data = make(spec, 12)
    full = run(data, SCALE128)
    rows = [0, 1, 5, 36, 37]
    part = run(data, SCALE128, rows=rows)
    np.testing.assert_allclose(part[rows], full[rows], rtol=0, atol=1e-14)
    others = np.setdiff1d(np.arange(38), rows)
    assert np.isnan(part[others]).all()


# ---------------------------------------------------------------- mutation test

MUTANTS = {
    "exclusive_diagonal": ("np.arange(kf.shape[0])[None, :] > pos[:, None]", "np.arange(kf.shape[0])[None, :] >= pos[:, None]"),
    "sees_one_future_key": ("np.arange(kf.shape[0])[None, :] > pos[:, None]", "np.arange(kf.shape[0])[None, :] > pos[:, None] + 1"),
    "interleaved_head_groups": ("hs = slice(g * G, (g + 1) * G)", "hs = slice(g, Hq, n_kv_heads)"),
    "missing_scale": ("logits = scale * (qf", "logits = (qf"),
    "missing_normalisation": ("@ vf).reshape(r, G, D) / den", "@ vf).reshape(r, G, D)"),
    "history_after_new": ("parts.insert(0, np.asarray(hist_bits, dtype=np.uint16))", "parts.append(np.asarray(hist_bits, dtype=np.uint16))"),
    "positions_from_zero": ("_attend(qf, K[:nk, g, :], V[:nk, g, :], c + blk, scale, with_abs)",
                            "_attend(qf, K[:nk, g, :], V[:nk, g, :], blk, scale, with_abs)"),
    "bf16_low_half": ("(b.astype(np.uint32) << 16)", "(b.astype(np.uint32) << 15)"),
    # the entry point's assembly of each request's keys and values
    "entry_history_and_new_swapped": ("ks.append(logical_kv(data.k_hist[s], data.k_new[qs:qs + n]))",
                                      "ks.append(logical_kv(data.k_new[qs:qs + n], data.k_hist[s]))"),
    "entry_new_rows_from_zero": ("data.k_new[qs:qs + n]))", "data.k_new[0:n]))"),
    "entry_values_from_keys": ("vs.append(logical_kv(data.v_hist[s], data.v_new[qs:qs + n]))",
                               "vs.append(logical_kv(data.k_hist[s], data.k_new[qs:qs + n]))"),
    # the weighted |V| output
    "abs_of_signed_values": ("@ np.abs(vf)", "@ vf"),
}


def mutant(name):
    src = open(OA.__file__).read()
    a, b = MUTANTS[name]
    assert src.count(a) == 1, name
    mod = types.ModuleType("oracle_mutant_" + name)
    exec(compile(src.replace(a, b), "<mutant>", "exec"), mod.__dict__)
    return mod


def pins_pass(mod) -> bool:
    """The brute-force and library pins, run against a candidate oracle module."""
    try:
        for seed in range(3):
            d = make(tiny_spec(seed), seed)
            o, a = run(d, 0.37, mod, with_abs=True)
            bo, ba = brute_force(d, 0.37, with_abs=True)
            if not (np.allclose(o, bo, rtol=0, atol=1e-12) and np.allclose(a, ba, rtol=0, atol=1e-12)):
                return False
        spec = I.random_small_step(1, max_seqs=4, max_n=40, max_c=90)
        d = make(spec, 1)
        if not np.allclose(run(d, SCALE128, mod), sdpa_reference(d, SCALE128), rtol=0, atol=1e-12):
            return False
    except Exception:
        return False
    return True


def test_pins_accept_the_oracle():
    assert pins_pass(OA)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_planted_mistake(name):
    assert not pins_pass(mutant(name)), f"mutant {name} survived the pins"
