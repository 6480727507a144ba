"""GPU parity of the rotary embedding fused with the page write (ppas_rope_kv_append)
against the CPU oracle, through the C ABI.

Bound for a rotated element (derived from the arithmetic the kernel states): the
angle is reduced in fp64 and rounded to fp32 (|error| <= 2^-24 * pi), cos/sin in fp32
(about one ulp), the two products and the fused add in fp32, then one rounding to
bf16 (at most half an ulp; with 8 significant bits that is at most 2^-8 of the value).
So
    |gpu - exact| <= 2^-8 |exact| + 1e-6 (|x_i| + |x_{i+64}|),
the second term covering every fp32 step with margin. V is copied: bit-exact. Every
pool byte no request owns keeps its sentinel.
"""
import numpy as np
import pytest

import oracle.attention as OA
import oracle.kv_cache as OK
import oracle.rope as R
from paper_2608_15171_amd import inputs as I

pytestmark = pytest.mark.gpu

SENTINEL = 0xFFFF


@pytest.fixture(scope="module")
def lib():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2608_15171_amd import ppas, step
    return ppas, step, torch


def check_rotated(gpu_bits, ref, x_bits, label):
    gpu = R.bf16_bits_to_f64(gpu_bits)
    x = R.bf16_bits_to_f64(x_bits)
    D = x.shape[-1]
    pair = np.abs(x[..., :D // 2]) + np.abs(x[..., D // 2:])
    tol = 2.0 ** -8 * np.abs(ref) + 1e-6 * np.concatenate([pair, pair], axis=-1)
    err = np.abs(gpu - ref)
    exact = float(np.mean(gpu_bits == R.f64_to_bf16_bits(ref))) if ref.size else 1.0
    worst = float((err / np.maximum(tol, 1e-300)).max()) if ref.size else 0.0
    print(f"{label}: n={ref.size} max_abs={err.max() if ref.size else 0:.3e} worst/tol={worst:.3f} "
          f"rne_equal={exact:.5f}", flush=True)
    assert np.isfinite(gpu).all(), label
    assert (err <= tol).all(), f"{label}: {int((err > tol).sum())} elements beyond the bound"
    assert exact >= 0.98, f"{label}: only {exact:.4f} equal to the nearest-even rounding of the exact value"


def run_rope(lib, spec, seed, theta, permute=True, spare=4):
    ppas, step, torch = lib
    data = I.make_step_data(spec, seed, with_history=False)
    bt, npages = I.make_block_table(spec, seed, permute=permute, spare_pages=spare)
    ds = step.DeviceStep(data, bt, npages, pool_fill=SENTINEL)
    k0, v0 = step.bits_of(ds.k_pages), step.bits_of(ds.v_pages)
    ds.rope_append(theta)
    torch.cuda.synchronize()
    return data, bt, ds, k0, v0


def check_step(lib, spec, seed, theta, label, permute=True):
    ppas, step, torch = lib
    print(f"{label}: seed={seed} theta={theta} seqs={len(spec.seqs)} rows={spec.n_rows}", flush=True)
    data, bt, ds, k0, v0 = run_rope(lib, spec, seed, theta, permute)
    q_ref, k_ref = R.rope_step(data.q, data.k_new, data.desc, theta)
    check_rotated(step.bits_of(ds.q), q_ref, data.q, label + " q")
    kp, vp = step.bits_of(ds.k_pages), step.bits_of(ds.v_pages)
    # V: the oracle's append, bit for bit (untouched slots keep the sentinel)
    assert np.array_equal(vp, R.rope_kv_append(k0, v0, data.q, data.k_new, data.v_new, data.desc, bt, 16, theta)[2])
    # K: each request's new positions hold its rotated keys ...
    for s, (qs, n, c) in enumerate(data.desc.tolist()):
        kg, _ = OK.gather(kp, vp, bt[s], c + n, 16)
        check_rotated(kg[c:], k_ref[qs:qs + n], data.k_new[qs:qs + n], f"{label} k seq{s}")
    # ... and nothing else changed: putting the unrotated keys back where the oracle
    # places them gives the oracle's plain append of the whole pool.
    k_back, _ = OK.append(kp, vp, data.k_new, data.v_new, data.desc, bt, 16)
    assert np.array_equal(k_back, OK.append(k0, v0, data.k_new, data.v_new, data.desc, bt, 16)[0])


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("theta", [1e6, 1e4])
def test_random_steps(lib, seed, theta):
    spec = I.random_small_step(seed, max_seqs=6, max_n=70, max_c=300)
    check_step(lib, spec, seed, theta, "random")


def test_partial_pages_decode_rows_and_position_zero(lib):
    """Chunks starting and ending mid-page, single-token rows, and a request at
    position 0, whose first row must come back bit-identical (angle 0)."""
    ppas, step, torch = lib
    spec = I.StepSpec("edges", [I.Seq(1, 0, 0), I.Seq(1, 15, 1), I.Seq(1, 16, 2), I.Seq(3, 14, 3),
                                I.Seq(17, 31, 4), I.Seq(40, 0, 5)])
    check_step(lib, spec, 7, 1e6, "edges")
    data, bt, ds, _, _ = run_rope(lib, spec, 7, 1e6)
    q = step.bits_of(ds.q)
    assert np.array_equal(q[0], data.q[0])                      # request 0: position 0
    qs5 = int(data.desc[5, 0])
    assert np.array_equal(q[qs5], data.q[qs5])                  # request 5's first row: position 0


def test_more_requests_than_one_launch_takes(lib):
    """Over 64 requests: the host splits the work into several launches."""
    g = np.random.default_rng(11)
    spec = I.StepSpec("many", [I.Seq(int(g.integers(1, 4)), int(g.integers(0, 200)), i) for i in range(150)])
    check_step(lib, spec, 11, 1e6, "many")


def test_tp2_shard_shape(lib):
    spec = I.random_small_step(5, max_seqs=4, max_n=50, max_c=200, n_q_heads=8, n_kv_heads=1)
    check_step(lib, spec, 5, 1e6, "tp2")


@pytest.mark.parametrize("cfg", [2, 3])
def test_full_size_steps(lib, cfg):
    """The MBT=2048 step (positions up to 25,032) and the 16,384-token chunk (positions
    8,616..24,999), every element compared."""
    check_step(lib, I.CONFIGS[cfg](0), 0, 1e6, f"config{cfg}")


def test_identity_block_table_gives_the_same_rows(lib):
    ppas, step, torch = lib
    spec = I.random_small_step(2, max_seqs=5, max_n=40, max_c=100)
    _, _, a, _, _ = run_rope(lib, spec, 2, 1e6, permute=True)
    _, _, b, _, _ = run_rope(lib, spec, 2, 1e6, permute=False)
    assert np.array_equal(step.bits_of(a.q), step.bits_of(b.q))


def test_empty_step_is_a_no_op(lib):
    ppas, step, torch = lib
    spec = I.random_small_step(1, max_seqs=2, max_n=5, max_c=10)
    data, bt, ds, k0, v0 = run_rope(lib, spec, 1, 1e6)
    q1, k1 = step.bits_of(ds.q), step.bits_of(ds.k_pages)
    ppas.rope_kv_append(ds.shape, 1e6, ds.q, ds.k_pages, ds.v_pages, ds.k_new, ds.v_new,
                        np.zeros((0, 3), np.int32), ds.bt, ds.bt_host)
    torch.cuda.synchronize()
    assert np.array_equal(step.bits_of(ds.q), q1) and np.array_equal(step.bits_of(ds.k_pages), k1)


@pytest.mark.parametrize("seed", range(2))
def test_attention_after_rotation(lib, seed):
    """Rotation, then the step's attention, against the oracle's attention over the
    oracle's own rotated rows (rounded to bf16 nearest-even by the oracle)."""
    ppas, step, torch = lib
    spec = I.random_small_step(seed + 20, max_seqs=5, max_n=60, max_c=250)
    data = I.make_step_data(spec, seed)
    bt, npages = I.make_block_table(spec, seed, spare_pages=3)
    ds = step.DeviceStep(data, bt, npages, pool_fill=SENTINEL)
    ds.fill_history()
    ds.rope_append(1e6)
    ds.attend()
    torch.cuda.synchronize()
    q_rot, k_rot = R.rope_step(data.q, data.k_new, data.desc, 1e6)
    rotated = I.StepData(data.spec, data.desc, R.f64_to_bf16_bits(q_rot), R.f64_to_bf16_bits(k_rot), data.v_new,
                         data.k_hist, data.v_hist)
    ref = OA.step_attention_from_data(rotated, ds.shape.scale)
    err = np.abs(ds.out_f64() - ref)
    print(f"attention after rotation seed={seed}: max_abs={err.max():.3e} mean_abs={err.mean():.3e}", flush=True)
    assert err.max() <= 1e-2 and err.mean() <= 1e-3
