"""The seeded input generator (CPU only): bf16 rounding, determinism, descriptor packing,
block-table structure and the four single-step workloads."""
import numpy as np
import pytest
import torch

from paper_2608_15171_amd import inputs as I
from paper_2608_15171_amd import metrics as M


def test_bf16_rounding_matches_torch():
    g = I.rng(0, 1)
    x = np.concatenate([g.standard_normal(100000).astype(np.float32) * 10.0 ** g.integers(-6, 6, 100000),
                        np.float32([0.0, -0.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 65504.0])])
    x = x.astype(np.float32)
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(I.f32_to_bf16_bits(x), want)


def test_request_data_does_not_depend_on_neighbours():
    a = I.make_step_data(I.StepSpec("a", [I.Seq(3, 5, 7)]), 1)
    b = I.make_step_data(I.StepSpec("b", [I.Seq(1, 2, 0), I.Seq(3, 5, 7)]), 1)
    assert np.array_equal(a.q, b.q[1:]) and np.array_equal(a.k_hist[0], b.k_hist[1])


def test_block_table_is_a_partition():
    spec = I.config_high_pressure(0)
    bt, n = I.make_block_table(spec, 0)
    used = bt[bt >= 0]
    assert len(np.unique(used)) == len(used) == n
    for s, k in enumerate(spec.pages_per_seq()):
        assert (bt[s, :k] >= 0).all() and (bt[s, k:] == -1).all()


def test_workload_shapes():
    s1, s2, s3, s4 = (I.CONFIGS[k](0) for k in (1, 2, 3, 4))
    assert [(q.n_query, q.cached_len) for q in s1.seqs] == [(1, 1024)] * 4 + [(512, 0)]
    assert s2.seqs[-1] == I.Seq(2048, 22528, 8) and all(25000 <= q.cached_len <= 25032 for q in s2.seqs[:8])
    assert s3.seqs == [I.Seq(16384, 8616, 0)] and 8616 + 16384 == 25000
    dec = [q for q in s4.seqs if q.n_query == 1]
    pre = [q for q in s4.seqs if q.n_query > 1]
    assert len(dec) == 48 and all(20000 <= q.cached_len <= 30064 for q in dec)
    assert len(pre) == 2 and all(q.n_query == 1024 for q in pre)
    for q, L in zip(pre, s4.info["prompt_lens"]):
        assert 20000 <= L <= 30000 and q.cached_len + 1024 <= L
    assert M.visible_pairs(s3) == 16384 * 8616 + 16384 * 16385 // 2
    assert abs(M.flops(s3) - 2.2560e12) / 2.256e12 < 1e-4


def test_chunk_schedule_covers_the_prompt_once():
    from paper_2608_15171_amd import chunk_replay as CR
    from paper_2608_15171_amd import metrics as M
    specs = CR.chunk_specs(16384, 2048)
    assert len(specs) == 8
    assert [(s.seqs[0].n_query, s.seqs[0].cached_len) for s in specs] == [(2048, 2048 * k) for k in range(8)]
    # chunking changes the schedule, not the work: visible pairs add up to the single chunk's
    single = CR.chunk_specs(16384, 16384)
    assert sum(M.visible_pairs(s) for s in specs) == M.visible_pairs(single[0]) == 16384 * 16385 // 2
    with pytest.raises(ValueError):
        CR.chunk_specs(1000, 300)
    bt = CR.prompt_block_table(0, 16384)
    assert bt.shape == (1, 1024) and sorted(bt[0].tolist()) == list(range(1024))
