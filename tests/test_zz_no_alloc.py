"""ppas_attn_step_noalloc (the entry point for callers that cannot allocate)
against ppas_attn_step, through the C ABI.

Both calls run the same plan and kernels, so their outputs must be bit-identical;
each is also held to the oracle gates (max |gpu - oracle| <= 1e-2, mean <= 1e-3).
Two calls in a row share the library's fixed device array: the first a step with
~35 MB of split partials, the second a smaller step, so the second call runs on
the first call's leftovers. A step too large for the array must be refused with
nothing enqueued.
"""
import numpy as np
import pytest

import oracle.attention as OA
from paper_2608_15171_amd import inputs as I

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lib():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2608_15171_amd import ppas, step
    return ppas, step, torch


def _step(lib, spec, seed):
    ppas, step, torch = lib
    data = I.make_step_data(spec, seed)
    bt, npages = I.make_block_table(spec, seed, spare_pages=3)
    ds = step.DeviceStep(data, bt, npages)
    ds.fill_history()
    ds.append()
    torch.cuda.synchronize()
    return data, ds


def _both(lib, ds):
    """(ppas_attn_step output, ppas_attn_step_noalloc output) as bf16 bit patterns."""
    ppas, step, torch = lib
    ds.out.zero_()
    ds.attend()
    torch.cuda.synchronize()
    ref = step.bits_of(ds.out).copy()
    ds.out.zero_()
    ppas.attn_step_noalloc(ds.shape, ds.out, ds.q, ds.k_pages, ds.v_pages, ds.desc, ds.bt, ds.bt_host)
    torch.cuda.synchronize()
    return ref, step.bits_of(ds.out).copy()


def _gates(ds, data, rows):
    ref = OA.step_attention_from_data(data, ds.shape.scale, rows=rows)   # full size, these rows filled
    err = np.abs(ds.out_f64()[rows] - ref[rows])
    assert np.isfinite(err).all() and err.max() <= 1e-2 and err.mean() <= 1e-3, (err.max(), err.mean())
    return float(err.max())


def test_noalloc_two_calls_match_attn_step(lib):
    ppas, step, torch = lib
    # first call: the 2,048-token chunk at 22,528 plus 8 decode rows (split rows
    # with ~35 MB of partials in the fixed array)
    spec = I.config_small_budget(0)
    data, ds = _step(lib, spec, 0)
    print(f"noalloc call 1: {spec.name} rows={spec.n_rows}", flush=True)
    a, b = _both(lib, ds)
    assert np.array_equal(a, b), f"{int((a != b).sum())} output elements differ from ppas_attn_step"
    rows = np.r_[0:8, 8:24, spec.n_rows - 16:spec.n_rows]   # decode rows, first and last chunk rows
    print(f"  max_abs vs oracle {_gates(ds, data, rows):.2e}", flush=True)
    del ds
    torch.cuda.empty_cache()
    # second call, smaller: a 512-token chunk plus 4 decode rows of 1,024 keys
    spec = I.config_small(0)
    data, ds = _step(lib, spec, 0)
    print(f"noalloc call 2: {spec.name} rows={spec.n_rows}", flush=True)
    a, b = _both(lib, ds)
    assert np.array_equal(a, b), f"{int((a != b).sum())} output elements differ from ppas_attn_step"
    print(f"  max_abs vs oracle {_gates(ds, data, np.arange(spec.n_rows)):.2e}", flush=True)


def test_noalloc_refuses_step_beyond_the_array(lib):
    ppas, step, torch = lib
    # 1,000 decode rows of 30,001 keys plus two 1,024-token chunks: ~72 MB of split
    # partials, more than the array holds. Every buffer the step names exists and
    # every block-table entry is page 0 of a one-page pool, so nothing could be
    # read out of bounds even if a launch were made.
    d, qs = [], 0
    for _ in range(1000):
        d.append((qs, 1, 30000))
        qs += 1
    for c in (12000, 5000):
        d.append((qs, 1024, c))
        qs += 1024
    desc = np.array(d, dtype=np.int32)
    shape = ppas.make_shape(num_pages=1)
    stride = (30001 + 15) // 16   # pages of the longest request
    bt = torch.zeros((len(desc), stride), dtype=torch.int32, device="cuda")
    q = torch.zeros((qs, 16, 128), dtype=torch.bfloat16, device="cuda")
    out = torch.zeros_like(q)
    kp = torch.zeros((1, 2, 16, 16, 8), dtype=torch.bfloat16, device="cuda")
    vp = torch.zeros((1, 2, 128, 16), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ppas.PPASError) as ex:
        ppas.attn_step_noalloc(shape, out, q, kp, vp, desc, bt)
    assert ex.value.status == ppas.PPAS_ENOSPACE
    torch.cuda.synchronize()
    assert int(out.view(torch.int16).abs().sum()) == 0
