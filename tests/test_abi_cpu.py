"""The C ABI on the CPU: the library loads, exports every declared entry point,
validates step descriptions without touching a GPU, and plans work that covers
every visible (row, head, key) triple exactly once."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2608_15171_amd import inputs as I

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ppas = pytest.importorskip("paper_2608_15171_amd.ppas", reason="libppas.so not built")


def declared_functions():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            txt = open(os.path.join(ROOT, "include", fn)).read()
            txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
            names |= set(re.findall(r"\b(ppas_[a-z_0-9]+)\s*\(", txt))
    return sorted(names)


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) >= 7
    lib = ctypes.CDLL(ppas.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings():
    for st in (0, -1, -2, -3, -4, -5):
        assert ppas.status_string(st).startswith("PPAS_")
    assert "unknown" in ppas.status_string(7)


def shape(**kw):
    base = dict(n_q_heads=16, n_kv_heads=2, num_pages=100)
    base.update(kw)
    return ppas.make_shape(**base)


GOOD = np.array([[0, 1, 30], [1, 20, 5]], dtype=np.int32)
BT = np.array([[0, 1, -1], [2, 3, -1]], dtype=np.int32)


def test_validate_good_and_empty():
    assert ppas.validate_step(shape(), GOOD, BT) == ppas.PPAS_OK
    assert ppas.validate_step(shape(), np.zeros((0, 3), np.int32), None, 1) == ppas.PPAS_OK


@pytest.mark.parametrize("desc,code", [
    ([[0, 0, 30], [0, 20, 5]], "EINVAL"),          # n_query 0
    ([[0, 1, -1], [1, 20, 5]], "EINVAL"),          # negative cached_len
    ([[1, 1, 30], [2, 20, 5]], "EINVAL"),          # query_start not from 0
    ([[0, 1, 30], [2, 20, 5]], "EINVAL"),          # gap between requests
    ([[0, 1, 60], [1, 20, 5]], "EINVAL"),          # 61 tokens need 4 pages > stride 3
])
def test_validate_bad_descriptors(desc, code):
    assert ppas.validate_step(shape(), np.array(desc, np.int32), BT) == getattr(ppas, "PPAS_" + code)


def test_validate_shapes():
    assert ppas.validate_step(shape(head_dim=64), GOOD, BT) == ppas.PPAS_EUNSUPPORTED
    assert ppas.validate_step(shape(page_size=32), GOOD, BT) == ppas.PPAS_EUNSUPPORTED
    assert ppas.validate_step(shape(n_q_heads=8), GOOD, BT) == ppas.PPAS_EUNSUPPORTED
    assert ppas.validate_step(shape(n_q_heads=8, n_kv_heads=1), GOOD, BT) == ppas.PPAS_OK
    assert ppas.validate_step(shape(n_q_heads=15), GOOD, BT) == ppas.PPAS_EINVAL
    for sc in (0.0, -1.0, float("nan"), float("inf")):
        assert ppas.validate_step(shape(scale=sc), GOOD, BT) == ppas.PPAS_EINVAL
    assert ppas.validate_step(shape(num_pages=0), GOOD, BT) == ppas.PPAS_EINVAL


def test_validate_block_table_range_and_overlap():
    assert ppas.validate_step(shape(num_pages=3), GOOD, BT) == ppas.PPAS_ERANGE
    bad = BT.copy()
    bad[1, 0] = -1
    assert ppas.validate_step(shape(), GOOD, bad) == ppas.PPAS_ERANGE
    # request 0 writes position 30 -> (page 1, slot 14); request 1 writes 5..24 -> (page 2, 5..15), (page 1, 0..8)
    ov = np.array([[0, 1, -1], [2, 1, -1]], np.int32)
    assert ppas.validate_step(shape(), GOOD, ov) == ppas.PPAS_OK       # different slots of page 1
    # request 0 at position 21 -> (page 1, slot 5); request 1 writes (page 1, slots 5..15): a clash
    ov2 = np.array([[0, 1, -1], [1, 3, -1]], np.int32)
    assert ppas.validate_step(shape(), np.array([[0, 1, 21], [1, 20, 5]], np.int32), ov2) == ppas.PPAS_EINVAL


def test_validation_cost_does_not_grow_with_the_pool():
    """The write-overlap check follows the pages a step writes: a step of 64 requests
    over a pool of a million pages validates about as fast as over a pool just large
    enough for it (the check once zeroed a bitmap of the whole pool per call)."""
    import time
    g = I.rng(5, 1)
    seqs = [I.Seq(1, int(c), i) for i, c in enumerate(g.integers(20000, 30000, size=60))]
    seqs += [I.Seq(1024, 4096 * k, 60 + k) for k in range(4)]
    spec = I.StepSpec("pool", seqs)
    desc = spec.descriptors()
    need = int(spec.pages_per_seq().sum())

    def best(num_pages):
        bt, _ = I.make_block_table(spec, 5, spare_pages=num_pages - need)
        sh = shape(num_pages=num_pages)
        assert ppas.validate_step(sh, desc, bt) == ppas.PPAS_OK
        ts = []
        for _ in range(30):
            t0 = time.perf_counter()
            ppas.validate_step(sh, desc, bt)
            ts.append(time.perf_counter() - t0)
        return min(ts)

    small, large = best(need), best(1 << 20)
    print(f"validate: {need} pages {small * 1e6:.1f} us, 1M pages {large * 1e6:.1f} us")
    assert large < 2.0 * small + 20e-6


def test_calls_reject_bad_input_before_any_device_work():
    import torch
    sh = shape()
    st = ppas._lib.ppas_attn_step(ctypes.byref(sh), None, None, None, None, GOOD.ctypes.data, 2, None, 3,
                                  BT.ctypes.data, None, 0, None)
    assert st == ppas.PPAS_EINVAL
    bad = np.array([[0, 0, 1]], np.int32)
    st = ppas._lib.ppas_kv_append(ctypes.byref(sh), 1, 1, 1, 1, bad.ctypes.data, 1, 1, 3, None, None)
    assert st == ppas.PPAS_EINVAL
    assert ppas.attn_workspace_bytes(sh, bad) == 0
    assert ppas.attn_workspace_bytes(sh, GOOD) > 0
    for theta in (0.0, -1.0, float("nan"), float("inf")):
        st = ppas._lib.ppas_rope_kv_append(ctypes.byref(sh), theta, 1, 1, 1, 1, 1, GOOD.ctypes.data, 2,
                                           1, 3, BT.ctypes.data, None)
        assert st == ppas.PPAS_EINVAL, theta
    st = ppas._lib.ppas_rope_kv_append(ctypes.byref(sh), 1e6, 1, 1, 1, 1, 1, bad.ctypes.data, 1, 1, 3, None, None)
    assert st == ppas.PPAS_EINVAL
    st = ppas._lib.ppas_rope_kv_append(ctypes.byref(sh), 1e6, None, 1, 1, 1, 1, GOOD.ctypes.data, 2, 1, 3,
                                       BT.ctypes.data, None)
    assert st == ppas.PPAS_EINVAL                               # no q


def test_noalloc_refuses_oversized_steps_on_the_host():
    """ppas_attn_step_noalloc checks the step against its fixed device array before
    any HIP work: 1,000 decode rows of 30,001 keys plus two 1,024-token chunks need
    ~72 MB of split partials (> PPAS_NOALLOC_SCRATCH_BYTES = 64 MiB)."""
    d, qs = [], 0
    for _ in range(1000):
        d.append((qs, 1, 30000))
        qs += 1
    for c in (12000, 5000):
        d.append((qs, 1024, c))
        qs += 1024
    desc = np.array(d, dtype=np.int32)
    sh = shape(num_pages=10 ** 6)
    assert ppas.attn_workspace_bytes(sh, desc) > 64 << 20
    st = ppas._lib.ppas_attn_step_noalloc(ctypes.byref(sh), 1, 1, 1, 1, desc.ctypes.data, len(desc), 1, 1876,
                                          None, None)
    assert st == ppas.PPAS_ENOSPACE
    st = ppas._lib.ppas_attn_step_noalloc(ctypes.byref(sh), None, 1, 1, 1, GOOD.ctypes.data, 2, 1, 3, None, None)
    assert st == ppas.PPAS_EINVAL                               # no output buffer
    bad = np.array([[0, 0, 1]], np.int32)
    st = ppas._lib.ppas_attn_step_noalloc(ctypes.byref(sh), 1, 1, 1, 1, bad.ctypes.data, 1, 1, 3, None, None)
    assert st == ppas.PPAS_EINVAL                               # bad descriptor


def test_gateup_proj_validates_before_any_device_work():
    f = ppas._lib.ppas_gateup_proj
    assert f(1, 1, 1, 0, 64, 8, None, 0, None, None) == ppas.PPAS_OK                 # no tokens: nothing to do
    assert f(1, 1, 1, 4, 96, 8, None, 0, None, None) == ppas.PPAS_EUNSUPPORTED       # hidden not a multiple of 64
    assert f(1, 1, 1, -1, 64, 8, None, 0, None, None) == ppas.PPAS_EINVAL
    assert f(1, 1, 1, 4, 0, 8, None, 0, None, None) == ppas.PPAS_EINVAL
    assert f(1, 1, 1, 4, 64, 0, None, 0, None, None) == ppas.PPAS_EINVAL
    assert f(None, 1, 1, 4, 64, 8, None, 0, None, None) == ppas.PPAS_EINVAL
    assert f(1, 1, 1, 4, 64, 8, None, 1024, None, None) == ppas.PPAS_EINVAL         # workspace size without a buffer
    assert f(1, 1, 1, 2 ** 31 - 1, 64, 8, None, 0, None, None) == ppas.PPAS_ERANGE
    half = ppas.events(start=1)
    assert f(1, 1, 1, 4, 64, 8, None, 0, ctypes.byref(half), None) == ppas.PPAS_EINVAL   # start without stop


def test_gateup_workspace_sizing():
    """Split reductions only when the 256 x 256 tiles are fewer than the compute units
    (256 without a device): one tile row of 22016 columns does not split; a decode-sized
    down projection (16 tokens, 11008 -> 2048: 8 tiles) splits 32 ways, a 2k chunk's
    (64 tiles) 4 ways."""
    W = ppas.gateup_workspace_bytes
    assert W(2048, 2048, 22016) == 0
    assert W(16, 11008, 2048) == 32 * 16 * 2048 * 4
    assert W(2048, 11008, 2048) == 4 * 2048 * 2048 * 4
    assert W(16, 2048, 2048) == 8 * 16 * 2048 * 4       # at least four 64-feature stages per split
    assert W(0, 2048, 2048) == 0 and W(4, 96, 8) == 0


def test_gateup_act_validates_before_any_device_work():
    f = ppas._lib.ppas_gateup_act
    assert f(1, 1, 1, 0, 64, 4, None, 0, None, None) == ppas.PPAS_OK                 # no tokens: nothing to do
    assert f(1, 1, 1, 4, 96, 4, None, 0, None, None) == ppas.PPAS_EUNSUPPORTED       # hidden not a multiple of 64
    assert f(1, 1, 1, -1, 64, 4, None, 0, None, None) == ppas.PPAS_EINVAL
    assert f(1, 1, 1, 4, 64, 0, None, 0, None, None) == ppas.PPAS_EINVAL            # no intermediate features
    assert f(1, 1, 1, 4, 64, -3, None, 0, None, None) == ppas.PPAS_EINVAL
    assert f(1, 1, None, 4, 64, 4, None, 0, None, None) == ppas.PPAS_EINVAL
    assert f(1, 1, 1, 4, 64, 2 ** 30, None, 0, None, None) == ppas.PPAS_ERANGE     # 2 n_inter weight rows overflow
    assert f(1, 1, 1, 4, 64, 4, None, 1024, None, None) == ppas.PPAS_EINVAL
    half = ppas.events(stop=1)
    assert f(1, 1, 1, 4, 64, 4, None, 0, ctypes.byref(half), None) == ppas.PPAS_EINVAL


def test_stream_read_validates_before_any_device_work():
    """Only argument errors and the empty read: each returns before the device is touched."""
    f = ppas._lib.ppas_stream_read
    assert f(16, 0, 16, None, None) == ppas.PPAS_OK                  # nothing to read
    assert f(16, 24, 16, None, None) == ppas.PPAS_EINVAL             # not whole 16-byte words
    assert f(8, 16, 16, None, None) == ppas.PPAS_EINVAL              # buffer not 16-byte aligned
    assert f(16, 16, 2, None, None) == ppas.PPAS_EINVAL              # sink not 4-byte aligned
    assert f(None, 16, 16, None, None) == ppas.PPAS_EINVAL
    assert f(16, 16, None, None, None) == ppas.PPAS_EINVAL
    half = ppas.events(start=1)
    assert f(16, 0, 16, ctypes.byref(half), None) == ppas.PPAS_EINVAL


def test_gateup_act_workspace_is_the_projection_s():
    """The activated projection splits like the projection of its 2 n_inter weight rows
    (its partials keep the weight-row layout)."""
    for T, H, I in ((16, 2048, 11008), (2048, 2048, 11008), (16, 2048, 1024), (300, 128, 40)):
        assert ppas.gateup_act_workspace_bytes(T, H, I) == ppas.gateup_workspace_bytes(T, H, 2 * I)
    assert ppas.gateup_act_workspace_bytes(16, 2048, 0) == 0
    assert ppas.gateup_act_workspace_bytes(16, 2048, 2 ** 30) == 0


def check_coverage(spec, items):
    """Every (row, query head) sees keys 0..p split over items without gaps or overlaps,
    and each item gives each of its rows at least one visible key."""
    desc = spec.descriptors()
    cover = {}
    for kind, s, g, row0, pos0, npos, lo, hi in items.tolist():
        qs, n, c = (int(x) for x in desc[s])
        assert kind == (1 if n == 1 else 0)
        assert qs <= row0 and row0 + npos <= qs + n and pos0 == c + (row0 - qs)
        for r in range(npos):
            p = pos0 + r
            assert lo <= p, "an item with no visible key for one of its rows"
            for h in range(g * 8, g * 8 + 8):
                cover.setdefault((row0 + r, h), []).append((lo, min(hi, p + 1)))
    assert len(cover) == spec.n_rows * spec.n_q_heads
    for s in range(len(desc)):
        qs, n, c = (int(x) for x in desc[s])
        for i in range(n):
            for h in range(spec.n_q_heads):
                rng = sorted(cover[(qs + i, h)])
                assert rng[0][0] == 0 and rng[-1][1] == c + i + 1
                for a, b in zip(rng, rng[1:]):
                    assert a[1] == b[0]


@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("splits", [(0, 0), (64, 32), (128, 96)])
@pytest.mark.parametrize("tile", [16, 32])
def test_plan_covers_visible_keys_once(seed, splits, tile):
    spec = I.random_small_step(seed, max_seqs=6, max_n=70, max_c=300)
    opts = ppas.plan_opts(splits[0], splits[1], tile)
    items = ppas.plan_items(shape(), spec.descriptors(), num_cus=256, opts=opts)
    check_coverage(spec, items)
    assert items[items[:, 0] == 0, 5].max(initial=0) <= tile


def test_tile_shape_choice():
    """32-position tiles only for steps whose prefill fills the chip on its own and whose
    decode work is a small share; every other step keeps 16-position tiles."""
    def npos_max(spec):
        items = ppas.plan_items(shape(), spec.descriptors(), num_cus=256)
        return int(items[items[:, 0] == 0, 5].max())
    assert npos_max(I.config_large_budget(0)) == 32        # one 16,384-token chunk
    assert npos_max(I.config_small_budget(0)) == 16        # 2,048-token chunk: too few large tiles
    assert npos_max(I.config_small(0)) == 16
    assert npos_max(I.config_high_pressure(0)) == 16       # decode-heavy
    heavy = I.StepSpec("16k+decodes", [I.Seq(1, 25000, i) for i in range(40)] + [I.Seq(16384, 8616, 99)])
    assert npos_max(heavy) == 16
    for bad in (ppas.plan_opts(tile_positions=24), ppas.plan_opts(prefill_split=-1), ppas.plan_opts(decode_split=-5),
                ppas.plan_opts(num_cus=-1)):
        with pytest.raises(ppas.PPASError):
            ppas.plan_items(shape(), I.config_small(0).descriptors(), opts=bad)


def test_options_are_per_call():
    """Planning choices travel with the call: a plan made with forced splits does not
    change the plan of the next call without them."""
    spec = I.config_small_budget(0)
    base = ppas.plan_items(shape(), spec.descriptors())
    forced = ppas.plan_items(shape(), spec.descriptors(), opts=ppas.plan_opts(64, 32, 32))
    again = ppas.plan_items(shape(), spec.descriptors())
    assert not np.array_equal(base, forced) and np.array_equal(base, again)
    assert forced[forced[:, 0] == 0, 5].max() == 32


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_plan_covers_workloads(cfg):
    spec = I.CONFIGS[cfg](0)
    items = ppas.plan_items(shape(), spec.descriptors(), num_cus=256)
    if cfg in (1, 2):
        check_coverage(spec, items)
    # longest first within each kind: the first eighth of a kind's items holds at
    # least as many keys on average as its last eighth
    for kind in (0, 1):
        span = (items[:, 7] - items[:, 6])[items[:, 0] == kind]
        if len(span):
            k = max(1, len(span) // 8)
            assert span[:k].mean() >= span[-k:].mean()
    dec_at = np.flatnonzero(items[:, 0] == 1)
    if cfg in (1, 4):
        # decode work comparable to the prefill work: the kinds are interleaved,
        # each advancing through the launch at about the same fraction of its work
        assert 0 < len(dec_at) < len(items)
        assert dec_at.min() < len(items) // 4 and dec_at.max() >= len(items) * 3 // 4
    elif len(dec_at):
        # decode a small share of the step: decode items fill the tail
        assert np.array_equal(dec_at, np.arange(len(items) - len(dec_at), len(items)))


def test_plan_is_deterministic():
    spec = I.config_high_pressure(0)
    a = ppas.plan_items(shape(), spec.descriptors())
    b = ppas.plan_items(shape(), spec.descriptors())
    assert np.array_equal(a, b)


@pytest.mark.parametrize("decode_split", [0, 8192, 1 << 20])
def test_decode_items_never_exceed_the_page_id_capacity(decode_split):
    """A decode work item holds the page ids of its blocks in lane registers (32 blocks of
    32 keys per register; four registers per wave of the four-wave kernel, two per wave of
    the eight-wave one): its key range is capped at 16,384 keys, also when a larger split
    is requested."""
    spec = I.StepSpec("long-decodes", [I.Seq(1, c, i) for i, c in enumerate([0, 8191, 8192, 60000, 300000])])
    items = ppas.plan_items(shape(), spec.descriptors(), num_cus=8, opts=ppas.plan_opts(0, decode_split))
    dec = items[items[:, 0] == 1]
    assert (dec[:, 7] - dec[:, 6]).max() <= 16384
    assert (dec[:, 6] % 32 == 0).all(), "decode key ranges start on 32-key blocks"
    check_coverage(spec, items)


@pytest.mark.parametrize("num_cus", [256, 80])
def test_decode_only_steps_take_even_pieces_about_one_per_cu(num_cus):
    """A step of decode rows only: each (row, KV head) stream is cut into even pieces
    on 32-key blocks, about one item per CU over the step; an explicit decode split
    keeps the fixed-size pieces."""
    spec = I.config_pressure_decode_only(0)
    items = ppas.plan_items(shape(), spec.descriptors(), num_cus=num_cus)
    assert (items[:, 0] == 1).all()
    kend = np.array([c + 1 for _, _, c in spec.descriptors().tolist()] * 2)     # one stream per KV head
    want = np.maximum(-(-kend // (16384 - 32)), (kend * num_cus + kend.sum() // 2) // kend.sum())
    assert len(items) == want.sum(), (len(items), want.sum())
    if num_cus == 256:
        assert 0.8 * num_cus <= len(items) <= 1.25 * num_cus, len(items)
    assert (items[:, 6] % 32 == 0).all() and (items[:, 7] - items[:, 6]).max() <= 16384
    for (s, g) in {(int(a), int(b)) for a, b in items[:, 1:3]}:
        mine = items[(items[:, 1] == s) & (items[:, 2] == g)]
        span = mine[:, 7] - mine[:, 6]
        assert span.max() - span.min() < 64, (s, g, span)     # boundaries on 32-key blocks
    check_coverage(spec, items)
    fixed = ppas.plan_items(shape(), spec.descriptors(), num_cus=num_cus, opts=ppas.plan_opts(0, 4096))
    assert ((fixed[:, 7] - fixed[:, 6]) <= 4096).all() and (fixed[:, 6] % 4096 == 0).all()


def test_binding_fails_loudly_without_the_library(tmp_path):
    """No fallback: a copy of the package without libppas.so refuses to import its
    binding (and the device-step module built on it)."""
    import shutil
    import subprocess
    import sys
    src = os.path.dirname(ppas.__file__)
    dst = tmp_path / "paper_2608_15171_amd"
    dst.mkdir()
    for name in os.listdir(src):
        if name.endswith(".py"):
            shutil.copy(os.path.join(src, name), dst / name)
    for mod in ("paper_2608_15171_amd.ppas", "paper_2608_15171_amd.step"):
        r = subprocess.run([sys.executable, "-c", f"import {mod}"], cwd=tmp_path, capture_output=True, text=True,
                           env={**os.environ, "PYTHONPATH": str(tmp_path)}, timeout=120)
        assert r.returncode != 0, mod
        assert "ImportError" in r.stderr and "libppas.so is missing" in r.stderr, r.stderr[-2000:]
