"""Pins for the page-scatter oracle (CPU only): a scalar loop over tokens, heads and
features, a hand-worked address example, untouched-slot sentinels, and the
write/read round trip through the block table."""
import numpy as np
import pytest

import oracle.kv_cache as OK
from paper_2608_15171_amd import inputs as I


def scalar_append(kp, vp, k_new, v_new, desc, bt, P):
    kp = kp.copy()
    vp = vp.copy()
    for s in range(len(desc)):
        qs, n, c = (int(x) for x in desc[s])
        for i in range(n):
            pos = c + i
            page, slot = int(bt[s][pos // P]), pos % P
            for g in range(k_new.shape[1]):
                for d in range(k_new.shape[2]):
                    kp[page, g, d // 8, slot, d % 8] = k_new[qs + i, g, d]
                    vp[page, g, d, slot] = v_new[qs + i, g, d]
    return kp, vp


def pools(num_pages, Hkv, P, D, fill=0xFFFF):
    return (np.full((num_pages, Hkv, D // 8, P, 8), fill, np.uint16), np.full((num_pages, Hkv, D, P), fill, np.uint16))


@pytest.mark.parametrize("seed", range(5))
def test_matches_scalar_loop(seed):
    spec = I.random_small_step(seed, max_seqs=4, max_n=20, max_c=40)
    spec.head_dim = 8
    data = I.make_step_data(spec, seed, with_history=False)
    bt, npages = I.make_block_table(spec, seed, permute=True, spare_pages=3)
    kp, vp = pools(npages, 2, 16, 8)
    a = OK.append(kp, vp, data.k_new, data.v_new, data.desc, bt, 16)
    b = scalar_append(kp, vp, data.k_new, data.v_new, data.desc, bt, 16)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_hand_worked_addresses():
    # one request, 14 cached tokens, 3 new: positions 14, 15, 16 with pages [7, 2]
    # -> (page 7, slot 14), (page 7, slot 15), (page 2, slot 0); D = 16 features = 2 key chunks
    P, D = 16, 16
    kp, vp = pools(8, 1, P, D)
    k_new = np.arange(3 * D, dtype=np.uint16).reshape(3, 1, D)
    v_new = k_new + 100
    desc = np.array([[0, 3, 14]])
    bt = np.array([[7, 2]])
    ka, va = OK.append(kp, vp, k_new, v_new, desc, bt, P)
    # key feature d of a token sits in chunk d // 8, at offset d % 8 of that token's slot
    assert ka[7, 0, 0, 14].tolist() == list(range(0, 8)) and ka[7, 0, 1, 14].tolist() == list(range(8, 16))
    assert ka[7, 0, 0, 15].tolist() == list(range(16, 24)) and ka[2, 0, 1, 0].tolist() == list(range(40, 48))
    assert va[7, 0, :, 14].tolist() == list(range(100, 116)) and va[2, 0, :, 0].tolist() == list(range(132, 148))
    changed = (ka != 0xFFFF).sum() + (va != 0xFFFF).sum()
    assert changed == 2 * 3 * D


def test_only_written_slots_change_and_round_trip():
    spec = I.StepSpec("rt", [I.Seq(1, 30, 0), I.Seq(21, 5, 1), I.Seq(16, 16, 2)], head_dim=8)
    data = I.make_step_data(spec, 3)
    bt, npages = I.make_block_table(spec, 3, spare_pages=2)
    kp, vp = pools(npages, 2, 16, 8)
    kp, vp = OK.fill_history(kp, vp, data.k_hist, data.v_hist, bt, 16)
    before = (kp.copy(), vp.copy())
    ka, va = OK.append(kp, vp, data.k_new, data.v_new, data.desc, bt, 16)
    assert (ka != before[0]).sum() <= spec.n_rows * 2 * 8
    assert (ka != 0xFFFF).sum() == sum(spec.kv_lens()) * 2 * 8      # nothing outside the requests' positions
    for s in range(3):
        qs, n, c = (int(x) for x in data.desc[s])
        k, v = OK.gather(ka, va, bt[s], c + n, 16)
        assert np.array_equal(k[:c], data.k_hist[s]) and np.array_equal(k[c:], data.k_new[qs:qs + n])
        assert np.array_equal(v[:c], data.v_hist[s]) and np.array_equal(v[c:], data.v_new[qs:qs + n])


# ---------------------------------------------------------------- mutation test
# Plausible mistakes planted in a copy of the oracle's append; the pins above, run
# against the copy, must reject each one.

MUTANTS = {
    "slot_off_by_one": ("slot = pos % page_size\n        H, D = k_new", "slot = (pos + 1) % page_size\n        H, D = k_new"),
    "positions_from_zero": ("pos = c + np.arange(n)", "pos = np.arange(n)"),
    "logical_page_as_physical": ("page = np.asarray(block_table)[s, pos // page_size]\n        slot = pos % page_size\n        H, D",
                                 "page = pos // page_size\n        slot = pos % page_size\n        H, D"),
    "key_features_strided": ("k_new[qs:qs + n].reshape(n, H, D // 8, 8)",
                             "k_new[qs:qs + n].reshape(n, H, 8, D // 8).transpose(0, 1, 3, 2)"),
    "rows_from_zero": ("kp[page, :, :, slot, :] = k_new[qs:qs + n]", "kp[page, :, :, slot, :] = k_new[0:n]"),
    "values_from_keys": ("vp[page, :, :, slot] = v_new[qs:qs + n]", "vp[page, :, :, slot] = k_new[qs:qs + n]"),
}


def mutant(name):
    import types
    src = open(OK.__file__).read()
    a, b = MUTANTS[name]
    assert src.count(a) == 1, name
    mod = types.ModuleType("kv_cache_mutant_" + name)
    exec(compile(src.replace(a, b), "<mutant>", "exec"), mod.__dict__)
    return mod


def pins_pass(mod) -> bool:
    """The scalar-loop pin (two key chunks per head, several requests per step) and
    the hand-worked addresses, run against a candidate oracle module."""
    try:
        for seed in range(3):
            spec = I.random_small_step(seed, max_seqs=4, max_n=20, max_c=40)
            spec.head_dim = 16
            data = I.make_step_data(spec, seed, with_history=False)
            bt, npages = I.make_block_table(spec, seed, permute=True, spare_pages=3)
            kp, vp = pools(npages, 2, 16, 16)
            a = mod.append(kp, vp, data.k_new, data.v_new, data.desc, bt, 16)
            b = scalar_append(kp, vp, data.k_new, data.v_new, data.desc, bt, 16)
            if not (np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])):
                return False
        kp, vp = pools(8, 1, 16, 16)
        k_new = np.arange(48, dtype=np.uint16).reshape(3, 1, 16)
        ka, va = mod.append(kp, vp, k_new, k_new + 100, np.array([[0, 3, 14]]), np.array([[7, 2]]), 16)
        if ka[2, 0, 1, 0].tolist() != list(range(40, 48)) or va[7, 0, :, 15].tolist() != list(range(116, 132)):
            return False
    except Exception:
        return False
    return True


def test_pins_accept_the_oracle():
    assert pins_pass(OK)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_planted_mistake(name):
    assert not pins_pass(mutant(name)), f"mutant {name} survived the pins"
