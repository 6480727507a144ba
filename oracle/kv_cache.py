"""Where a step's new keys and values go in the paged KV cache.

TEST INFRASTRUCTURE (see the package docstring): never called by the product path.

Prefill and decode store each processed token's key and value in the KV cache
(Section 2); the cache is paged (Section 7, PagedAttention). The paper fixes no
page layout; the reading used throughout is:

  * page size P tokens; request s's logical page j (positions jP..jP+P-1) lives in
    physical page block_table[s, j];
  * the K pool is [num_pages, Hkv, D/8, P, 8]: within a page, one KV head's keys
    are split into D/8 chunks of 8 consecutive features, and each chunk holds
    the P tokens' 8 features contiguously (chunk-major);
  * the V pool is [num_pages, Hkv, D, P]: within a page, one KV head's values are
    stored feature-major, P consecutive tokens per feature.

A request with n new tokens after c cached ones writes positions c..c+n-1:
token i of the request (row qs+i of the step) goes to page
block_table[s, (c+i) // P], slot (c+i) % P. Nothing else in the pools changes.
"""
from __future__ import annotations

import numpy as np


def append(k_pool, v_pool, k_new, v_new, desc, block_table, page_size: int):
    """Return copies of the pools with every request's new rows written.

    k_pool: [num_pages, Hkv, D/8, P, 8]; v_pool: [num_pages, Hkv, D, P]; k_new, v_new: [T, Hkv, D];
    desc: [S, 3] of (query_start, n_query, cached_len); block_table: [S, stride].
    """
    kp = np.array(k_pool, copy=True)
    vp = np.array(v_pool, copy=True)
    for s in range(len(desc)):
        qs, n, c = (int(x) for x in desc[s])
        pos = c + np.arange(n)
        page = np.asarray(block_table)[s, pos // page_size]
        slot = pos % page_size
        H, D = k_new.shape[1], k_new.shape[2]
        kp[page, :, :, slot, :] = k_new[qs:qs + n].reshape(n, H, D // 8, 8)
        vp[page, :, :, slot] = v_new[qs:qs + n]
    return kp, vp


def gather(k_pool, v_pool, block_table_row, length: int, page_size: int):
    """Read a request's positions 0..length-1 back out of the pools as logical
    [length, Hkv, D] key and value arrays."""
    pos = np.arange(length)
    page = np.asarray(block_table_row)[pos // page_size]
    slot = pos % page_size
    kc = np.asarray(k_pool)[page, :, :, slot, :]              # [length, Hkv, D/8, 8]
    k = kc.reshape(length, kc.shape[1], -1)
    v = np.asarray(v_pool)[page, :, :, slot]
    return k, v


def fill_history(k_pool, v_pool, k_hist, v_hist, block_table, page_size: int):
    """Pools holding every request's cached positions 0..c-1 (k_hist[s], v_hist[s])."""
    kp = np.array(k_pool, copy=True)
    vp = np.array(v_pool, copy=True)
    for s in range(len(k_hist)):
        if k_hist[s] is None or len(k_hist[s]) == 0:
            continue
        pos = np.arange(len(k_hist[s]))
        page = np.asarray(block_table)[s, pos // page_size]
        slot = pos % page_size
        L, H, D = k_hist[s].shape
        kp[page, :, :, slot, :] = k_hist[s].reshape(L, H, D // 8, 8)
        vp[page, :, :, slot] = v_hist[s]
    return kp, vp
