"""Run a multi-request serving trace through the attention path, layer by layer.

The step compositions come from the P-PAS generator (ppas_trace). Every layer
owns its own K/V page pools; all layers share one block table (request r's
pages are the same page ids in every layer's pools). Each step is planned once
(a step plan) and, in each layer, appends the step's new keys/values and runs
the step's attention with that plan; the kernels' own times are taken from the
HIP events their launches record.

Synthetic inputs: request r's query / key / value rows at position p of layer l
are rows base_q[r] + 97 l + p (base_kv[r] + 97 l + p) of seeded bf16 banks, so
the logical keys and values of any request at any step can be rebuilt on the
host for checking. Token content does not affect timing.
"""
from __future__ import annotations

import math
import time
from dataclasses import dataclass

import numpy as np

from . import inputs as I
from . import metrics as M
from . import ppas
from . import ppas_trace as PT
from .hip_events import HipEvents

LAYER_SHIFT = 97


@dataclass
class TraceSetup:
    steps: list
    requests: list
    req_index: dict            # req_id -> row of the block table
    block_table: np.ndarray    # [R, stride] int32
    num_pages: int
    base_q: np.ndarray         # [R] bank row of position 0 in layer 0
    base_kv: np.ndarray
    bank_rows: int


def make_setup(seed: int, n_bursts: int = 16, burst_size: int = 4, mean_gap: float = 160.0,
               mode: str = "ppas", mbt: int = 16384, prompt_range=(20000, 30000),
               output_range=(16, 64), layers: int = 36, b_max: int = PT.B_MAX, b_cap: int = PT.B_CAP) -> TraceSetup:
    reqs = PT.bursty_requests(seed, n_bursts, burst_size, mean_gap, prompt_range, output_range)
    steps = PT.run_trace(reqs, mode=mode, mbt=mbt, b_max=b_max, b_cap=b_cap)
    req_index = {r.req_id: i for i, r in enumerate(reqs)}
    # every request gets pages for its whole life (prompt + outputs) up front
    lens = np.array([r.prompt_len + r.output_len for r in reqs])
    pages = (lens + I.PAGE - 1) // I.PAGE
    total = int(pages.sum())
    perm = I.rng(seed, 7).permutation(total)
    stride = int(pages.max())
    bt = np.full((len(reqs), stride), -1, dtype=np.int32)
    at = 0
    for i, k in enumerate(pages):
        bt[i, :k] = perm[at:at + k]
        at += int(k)
    maxlen = int(lens.max()) + LAYER_SHIFT * layers + 1
    bank_rows = 1 << int(math.ceil(math.log2(2 * maxlen)))
    g = I.rng(seed, 21)
    base_q = g.integers(0, bank_rows - maxlen, size=len(reqs))
    base_kv = g.integers(0, bank_rows - maxlen, size=len(reqs))
    return TraceSetup(steps, reqs, req_index, bt, total, base_q, base_kv, bank_rows)


def make_banks(seed: int, bank_rows: int):
    """Host bf16 bit banks: Q [rows, 16, 128], K and V [rows, 2, 128]."""
    q = I.normal_bf16(I.rng(seed, 31), (bank_rows, I.HQ, I.HEAD_DIM))
    k = I.normal_bf16(I.rng(seed, 32), (bank_rows, I.HKV, I.HEAD_DIM))
    v = I.normal_bf16(I.rng(seed, 33), (bank_rows, I.HKV, I.HEAD_DIM))
    return q, k, v


def step_rows(setup: TraceSetup, step, layer: int):
    """Bank row indices of the step's query rows (for Q) and of its new K/V rows."""
    iq, ikv = [], []
    for s in step.spec.seqs:
        r = setup.req_index[s.req_id]
        pos = s.cached_len + np.arange(s.n_query)
        iq.append(setup.base_q[r] + LAYER_SHIFT * layer + pos)
        ikv.append(setup.base_kv[r] + LAYER_SHIFT * layer + pos)
    return np.concatenate(iq), np.concatenate(ikv)


def logical_kv_rows(setup: TraceSetup, req_id: int, layer: int, length: int):
    r = setup.req_index[req_id]
    return setup.base_kv[r] + LAYER_SHIFT * layer + np.arange(length)


def _upload(x: np.ndarray, device):
    """Host array -> device tensor without a host wait: the copy starts from a newly
    allocated pinned tensor, stream-ordered, so the loop can enqueue the next steps
    while the GPU runs (a copy from pageable memory would wait for the stream)."""
    import torch
    pinned = torch.empty(x.shape, dtype=torch.from_numpy(x[:0]).dtype, pin_memory=True)
    pinned.numpy()[...] = x
    return pinned.to(device, non_blocking=True)


def run(setup: TraceSetup, banks, layers: int, device="cuda", check=(), progress=None):
    """Run every step of the trace in every layer. `check` lists (step index, layer)
    pairs whose outputs are copied back to the host. Returns a dict of timings and
    the checked outputs.

    Each scheduler step is planned once (ppas_step_plan_create: validation, the
    attention work list and the page-write list) and the plan serves the step's
    page write and attention in every layer. The step's synthetic inputs for all
    layers are gathered from the banks in one pass before its layers run."""
    import torch
    from .step import to_device_bf16

    qb, kb, vb = (to_device_bf16(x, device) for x in banks)
    D, H, P = I.HEAD_DIM, I.HKV, I.PAGE
    shape = ppas.make_shape(I.HQ, I.HKV, setup.num_pages)
    pools = [(torch.zeros((setup.num_pages, H, D // 8, P, 8), dtype=torch.bfloat16, device=device),
              torch.zeros((setup.num_pages, H, D, P), dtype=torch.bfloat16, device=device)) for _ in range(layers)]
    ev = HipEvents()
    # every launch's timing events, created before the timed loop (creating them inside
    # it cost the host ~20 us per layer)
    n_launch = len(setup.steps) * layers
    ev_pool = [ev.create() for _ in range(4 * n_launch)]
    attn_events, app_events, gather_events = [], [], []
    checks = {}
    want = set(check)
    ws = torch.empty(256, dtype=torch.uint8, device=device)
    shift = (LAYER_SHIFT * torch.arange(layers, device=device, dtype=torch.int64))[:, None]
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    h0 = time.perf_counter()
    for si, st in enumerate(setup.steps):
        desc = st.spec.descriptors()
        rows = [setup.req_index[s.req_id] for s in st.spec.seqs]
        bt_host = np.ascontiguousarray(setup.block_table[rows])
        bt = _upload(bt_host, device)
        plan = ppas.StepPlan(shape, desc, bt_host)
        if ws.numel() < plan.workspace_bytes:
            ws = torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=device)
        T = st.spec.n_rows
        out = torch.empty((T, I.HQ, D), dtype=torch.bfloat16, device=device)
        iq0, ikv0 = step_rows(setup, st, 0)
        g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        g0.record()
        iq = (_upload(iq0, device)[None, :] + shift).reshape(-1)
        ikv = (_upload(ikv0, device)[None, :] + shift).reshape(-1)
        q_all = torch.index_select(qb, 0, iq).view(layers, T, I.HQ, D)
        k_all = torch.index_select(kb, 0, ikv).view(layers, T, H, D)
        v_all = torch.index_select(vb, 0, ikv).view(layers, T, H, D)
        g1.record()
        gather_events.append((g0, g1))
        for layer in range(layers):
            kp, vp = pools[layer]
            k = 4 * (si * layers + layer)
            a0, a1, e0, e1 = ev_pool[k:k + 4]
            plan.kv_append(kp, vp, k_all[layer], v_all[layer], bt, ppas.events(a0, a1))
            app_events.append((a0, a1))
            plan.attn_step(out, q_all[layer], kp, vp, bt, ws, ppas.events(e0, e1))
            attn_events.append((e0, e1))
            if (si, layer) in want:
                checks[(si, layer)] = out.float().cpu().numpy()
        plan.close()
        if progress and si % 100 == 0:
            progress(si, len(setup.steps))
    t1.record()
    host_ms = (time.perf_counter() - h0) * 1e3
    torch.cuda.synchronize()
    attn_ms = [ev.elapsed_ms(a, b) for a, b in attn_events]
    app_ms = [ev.elapsed_ms(a, b) for a, b in app_events]
    gather_ms = [a.elapsed_time(b) for a, b in gather_events]
    for a, b in attn_events + app_events:
        ev.destroy(a)
        ev.destroy(b)
    flops = sum(M.flops(s.spec) for s in setup.steps) * layers
    dec_bytes = sum(M.kv_bytes(s.spec, "decode") for s in setup.steps) * layers
    # per scheduler iteration: attention + page writes summed over the layers
    step_ms = (np.asarray(attn_ms) + np.asarray(app_ms)).reshape(len(setup.steps), layers).sum(axis=1)
    return {"attn_ms_total": float(np.sum(attn_ms)), "kv_append_ms_total": float(np.sum(app_ms)),
            "gather_ms_total": float(np.sum(gather_ms)), "step_ms": step_ms,
            "wall_ms": t0.elapsed_time(t1), "host_enqueue_ms": host_ms, "launches": len(attn_ms), "flops": flops,
            "decode_kv_bytes": dec_bytes, "attn_ms_max": float(np.max(attn_ms)), "checks": checks}


def oracle_inputs(setup: TraceSetup, banks, step_index: int, layer: int):
    """A StepData-like object with the logical inputs of one step in one layer."""
    qbank, kbank, vbank = banks
    st = setup.steps[step_index]
    iq, ikv = step_rows(setup, st, layer)
    kh, vh = [], []
    for s in st.spec.seqs:
        rows = logical_kv_rows(setup, s.req_id, layer, s.cached_len)
        kh.append(kbank[rows])
        vh.append(vbank[rows])
    return I.StepData(st.spec, st.spec.descriptors(), qbank[iq], kbank[ikv], vbank[ikv], kh, vh)
