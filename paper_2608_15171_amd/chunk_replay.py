"""Prefill of one prompt as several chunks or as a single chunk.

Section 6.1 (Figure 4a) compares the attention time of prefilling one
16,384-token prompt as eight 2k chunks with prefilling it as one 16k chunk:
every chunk attends to the whole prefix cached before it, so the chunks grow
slower as the prefix grows and their sum exceeds the single chunk's time. This
module replays that comparison on the attention path. The prompt's K/V enter the
paged cache chunk by chunk (ppas_kv_append); each chunk's rows then attend over
the prefix cached so far in one step of their own (ppas_attn_step). Both
schedules compute the same rows (chunking changes the schedule, not the
result), so their outputs agree up to rounding.

Inputs are seeded bf16 N(0,1) Q/K/V rows for positions 0..prompt-1 at the
Qwen2.5-3B attention shape (16 query heads, 2 KV heads, head_dim 128) and a
seeded permutation of the prompt's pages.
"""
from __future__ import annotations

import numpy as np

from . import inputs as I
from . import metrics as M
from . import ppas
from .hip_events import HipEvents

_STREAM = 41   # seed stream kind of this module's inputs (distinct from inputs.py's kinds)


def chunk_specs(prompt: int, chunk: int) -> list:
    """One step per chunk: chunk k holds positions k*chunk .. (k+1)*chunk-1 of request 0."""
    if prompt <= 0 or chunk <= 0 or prompt % chunk:
        raise ValueError(f"prompt {prompt} must be a positive multiple of chunk {chunk}")
    return [I.StepSpec(f"chunk{k}-of-{prompt // chunk}", [I.Seq(chunk, k * chunk, 0)])
            for k in range(prompt // chunk)]


def prompt_bits(seed: int, prompt: int):
    """Host bf16 bits of the prompt's Q [P, 16, 128], K and V [P, 2, 128]."""
    q = I.normal_bf16(I.rng(seed, _STREAM, 0), (prompt, I.HQ, I.HEAD_DIM))
    k = I.normal_bf16(I.rng(seed, _STREAM, 1), (prompt, I.HKV, I.HEAD_DIM))
    v = I.normal_bf16(I.rng(seed, _STREAM, 2), (prompt, I.HKV, I.HEAD_DIM))
    return q, k, v


def prompt_block_table(seed: int, prompt: int) -> np.ndarray:
    pages = (prompt + I.PAGE - 1) // I.PAGE
    return I.rng(seed, _STREAM, 3).permutation(pages).astype(np.int32).reshape(1, pages)


class Replay:
    """Device state for one prompt: its Q/K/V rows, one K/V page pool and the output."""

    def __init__(self, prompt: int, seed: int = 0, device: str = "cuda"):
        import torch

        from .step import to_device_bf16
        self.prompt, self.seed = prompt, seed
        self.q_bits, self.k_bits, self.v_bits = prompt_bits(seed, prompt)
        self.bt_host = prompt_block_table(seed, prompt)
        pages = self.bt_host.shape[1]
        self.shape = ppas.make_shape(I.HQ, I.HKV, pages)
        self.q, self.k, self.v = (to_device_bf16(x, device) for x in (self.q_bits, self.k_bits, self.v_bits))
        self.bt = torch.from_numpy(self.bt_host).to(device)
        D, H, P = I.HEAD_DIM, I.HKV, I.PAGE
        self.k_pages = torch.zeros((pages, H, D // 8, P, 8), dtype=torch.bfloat16, device=device)
        self.v_pages = torch.zeros((pages, H, D, P), dtype=torch.bfloat16, device=device)
        self.out = torch.empty((prompt, I.HQ, D), dtype=torch.bfloat16, device=device)
        self.ws = torch.empty(256, dtype=torch.uint8, device=device)
        self.events = HipEvents()

    def run(self, chunk: int) -> list:
        """Prefill the whole prompt in chunks of `chunk` tokens; returns each chunk's
        attention kernel time in ms (HIP events the packed launch records)."""
        import torch
        specs = chunk_specs(self.prompt, chunk)
        plans = [ppas.StepPlan(self.shape, s.descriptors(), self.bt_host) for s in specs]
        need = max(p.workspace_bytes for p in plans)
        if self.ws.numel() < need:
            self.ws = torch.empty(need, dtype=torch.uint8, device=self.q.device)
        evs = []
        for s, plan in zip(specs, plans):
            desc = s.descriptors()
            lo = int(desc[0, 2])
            hi = lo + int(desc[0, 1])
            plan.kv_append(self.k_pages, self.v_pages, self.k[lo:hi], self.v[lo:hi], self.bt)
            e0, e1 = self.events.create(), self.events.create()
            plan.attn_step(self.out[lo:hi], self.q[lo:hi], self.k_pages, self.v_pages, self.bt, self.ws,
                           ppas.events(e0, e1))
            evs.append((e0, e1))
        torch.cuda.synchronize()
        for plan in plans:
            plan.close()
        ms = [self.events.elapsed_ms(a, b) for a, b in evs]
        for a, b in evs:
            self.events.destroy(a)
            self.events.destroy(b)
        return ms

    def out_f64(self) -> np.ndarray:
        return self.out.float().cpu().numpy().astype(np.float64)

    def oracle_inputs(self):
        """The prompt as one step for the oracle: (q_bits, desc, [K], [V])."""
        desc = np.array([[0, self.prompt, 0]], dtype=np.int32)
        return self.q_bits, desc, [self.k_bits], [self.v_bits]


def flops(prompt: int) -> float:
    """Algorithmic attention FLOP of the whole prompt (the same for every chunking)."""
    return M.flops(I.StepSpec("prompt", [I.Seq(prompt, 0, 0)]))
