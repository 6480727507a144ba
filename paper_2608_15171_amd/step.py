"""Device buffers for one mixed step and the two library calls that run it.

Owns torch tensors only (device memory and streams); the cache writes and the
attention itself are the library's kernels (ppas.kv_append, ppas.attn_step).
"""
from __future__ import annotations

import numpy as np
import torch

from . import ppas
from .inputs import StepData


def to_device_bf16(bits: np.ndarray, device="cuda") -> torch.Tensor:
    """uint16 bf16 patterns -> a bf16 device tensor with the same bits."""
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(device)


def bits_of(t: torch.Tensor) -> np.ndarray:
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


class DeviceStep:
    """Q, the step's new K/V, the page pools, the block table, output and workspace of a step."""

    def __init__(self, data: StepData, block_table: np.ndarray, num_pages: int, device="cuda",
                 pool_fill: int = 0, scale: float | None = None):
        spec = data.spec
        self.data = data
        self.desc = np.ascontiguousarray(data.desc, dtype=np.int32)
        self.bt_host = np.ascontiguousarray(block_table, dtype=np.int32)
        self.shape = ppas.make_shape(spec.n_q_heads, spec.n_kv_heads, num_pages, scale, spec.head_dim, spec.page_size)
        self.device = device
        self.q = to_device_bf16(data.q, device)
        self.k_new = to_device_bf16(data.k_new, device)
        self.v_new = to_device_bf16(data.v_new, device)
        self.bt = torch.from_numpy(self.bt_host).to(device)
        P, D, H = spec.page_size, spec.head_dim, spec.n_kv_heads
        fill = torch.tensor([pool_fill], dtype=torch.int32).to(torch.int16).item() if pool_fill else 0
        self.k_pages = torch.full((num_pages, H, D // 8, P, 8), fill, dtype=torch.int16, device=device).view(torch.bfloat16)
        self.v_pages = torch.full((num_pages, H, D, P), fill, dtype=torch.int16, device=device).view(torch.bfloat16)
        self.out = torch.zeros((spec.n_rows, spec.n_q_heads, D), dtype=torch.bfloat16, device=device)
        ws = max(ppas.attn_workspace_bytes(self.shape, self.desc), 256)
        self.workspace = torch.empty(ws, dtype=torch.uint8, device=device)

    def fill_history(self, stream=None) -> None:
        """Write every request's cached positions 0..c-1 through the library's kv_append."""
        hist = [(s, len(k)) for s, k in enumerate(self.data.k_hist) if k is not None and len(k)]
        if not hist:
            return
        kh = np.concatenate([self.data.k_hist[s] for s, _ in hist])
        vh = np.concatenate([self.data.v_hist[s] for s, _ in hist])
        desc = np.zeros((len(hist), 3), dtype=np.int32)
        at = 0
        for i, (_, c) in enumerate(hist):
            desc[i] = (at, c, 0)
            at += c
        rows = [s for s, _ in hist]
        bt_host = np.ascontiguousarray(self.bt_host[rows])
        bt = torch.from_numpy(bt_host).to(self.device)
        ppas.kv_append(self.shape, self.k_pages, self.v_pages, to_device_bf16(kh, self.device),
                       to_device_bf16(vh, self.device), desc, bt, bt_host, stream)
        torch.cuda.synchronize()

    def plan(self, opts=None, validate: bool = True) -> "ppas.StepPlan":
        """A step plan for these descriptors (validated against the host block table
        unless validate is False); the workspace grows to what the plan needs."""
        p = ppas.StepPlan(self.shape, self.desc, self.bt_host if validate else None, self.bt_host.shape[1], opts)
        if self.workspace.numel() < p.workspace_bytes:
            self.workspace = torch.empty(p.workspace_bytes, dtype=torch.uint8, device=self.device)
        return p

    def append(self, stream=None, validate: bool = True, plan=None, events=None) -> None:
        if plan is not None or events is not None:
            p = plan or self.plan(validate=validate)
            p.kv_append(self.k_pages, self.v_pages, self.k_new, self.v_new, self.bt, events, stream)
            return
        ppas.kv_append(self.shape, self.k_pages, self.v_pages, self.k_new, self.v_new, self.desc, self.bt,
                       self.bt_host if validate else None, stream)

    def rope_append(self, theta: float, stream=None, validate: bool = True) -> None:
        """Rotate Q in place and the new K into the pages (rotary embedding), copy the new V."""
        ppas.rope_kv_append(self.shape, theta, self.q, self.k_pages, self.v_pages, self.k_new, self.v_new,
                            self.desc, self.bt, self.bt_host if validate else None, stream)

    def attend(self, stream=None, validate: bool = True, plan=None, opts=None, events=None) -> None:
        """ppas_attn_step; with a plan, planning options or events, the planned call."""
        if plan is not None or opts is not None or events is not None:
            p = plan or self.plan(opts, validate)
            if self.workspace.numel() < p.workspace_bytes:
                self.workspace = torch.empty(p.workspace_bytes, dtype=torch.uint8, device=self.device)
            p.attn_step(self.out, self.q, self.k_pages, self.v_pages, self.bt, self.workspace, events, stream)
            return
        ppas.attn_step(self.shape, self.out, self.q, self.k_pages, self.v_pages, self.desc, self.bt,
                       self.workspace, self.bt_host if validate else None, stream)

    def run(self, stream=None, opts=None) -> None:
        self.append(stream)
        self.attend(stream, opts=opts)

    def out_f64(self) -> np.ndarray:
        return self.out.float().cpu().numpy().astype(np.float64)
