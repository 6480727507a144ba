"""Measured time of one scheduler iteration of a Qwen2.5-3B-shaped decoder stack.

The cost function of the serving simulator (serving_sim): for an iteration's
descriptors it runs one decoder layer's kernels on the GPU and returns their
summed kernel time (HIP events recorded by each launch) times the layer count.
A layer here is the work the paper's profiling names for a prefill chunk and its
neighbours in the block (Section 6.1): the projections of the attention input
(Q, K and V in one GEMM), the rotary embedding fused with the page write of the
new keys and values, the packed attention over the paged cache (with its split
merge), the output projection, the fused gate-up projection with the MLP's gated
SiLU activation in its epilogue (ppas_gateup_act), and the down projection of its
output. All four projections run on the library's MFMA GEMM (ppas_gateup_proj
computes any y = x w^T with a hidden size that is a multiple of 64, splitting the
reduction across workgroups when the output has few tiles, as the decode-sized
and 2k-sized projections do). Left out: the two RMS norms and the residual adds
(elementwise, a few per cent of a prefill iteration at their HBM roofline) and
the once-per-iteration embedding, LM head and sampling.

Every request gets pages for its whole life (prompt + outputs) at set-up, in one
seeded permutation of the pool; the pools and the input banks hold random bf16
values (timing does not depend on them). Weights rotate over two copies
(2 x 154 MB, more than the 256 MB Infinity Cache), as a layer's weights would be
evicted by the other layers' between two of its launches.
"""
from __future__ import annotations

import numpy as np

from . import inputs as I
from . import ppas
from .hip_events import HipEvents

QWEN25_3B = {"layers": 36, "hidden": 2048, "inter": 11008, "q_heads": 16, "kv_heads": 2, "head_dim": 128,
             "rope_theta": 1e6}


class DecoderLayerCost:
    def __init__(self, requests, max_tokens: int = 16384, seed: int = 0, cfg: dict = QWEN25_3B,
                 weight_copies: int = 2, device: str = "cuda"):
        import torch
        self.torch = torch
        self.cfg = cfg
        self.device = device
        H, Hq, Hkv, D = cfg["hidden"], cfg["q_heads"], cfg["kv_heads"], cfg["head_dim"]
        lens = np.array([r.prompt_len + r.output_len for r in requests])
        pages = (lens + I.PAGE - 1) // I.PAGE
        total = int(pages.sum())
        perm = I.rng(seed, 41).permutation(total)
        self.stride = int(pages.max())
        self.bt_full = np.full((len(requests), self.stride), -1, dtype=np.int32)
        at = 0
        for i, k in enumerate(pages):
            self.bt_full[i, :k] = perm[at:at + k]
            at += int(k)
        self.row_of = {r.req_id: i for i, r in enumerate(requests)}
        self.shape = ppas.make_shape(Hq, Hkv, total)
        g = torch.Generator(device=device)
        g.manual_seed(seed)

        def rand(*shape, scale=1.0):
            return (torch.randn(*shape, generator=g, device=device, dtype=torch.float32) * scale).to(torch.bfloat16)

        self.kp = rand(total, Hkv, D // 8, I.PAGE, 8)
        self.vp = rand(total, Hkv, D, I.PAGE)
        T = max_tokens
        self.q = rand(T, Hq, D)
        self.kn = rand(T, Hkv, D)
        self.vn = rand(T, Hkv, D)
        self.x = rand(T, H)
        self.attn_out = torch.empty((T, Hq, D), dtype=torch.bfloat16, device=device)
        qkv_rows = (Hq + 2 * Hkv) * D
        self.y = {"qkv": torch.empty((T, qkv_rows), dtype=torch.bfloat16, device=device),
                  "o": torch.empty((T, H), dtype=torch.bfloat16, device=device),
                  "gate_up": torch.empty((T, cfg["inter"]), dtype=torch.bfloat16, device=device),
                  "down": torch.empty((T, H), dtype=torch.bfloat16, device=device)}
        self.w = [{"qkv": rand(qkv_rows, H, scale=0.02), "o": rand(H, Hq * D, scale=0.02),
                   "gate_up": rand(2 * cfg["inter"], H, scale=0.02), "down": rand(H, cfg["inter"], scale=0.02)}
                  for _ in range(weight_copies)]
        self.ws = torch.empty(256, dtype=torch.uint8, device=device)      # attention split partials
        self.gws = torch.empty(256, dtype=torch.uint8, device=device)     # projection split partials
        self.max_tokens = T
        self.hip = HipEvents()
        self.ev = [self.hip.create() for _ in range(16)]
        self.calls = 0
        self.parts_ms = {k: 0.0 for k in ("attention", "rope_append", "qkv", "o", "gate_up", "down")}
        torch.cuda.synchronize()

    def layer_ms(self, spec) -> dict:
        """One layer's kernels for the iteration's descriptors; their times in ms."""
        torch = self.torch
        desc = spec.descriptors()
        T = spec.n_rows
        if T > self.max_tokens:
            raise ValueError(f"{T} tokens exceed the banks' {self.max_tokens} rows")
        rows = [self.row_of[s.req_id] for s in spec.seqs]
        bt_host = np.ascontiguousarray(self.bt_full[rows])
        bt = torch.from_numpy(bt_host).to(self.device)
        plan = ppas.StepPlan(self.shape, desc, None, self.stride)
        if self.ws.numel() < plan.workspace_bytes:
            self.ws = torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=self.device)
        w = self.w[self.calls % len(self.w)]
        self.calls += 1
        e = self.ev
        H, I2 = self.cfg["hidden"], self.cfg["inter"]
        need = max(ppas.gateup_workspace_bytes(T, H, self.y["qkv"].shape[1]),
                   ppas.gateup_workspace_bytes(T, self.cfg["q_heads"] * self.cfg["head_dim"], H),
                   ppas.gateup_act_workspace_bytes(T, H, I2), ppas.gateup_workspace_bytes(T, I2, H))
        if self.gws.numel() < need:
            self.gws = torch.empty(need, dtype=torch.uint8, device=self.device)
        gws = self.gws
        ppas.gateup_proj(self.x[:T], w["qkv"], self.y["qkv"][:T], gws, ppas.events(e[0], e[1]))
        plan.rope_kv_append(self.cfg["rope_theta"], self.q[:T], self.kp, self.vp, self.kn[:T], self.vn[:T], bt,
                            ppas.events(e[2], e[3]))
        merge = plan.info.n_merge > 0
        plan.attn_step(self.attn_out[:T], self.q[:T], self.kp, self.vp, bt, self.ws,
                       ppas.events(e[4], e[5], *((e[6], e[7]) if merge else (None, None))))
        ppas.gateup_proj(self.attn_out[:T].view(T, -1), w["o"], self.y["o"][:T], gws, ppas.events(e[8], e[9]))
        ppas.gateup_act(self.x[:T], w["gate_up"], self.y["gate_up"][:T], gws, ppas.events(e[10], e[11]))
        ppas.gateup_proj(self.y["gate_up"][:T], w["down"], self.y["down"][:T], gws, ppas.events(e[12], e[13]))
        torch.cuda.synchronize()
        plan.close()
        el = self.hip.elapsed_ms
        out = {"qkv": el(e[0], e[1]), "rope_append": el(e[2], e[3]),
               "attention": el(e[4], e[7] if merge else e[5]), "o": el(e[8], e[9]),
               "gate_up": el(e[10], e[11]), "down": el(e[12], e[13])}
        for k, v in out.items():
            self.parts_ms[k] += v
        return out

    def __call__(self, spec) -> float:
        """Seconds of one iteration over all layers."""
        return sum(self.layer_ms(spec).values()) * 1e-3 * self.cfg["layers"]

    def close(self):
        for x in self.ev:
            self.hip.destroy(x)
        self.ev = []
