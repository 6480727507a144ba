"""GPU parity of the fused gate-up projection (ppas_gateup_proj) against the fp64
oracle (oracle/gemm.py), through the C ABI.

Bound per output element, derived from the kernel's arithmetic: the products of
two bf16 values are exact in fp32, the fp32 accumulation over H features moves
the sum s by at most H 2^-24 A (A = sum_k |x_k w_k|, from the oracle; doubled to
cover any internal order of the matrix cores), and rounding s to bf16 nearest
moves it by at most 2^-8 |s|:
    |gpu - y| <= 2^-8 |y| + (1 + 2^-8) 2 H 2^-24 A.
Ragged shapes (token rows and output columns not multiples of the 256 x 256 tile)
are compared on every element; the full Qwen2.5-3B sizes (hidden 2048, 22016
stacked gate/up rows) at 2,048 and 16,384 tokens on every element as well.
"""
import numpy as np
import pytest

import oracle.gemm as OG
from paper_2608_15171_amd import inputs as I

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lib():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2608_15171_amd import ppas, step
    return ppas, step, torch


def run(lib, xb, wb, split=True):
    """split: give the call the workspace it asks for (reductions split across workgroups
    when the output has fewer tiles than compute units); False: no workspace, no split."""
    ppas, step, torch = lib
    x = step.to_device_bf16(xb)
    w = step.to_device_bf16(wb)
    y = torch.full((xb.shape[0], wb.shape[0]), float("nan"), dtype=torch.bfloat16, device="cuda")
    n = ppas.gateup_workspace_bytes(xb.shape[0], xb.shape[1], wb.shape[0]) if split else 0
    ws = torch.full((max(n // 4, 1),), float("nan"), dtype=torch.float32, device="cuda") if n else None
    ppas.gateup_proj(x, w, y, ws)
    torch.cuda.synchronize()
    return y


def check(g, xb, wb, rows=None, label=""):
    """g: the GPU output of all rows, or of `rows` in that order."""
    y, a = OG.gate_up(xb, wb, rows=rows, with_abs=True)
    assert np.isfinite(g).all(), f"{label}: non-finite output"
    H = xb.shape[1]
    bound = 2.0 ** -8 * np.abs(y) + (1 + 2.0 ** -8) * 2 * H * 2.0 ** -24 * a + 1e-30
    err = np.abs(g - y)
    worst = float((err / bound).max())
    print(f"{label}: max_abs={err.max():.3e} err/bound={worst:.3f}", flush=True)
    assert worst <= 1.0, f"{label}: {int((err > bound).sum())} elements beyond the bound"


def f64(lib, y):
    return y.float().cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("T,H,N", [(1, 64, 1), (5, 64, 300), (31, 128, 33), (257, 128, 513), (300, 192, 520),
                                   (256, 256, 256), (513, 2048, 600), (700, 640, 1030),
                                   # split reductions: the decoder layer's other projections at decode and
                                   # chunk sizes (down 11008 -> 2048, QKV 2048 -> 2560, output 2048 -> 2048)
                                   (16, 11008, 2048), (3, 11008, 2050), (100, 2048, 2560), (2048, 11008, 2048),
                                   (600, 2048, 2048),
                                   # just over one round of workgroups' tiles, 64-row tail tiles among them
                                   (1125, 128, 15300)])
@pytest.mark.parametrize("split", [True, False])
def test_ragged_shapes_every_element(lib, T, H, N, split):
    ppas = lib[0]
    print(f"gate-up T={T} H={H} N={N} split={split} workspace={ppas.gateup_workspace_bytes(T, H, N)}", flush=True)
    xb = I.gateup_tokens(1, T, 0, hidden=H)
    wb = I.gateup_weight(1, hidden=H, inter=(N + 1) // 2)[:N]
    check(f64(lib, run(lib, xb, wb, split)), xb, wb, label=f"T{T} H{H} N{N} split={split}")


def test_split_reduction_is_deterministic(lib):
    ppas, step, torch = lib
    xb = I.gateup_tokens(2, 40, 0, hidden=11008)
    wb = I.gateup_weight(2, hidden=11008, inter=1024)
    a, b = run(lib, xb, wb), run(lib, xb, wb)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("T", [2048, 16384])
def test_qwen25_3b_sizes_every_row(lib, T):
    """Every element at the full sizes, checked in blocks of 2,048 token rows."""
    print(f"gate-up T={T} H={I.GATEUP_HIDDEN} N={2 * I.GATEUP_INTER}", flush=True)
    xb = I.gateup_tokens(0, T)
    wb = I.gateup_weight(0)
    y = run(lib, xb, wb)
    for r0 in range(0, T, 2048):
        rows = np.arange(r0, min(T, r0 + 2048))
        check(f64(lib, y[r0:rows[-1] + 1]), xb, wb, rows=rows, label=f"T{T} rows {r0}..{rows[-1]}")


def test_chunks_equal_whole_prompt_rows(lib):
    """Eight 2,048-token chunks projected one by one give the same bits as the rows of
    the 16,384-token prompt projected at once: each output element is the same
    sequence of MFMA k-steps wherever its row sits in a tile."""
    ppas, step, torch = lib
    wb = I.gateup_weight(0)
    whole = run(lib, I.gateup_tokens(0, 16384), wb)
    for c in range(8):
        part = run(lib, I.gateup_tokens(0, 2048, 2048 * c), wb)
        assert torch.equal(part.view(torch.int16), whole[2048 * c:2048 * (c + 1)].view(torch.int16)), c


def test_zero_tokens_is_a_no_op_and_bad_sizes_are_refused(lib):
    ppas, step, torch = lib
    x = torch.zeros((0, 64), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((8, 64), dtype=torch.bfloat16, device="cuda")
    y = torch.zeros((0, 8), dtype=torch.bfloat16, device="cuda")
    ppas.gateup_proj(x, w, y)
    x = torch.zeros((4, 96), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((8, 96), dtype=torch.bfloat16, device="cuda")
    y = torch.zeros((4, 8), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ppas.PPASError) as ex:
        ppas.gateup_proj(x, w, y)
    assert ex.value.status == ppas.PPAS_EUNSUPPORTED
