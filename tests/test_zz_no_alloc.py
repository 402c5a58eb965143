"""moe_grouped_swiglu_ffn_noalloc: the FFN entry point that allocates nothing.

It runs the kernels of moe_grouped_swiglu_ffn on the library's per-GPU
scratch. Checked through the C ABI against moe_grouped_swiglu_ffn on the same
inputs (and the oracle), on two calls in a row, the second with a smaller
input, for bf16 and fp32; a call whose fixed workspace exceeds the scratch is
refused before any launch.
"""
import dataclasses

import numpy as np
import pytest
import torch

import paper_2606_00735_amd as moe
from oracle import moe_oracle as O
from synth import CONFIGS
from synth.moe_inputs import make_experts, make_router
import gpu_helpers as G

pytestmark = pytest.mark.gpu

CASES = [
    # (workload, rows per local expert for call 1, for call 2 (smaller))
    ("mixtral", [9, 14, 3, 0, 11, 8, 12, 7], [5, 0, 2, 1, 0, 3, 0, 1]),     # decode schedule in both
    ("qwen3", [40] * 24 + [0] * 8, [3] * 4 + [0] * 28),                      # rounds (split), then decode schedule
    ("tiny", [17, 0, 30, 5, 9, 2, 1, 64], [4, 0, 1, 0, 0, 2, 0, 3]),          # fp32
]


def _run(name, rows, seed):
    sh = CONFIGS[name]
    E_local = len(rows)
    sh = dataclasses.replace(sh, E=max(sh.E, E_local), E_local=E_local)
    dt = torch.bfloat16 if sh.dtype == "bf16" else torch.float32
    wg, wu, wd = make_experts(sh, list(range(E_local)), seed=seed)
    m = sum(rows)
    x, *_ = make_router(sh, m, 0.0, seed=seed)
    M_cap = m + 3
    xp = np.zeros((M_cap, sh.H), np.float32)
    xp[:m] = x
    offsets = np.concatenate([[0], np.cumsum(rows)]).astype(np.int32)
    dxp, doff = G.up(xp, dt), G.up_i32(offsets)
    dw = [G.up(w, dt) for w in (wg, wu, wd)]
    y_ref_gpu, _ = moe.moe_grouped_swiglu_ffn(dxp, *dw, doff)
    y = torch.full((M_cap, sh.H), float("nan"), dtype=dt, device="cuda")
    moe.moe_grouped_swiglu_ffn_noalloc(dxp, *dw, doff, y_perm=y)
    torch.cuda.synchronize()
    got, ref = G.down(y)[:m], G.down(y_ref_gpu)[:m]
    h_ref, y_oracle = O.grouped_swiglu_ffn(x, wg, wu, wd, offsets, bf16=dt == torch.bfloat16)
    if dt == torch.bfloat16:
        scale = G.down_scale(h_ref, wd, offsets)
        G.check_bf16(got, ref, f"{name} noalloc vs moe_grouped_swiglu_ffn", scale=scale)
        G.check_bf16(got, y_oracle, f"{name} noalloc vs oracle", scale=scale)
    else:
        G.check_f32(got, ref, f"{name} noalloc vs moe_grouped_swiglu_ffn")
        G.check_f32(got, y_oracle, f"{name} noalloc vs oracle")
    assert torch.all(torch.isnan(y[m:].float())), "rows past the last expert must be left alone"


@pytest.mark.parametrize("name,rows1,rows2", CASES, ids=[c[0] for c in CASES])
def test_noalloc_matches_ffn_two_calls(name, rows1, rows2):
    print("CASE noalloc", name, sum(rows1), sum(rows2), flush=True)
    _run(name, rows1, seed=11)
    _run(name, rows2, seed=12)


def test_noalloc_refuses_oversize():
    """h alone beyond the scratch: refused on the host, nothing launched."""
    print("CASE noalloc oversize", flush=True)
    sh = CONFIGS["mixtral"]
    L = moe.load_library()
    scratch = L.moe_ffn_scratch_bytes()
    M_cap = scratch // (sh.I * 2) + 1
    st = L.moe_grouped_swiglu_ffn_noalloc(None, None, None, None, None, 8, sh.H, sh.I, 0, 0, M_cap, 1, None, None)
    assert st == 3  # MOE_ERR_WORKSPACE
