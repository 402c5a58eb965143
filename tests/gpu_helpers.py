"""Helpers for the GPU parity tests: uploads, oracle runs and tolerances.

Tolerances (fixed before any GPU run):
* integers (ids, counts, offsets, perm_src, dest) and copied rows (x_perm):
  bit-exact;
* router logits: bit-exact (the inputs sit on grids where every fp32
  partial sum is exact, so summation order cannot matter);
* gate weights: 1e-6 relative (exp and division differ by an ulp or two
  between libm and the GPU);
* fp32 layer outputs: max |gpu - oracle| <= 1e-4 * RMS(oracle);
* bf16 layer outputs: max |gpu - oracle| <= 1.5e-2 * RMS(oracle), except
  that at most 1e-4 of the elements may exceed it, each by no more than 4 bf16
  ulps of the magnitude of the terms that were summed into it (for the
  combine, sum_j |w_j y_j|; elsewhere the value itself). One bf16 ulp of a
  value above 2-4x RMS is already larger than 1.5e-2 * RMS, and where two
  expert terms cancel a one-ulp flip of a term is many ulps of the sum, so
  two correct pipelines that only accumulate in a different order (the fp32
  and fp64 oracles, for one) produce such outliers; a real bug (wrong row,
  expert or weight) moves values by about RMS, not by ulps.
* rows of tokens with no local expert: exactly zero.
"""
from __future__ import annotations

import numpy as np
import torch

from oracle import moe_oracle as O

DEV = "cuda"


def up(a, dtype):
    """numpy float32 array (bf16-representable for bf16) -> device tensor."""
    t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to(DEV).to(dtype).contiguous()


def up_i32(a):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, np.int32))).to(DEV)


def down(t):
    return t.detach().float().cpu().numpy() if t.dtype in (torch.bfloat16, torch.float16) else t.detach().cpu().numpy()


def bf16_ulp(v):
    a = np.maximum(np.abs(np.asarray(v, np.float64)), 2.0 ** -126)
    return 2.0 ** (np.floor(np.log2(a)) - 7)


def check_bf16(got, ref, what, scale=None, max_frac=1e-4, max_ulps=4.0, rel=1.5e-2):
    """The bf16 rule above; `scale` is the summed-term magnitude (>= |ref|)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    scale = np.abs(ref) if scale is None else np.maximum(np.asarray(scale, np.float64), np.abs(ref))
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite values"
    rms = float(np.sqrt(np.mean(ref ** 2))) if ref.size else 0.0
    d = np.abs(got - ref)
    tol = rel * rms
    viol = d > tol
    n = int(viol.sum())
    stat = float(d.max() / rms) if ref.size and rms > 0 else 0.0
    msg = f"{what}: max|d|/RMS={stat:.3e} violations={n}/{d.size}"
    assert n <= max_frac * d.size, msg
    if n:
        assert np.all(d[viol] <= max_ulps * bf16_ulp(scale[viol])), msg + " (beyond 4 ulps)"
    return stat, n


def check_f32(got, ref, what, rel=1e-4):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    rms = float(np.sqrt(np.mean(ref ** 2))) if ref.size else 0.0
    d = float(np.abs(got - ref).max()) if ref.size else 0.0
    assert d <= rel * max(rms, 1e-30), f"{what}: max|d|={d:.3e} RMS={rms:.3e}"
    return d / rms if rms else 0.0


def oracle_layer(li, acc="f32"):
    bf16 = li.shape.dtype == "bf16"
    return O.moe_layer(li.x, li.w_router, li.bias, li.shape.k, li.expert_map, li.w_gate, li.w_up,
                       li.w_down, bf16=bf16, acc=acc)


def upload_layer(li):
    dt = torch.bfloat16 if li.shape.dtype == "bf16" else torch.float32
    return dict(x=up(li.x, dt), w_router=up(li.w_router, dt), bias=up(li.bias, torch.float32),
                w_gate=up(li.w_gate, dt), w_up=up(li.w_up, dt), w_down=up(li.w_down, dt), dtype=dt)


def poison_bufs(T, k, H, E, E_local, dt):
    """Output buffers pre-filled with NaN / -7 so unwritten entries show up."""
    M_cap = T * k
    return dict(
        ids=torch.full((T, k), -7, dtype=torch.int32, device=DEV),
        weights=torch.full((T, k), float("nan"), dtype=torch.float32, device=DEV),
        counts=torch.full((E,), -7, dtype=torch.int32, device=DEV),
        offsets=torch.full((E_local + 1,), -7, dtype=torch.int32, device=DEV),
        x_perm=torch.full((M_cap, H), float("nan"), dtype=dt, device=DEV),
        perm_src=torch.full((M_cap,), -7, dtype=torch.int32, device=DEV),
        dest=torch.full((T * k,), -7, dtype=torch.int32, device=DEV),
        y_perm=torch.full((M_cap, H), float("nan"), dtype=dt, device=DEV),
        out=torch.full((T, H), float("nan"), dtype=dt, device=DEV),
    )


def combine_scale(weights, y_perm, dest, T, k):
    """sum_j |w[t,j]| |y_perm[dest[t,j]]| per output element (fp64)."""
    H = y_perm.shape[1]
    dest = np.asarray(dest).reshape(T, k)
    out = np.zeros((T, H))
    for j in range(k):
        m = dest[:, j] >= 0
        out[m] += np.abs(np.asarray(weights, np.float64)[m, j])[:, None] * np.abs(
            np.asarray(y_perm, np.float64)[dest[m, j]])
    return out


def down_scale(h, w_down, offsets):
    """|h| |W_down|^T per expert: magnitude of the terms summed into y."""
    offsets = np.asarray(offsets)
    out = np.zeros((int(offsets[-1]), w_down.shape[1]))
    for s in range(len(offsets) - 1):
        a, b = offsets[s], offsets[s + 1]
        if b > a:
            out[a:b] = np.abs(np.asarray(h[a:b], np.float64)) @ np.abs(np.asarray(w_down[s], np.float64)).T
    return out


def compare_layer(li, g, r, what, check_h=True):
    """Every stage of a GPU layer run (dict g of tensors) against the oracle r."""
    import paper_2606_00735_amd as moe
    T, k, E = li.T, li.shape.k, li.shape.E
    bf16 = li.shape.dtype == "bf16"
    assert np.array_equal(down(g["logits"]), r["logits"]), f"{what}: logits not bit-exact"
    assert np.array_equal(down(g["ids"]), r["ids"]), f"{what}: ids"
    np.testing.assert_allclose(down(g["weights"]), r["weights"], rtol=1e-6, atol=0, err_msg=what)
    assert np.array_equal(down(g["counts"]), r["counts"]), f"{what}: counts"
    assert np.array_equal(down(g["offsets"]), r["offsets"]), f"{what}: offsets"
    m = int(r["offsets"][-1])
    assert np.array_equal(down(g["perm_src"])[:m], r["perm_src"]), f"{what}: perm_src"
    assert np.array_equal(down(g["dest"]), r["dest"]), f"{what}: dest"
    assert np.array_equal(down(g["x_perm"])[:m], r["x_perm"]), f"{what}: x_perm"
    stats = {}
    if check_h and m:
        I = li.shape.I
        h = down(moe.ffn_hidden(g["h"], T * k, I, g["x_perm"].dtype))[:m]
        stats["h"] = (check_bf16 if bf16 else check_f32)(h, r["h"], what + " h")
    got_out = down(g["out"])
    empty = np.all(np.asarray(r["dest"]).reshape(T, k) < 0, axis=1)
    assert np.all(got_out[empty] == 0.0), f"{what}: rows without local experts are not zero"
    if bf16:
        stats["y"] = check_bf16(down(g["y_perm"])[:m], r["y_perm"], what + " y_perm",
                                scale=down_scale(r["h"], li.w_down, r["offsets"]))
        stats["out"] = check_bf16(got_out, r["out"], what + " out",
                                  scale=combine_scale(r["weights"], r["y_perm"], r["dest"], T, k))
    else:
        stats["y"] = check_f32(down(g["y_perm"])[:m], r["y_perm"], what + " y_perm")
        stats["out"] = check_f32(got_out, r["out"], what + " out")
    return stats
