"""Pins for the CPU oracle, collected so planted-mistake tests can rerun them.

Each ``pin_*`` function takes an oracle namespace (the real ``moe_oracle`` or a
copy with one function replaced by a plausible mistake) and raises
AssertionError when the oracle disagrees with something fixed independently of
it: the pure-Python brute force, closed forms, special cases whose answer is
known without running the layer, or invariants.
"""
from __future__ import annotations

import math

import numpy as np

from oracle import bruteforce as bf

F32 = np.float32


def tiny_inputs(seed=0, T=6, H=8, I=12, E=5, k=2, n_local=None, bf16=False,
                alpha=0.7):
    """Small grid-quantised inputs (router on exact grids, weights bf16 if asked)."""
    g = np.random.default_rng(seed)
    x = (np.clip(np.rint(g.standard_normal((T, H)) * 64), -255, 255) / 64).astype(F32)
    q = 8
    wr = (np.clip(np.rint(g.standard_normal((E, H)) / math.sqrt(H) * 2 ** q), -255, 255)
          * 2.0 ** -q).astype(F32)
    rank = g.permutation(E) + 1
    bias = (-alpha * np.log(rank.astype(np.float64))).astype(F32)
    if n_local is None:
        local = np.arange(E)
    else:
        local = np.sort(g.choice(E, n_local, replace=False))
    emap = np.full(E, -1, np.int32)
    emap[local] = np.arange(len(local))
    L = len(local)
    wg = (g.standard_normal((L, I, H)) / math.sqrt(H)).astype(F32)
    wu = (g.standard_normal((L, I, H)) / math.sqrt(H)).astype(F32)
    wd = (g.standard_normal((L, H, I)) / math.sqrt(I)).astype(F32)
    if bf16:
        import torch
        wg, wu, wd = (torch.from_numpy(a).to(torch.bfloat16).float().numpy() for a in (wg, wu, wd))
    return dict(x=x, w_router=wr, bias=bias, k=k, expert_map=emap,
                w_gate=wg, w_up=wu, w_down=wd, rank=rank)


def _run(o, inp, bf16):
    return o.moe_layer(inp["x"], inp["w_router"], inp["bias"], inp["k"],
                       inp["expert_map"], inp["w_gate"], inp["w_up"], inp["w_down"],
                       bf16=bf16)


def _bf16_ulp(v):
    a = np.maximum(np.abs(np.asarray(v, np.float64)), 2.0 ** -126)
    return 2.0 ** (np.floor(np.log2(a)) - 7)


def pin_bruteforce(o, seeds=(0, 1, 2), bf16=False, shard=False):
    """Oracle == pure-Python brute force on tiny inputs.

    Integer outputs and logits must match exactly; weights to 1e-6 relative;
    fp32 outputs to 1e-5 relative of RMS; bf16 outputs within 2 bf16 ulps of the
    brute force value (fp64 accumulation can flip a rounding of h or y).
    """
    for seed in seeds:
        inp = tiny_inputs(seed=seed, bf16=bf16, n_local=3 if shard else None)
        r = _run(o, inp, bf16)
        b = bf.layer(inp["x"].tolist(), inp["w_router"].tolist(), inp["bias"].tolist(),
                     inp["k"], inp["expert_map"].tolist(), inp["w_gate"].tolist(),
                     inp["w_up"].tolist(), inp["w_down"].tolist(), bf16)
        assert np.array_equal(r["logits"], np.array(b["logits"], F32)), "logits"
        assert np.array_equal(r["ids"], np.array(b["ids"])), "ids"
        np.testing.assert_allclose(r["weights"], np.array(b["weights"]), rtol=1e-6, atol=0)
        assert np.array_equal(r["counts"], np.array(b["counts"])), "counts"
        assert np.array_equal(r["offsets"], np.array(b["offsets"])), "offsets"
        assert np.array_equal(r["perm_src"], np.array(b["perm_src"], np.int64)), "perm_src"
        assert np.array_equal(r["dest"], np.array(b["dest"])), "dest"
        out_b = np.array(b["out"], np.float64).reshape(r["out"].shape)
        y_b = np.array(b["y_perm"], np.float64).reshape(r["y_perm"].shape)
        if bf16:
            assert np.all(np.abs(r["y_perm"] - y_b) <= 2 * _bf16_ulp(y_b) + 1e-30), "y_perm"
            assert np.all(np.abs(r["out"] - out_b) <= 2 * _bf16_ulp(out_b) + 1e-30), "out"
        else:
            rms = float(np.sqrt(np.mean(out_b ** 2))) or 1.0
            assert np.max(np.abs(r["y_perm"] - y_b)) <= 1e-5 * rms, "y_perm"
            assert np.max(np.abs(r["out"] - out_b)) <= 1e-5 * rms, "out"


def pin_tie_break(o):
    """W_r = 0 and b = 0: every logit ties, so ids must be 0..k-1 in order."""
    T, H, E, k = 7, 8, 6, 3
    x = np.ones((T, H), F32)
    z = o.router_logits(x, np.zeros((E, H), F32), np.zeros(E, F32))
    ids = o.topk_select(z, k)
    assert np.array_equal(ids, np.tile(np.arange(k), (T, 1))), "tie-break"
    w = o.topk_weights(z, ids)
    assert np.all(w == F32(1.0 / 3.0)) or np.allclose(w, 1.0 / 3.0, rtol=1e-7), "equal weights"


def pin_extreme_skew(o):
    """A huge rank bias dominates: ids = experts of rank 1..k, in rank order."""
    inp = tiny_inputs(seed=3, alpha=50.0, T=9, E=7, k=3)
    z = o.router_logits(inp["x"], inp["w_router"], inp["bias"])
    ids = o.topk_select(z, 3)
    by_rank = np.argsort(inp["rank"])[:3]
    assert np.array_equal(ids, np.tile(by_rank, (9, 1))), "extreme skew"


def pin_full_k(o):
    """k = E: ids is a permutation of all experts sorted by logit."""
    inp = tiny_inputs(seed=4, E=6, k=6)
    z = o.router_logits(inp["x"], inp["w_router"], inp["bias"])
    ids = o.topk_select(z, 6)
    for t in range(z.shape[0]):
        assert sorted(ids[t].tolist()) == list(range(6)), "k=E permutation"
        zs = z[t, ids[t]]
        assert np.all(zs[:-1] >= zs[1:]), "k=E order"


def pin_weights(o):
    """Closed-form softmax over the selected logits; sums to 1; k=1 gives 1.0."""
    g = np.random.default_rng(5)
    z = (g.standard_normal((50, 9)) * 3).astype(F32)
    for k in (1, 2, 4, 9):
        ids = o.topk_select(z, k)
        w = o.topk_weights(z, ids)
        zz = np.take_along_axis(z.astype(np.float64), ids.astype(np.int64), 1)
        full = np.exp(z.astype(np.float64) - z.max(1, keepdims=True))
        ref = np.take_along_axis(full, ids.astype(np.int64), 1)
        ref = ref / ref.sum(1, keepdims=True)   # softmax over E, then renormalise
        np.testing.assert_allclose(w, ref, rtol=1e-6, atol=0)
        assert np.all(np.abs(w.astype(np.float64).sum(1) - 1.0) <= k * 2.0 ** -23), "sum"
        assert np.all(zz[:, :1] >= zz), "first id holds the max"
        if k == 1:
            assert np.all(w == 1.0), "k=1 weight"


def pin_profile_and_permutation(o, shard=True):
    """Histogram, offsets and permutation invariants on a sharded layer."""
    inp = tiny_inputs(seed=6, T=40, E=9, k=3, n_local=4 if shard else None)
    r = _run(o, inp, False)
    T, k = 40, 3
    ids = r["ids"]
    assert int(r["counts"].sum()) == T * k, "sum counts"
    for e in range(9):
        assert r["counts"][e] == int((ids == e).sum()), "count per expert"
    emap = inp["expert_map"]
    local = [int(np.where(emap == s)[0][0]) for s in range(int((emap >= 0).sum()))]
    off = np.concatenate([[0], np.cumsum([r["counts"][e] for e in local])])
    assert np.array_equal(r["offsets"], off), "offsets"
    ps, dest = r["perm_src"].astype(np.int64), r["dest"].astype(np.int64)
    flat = ids.ravel()
    loc_assign = [i for i in range(T * k) if emap[flat[i]] >= 0]
    assert sorted(ps.tolist()) == loc_assign, "perm_src bijection"
    for s in range(len(local)):
        seg = ps[off[s]:off[s + 1]]
        assert np.all(np.diff(seg) > 0), "stable order within a segment"
        assert np.all(flat[seg] == local[s]), "segment holds its expert"
    assert np.array_equal(dest[ps], np.arange(len(ps))), "dest o perm_src = id"
    remote = [i for i in range(T * k) if emap[flat[i]] < 0]
    assert np.all(dest[remote] == -1), "remote dest"
    assert np.array_equal(r["x_perm"], inp["x"][ps // k]), "x_perm rows"


def dense_swiglu_f64(x, wg, wu, wd, bf16):
    """Dense SwiGLU MLP through torch (fp64), rounding with torch's bf16 cast."""
    import torch
    import torch.nn.functional as F
    X = torch.from_numpy(np.asarray(x, np.float64))
    G = F.linear(X, torch.from_numpy(np.asarray(wg, np.float64)))
    U = F.linear(X, torch.from_numpy(np.asarray(wu, np.float64)))
    h = F.silu(G) * U
    if bf16:
        h = h.float().to(torch.bfloat16).double()
    y = F.linear(h, torch.from_numpy(np.asarray(wd, np.float64)))
    if bf16:
        y = y.float().to(torch.bfloat16).double()
    return y.numpy()


def pin_single_expert_dense(o, bf16=False):
    """E = 1, k = 1: the layer is a dense SwiGLU MLP on every token."""
    inp = tiny_inputs(seed=7, T=16, E=1, k=1, bf16=bf16)
    r = _run(o, inp, bf16)
    ref = dense_swiglu_f64(inp["x"], inp["w_gate"][0], inp["w_up"][0], inp["w_down"][0], bf16)
    if bf16:
        assert np.all(np.abs(r["out"] - ref) <= 2 * _bf16_ulp(ref) + 1e-30), "dense bf16"
    else:
        rms = float(np.sqrt(np.mean(ref ** 2)))
        assert np.max(np.abs(r["out"] - ref)) <= 1e-5 * rms, "dense fp32"


def pin_identical_experts(o):
    """All experts equal: routing cannot matter, out = dense SwiGLU(x)."""
    inp = tiny_inputs(seed=8, T=20, E=6, k=3)
    for name in ("w_gate", "w_up", "w_down"):
        inp[name] = np.repeat(inp[name][:1], 6, axis=0)
    r = _run(o, inp, False)
    ref = dense_swiglu_f64(inp["x"], inp["w_gate"][0], inp["w_up"][0], inp["w_down"][0], False)
    rms = float(np.sqrt(np.mean(ref ** 2)))
    assert np.max(np.abs(r["out"] - ref)) <= 1e-5 * rms, "identical experts"


def pin_k1_gather(o):
    """k = 1: w = 1 exactly, so out is y_perm gathered back, bit for bit."""
    inp = tiny_inputs(seed=9, T=30, E=4, k=1, bf16=True)
    r = _run(o, inp, True)
    dest = r["dest"]
    assert np.all(dest >= 0)
    assert np.array_equal(r["out"], r["y_perm"][dest]), "k=1 gather"


def pin_idle_expert_not_read(o):
    """Experts with no tokens are never read: NaN weights there change nothing."""
    inp = tiny_inputs(seed=10, T=12, E=6, k=2, alpha=50.0)
    r0 = _run(o, inp, False)
    idle = [s for s in range(6) if r0["counts"][s] == 0]
    assert idle, "setup: need an idle expert"
    for s in idle:
        for name in ("w_gate", "w_up", "w_down"):
            inp[name][s] = np.nan
    r1 = _run(o, inp, False)
    assert np.array_equal(r0["out"], r1["out"]), "idle expert read"


def pin_empty_rows(o):
    """Tokens whose experts are all remote get an exactly zero output row."""
    inp = tiny_inputs(seed=11, T=25, E=8, k=1, n_local=2)
    r = _run(o, inp, False)
    no_local = np.all(r["dest"].reshape(25, 1) < 0, axis=1)
    assert no_local.any(), "setup"
    assert np.all(r["out"][no_local] == 0.0), "empty rows"
    assert np.all(np.any(r["out"][~no_local] != 0.0, axis=1)), "non-empty rows"


ALL_PINS = [
    ("bruteforce_fp32", lambda o: pin_bruteforce(o, bf16=False)),
    ("bruteforce_bf16", lambda o: pin_bruteforce(o, bf16=True, seeds=(0,))),
    ("bruteforce_shard", lambda o: pin_bruteforce(o, bf16=False, shard=True, seeds=(0, 1))),
    ("tie_break", pin_tie_break),
    ("extreme_skew", pin_extreme_skew),
    ("full_k", pin_full_k),
    ("weights", pin_weights),
    ("profile_and_permutation", pin_profile_and_permutation),
    ("single_expert_dense", pin_single_expert_dense),
    ("single_expert_dense_bf16", lambda o: pin_single_expert_dense(o, bf16=True)),
    ("identical_experts", pin_identical_experts),
    ("k1_gather", pin_k1_gather),
    ("idle_expert_not_read", pin_idle_expert_not_read),
    ("empty_rows", pin_empty_rows),
]
