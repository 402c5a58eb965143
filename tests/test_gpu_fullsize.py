"""GPU parity at the workloads' full sizes, in the bench's launch configuration.

At full size the oracle still computes the whole routing (logits, ids,
weights, counts, offsets, permutation) for every token, so those are checked
exactly everywhere; x_perm is checked by its defining property on the GPU;
layer outputs are checked on sampled tokens, which the oracle computes one
by one (``moe_layer_rows``), including tokens with no local expert.
"""
import numpy as np
import pytest
import torch

import paper_2606_00735_amd as moe
from oracle import moe_oracle as O
from synth import make_layer
import gpu_helpers as G

pytestmark = pytest.mark.gpu

FULL = [
    ("mixtral", 32, 0.0),
    ("mixtral", 4096, 1.0),
    ("qwen3", 128, 0.0),
    ("qwen3", 8192, 1.0),
    ("dsv3_shard", 16384, 0.0),
    ("dsv3_shard", 16384, 1.5),
    ("maverick_shard", 32768, 1.0),
]


@pytest.mark.parametrize("name,T,alpha", FULL, ids=[f"{n}-T{t}-a{a}" for n, t, a in FULL])
def test_fullsize(name, T, alpha):
    print("CASE fullsize", name, T, alpha, "seed 0", flush=True)
    li = make_layer(name, T, alpha, seed=0)
    k, E = li.shape.k, li.shape.E
    bf16 = li.shape.dtype == "bf16"
    d = G.upload_layer(li)
    bufs = G.poison_bufs(T, k, li.shape.H, E, len(li.local), d["dtype"])
    g = moe.moe_layer(d["x"], d["w_router"], d["bias"], k, li.expert_map, d["w_gate"], d["w_up"], d["w_down"],
                      logits=True, bufs=bufs)
    torch.cuda.synchronize()

    z = O.router_logits(li.x, li.w_router, li.bias)
    assert np.array_equal(G.down(g["logits"]), z), "logits"
    ids = O.topk_select(z, k)
    assert np.array_equal(G.down(g["ids"]), ids), "ids"
    np.testing.assert_allclose(G.down(g["weights"]), O.topk_weights(z, ids), rtol=1e-6, atol=0)
    counts = O.expert_histogram(ids, E)
    assert np.array_equal(G.down(g["counts"]), counts), "counts"
    offsets = O.local_offsets(counts, li.expert_map)
    assert np.array_equal(G.down(g["offsets"]), offsets), "offsets"
    _, perm_src, dest = O.permute(li.x, ids, li.expert_map, offsets)
    m = int(offsets[-1])
    assert np.array_equal(G.down(g["perm_src"])[:m], perm_src), "perm_src"
    assert np.array_equal(G.down(g["dest"]), dest), "dest"
    src_tok = g["perm_src"][:m].long() // k
    assert torch.equal(g["x_perm"][:m], d["x"][src_tok]), "x_perm rows"
    print(f"  M_loc={m} active={int((counts[li.local] > 0).sum())}/{len(li.local)} "
          f"max_Me={int(counts[li.local].max())}", flush=True)

    rng = np.random.default_rng(0)
    rows = rng.choice(T, size=min(T, 48), replace=False)
    no_local = np.where(np.all(dest.reshape(T, k) < 0, axis=1))[0]
    rows = np.unique(np.concatenate([rows, no_local[:4]]))
    ref = O.moe_layer_rows(li.x, li.w_router, li.bias, k, li.expert_map, li.w_gate, li.w_up, li.w_down,
                           bf16=bf16, rows=rows)
    got = G.down(g["out"])[rows]
    no_loc = np.all(dest.reshape(T, k)[rows] < 0, axis=1)
    assert np.all(got[no_loc] == 0.0), "rows without local experts must be zero"
    if bf16:
        G.check_bf16(got, ref["out"], f"{name} out rows", scale=ref["abs_terms"])
    else:
        G.check_f32(got, ref["out"], f"{name} out rows")
    assert np.all(np.isfinite(G.down(g["out"]))), "unwritten out rows"
    if bf16:
        # the bench's configuration: the FFN reading the routed rows of x
        # itself, over weights with padded rows, gives the same bits
        pw = [moe.pad_weight_rows(d[n]) for n in ("w_gate", "w_up", "w_down")]
        del d["w_gate"], d["w_up"], d["w_down"]
        fb = G.poison_bufs(T, k, li.shape.H, E, len(li.local), d["dtype"])
        fb.pop("x_perm")
        f = moe.moe_layer(d["x"], d["w_router"], d["bias"], k, li.expert_map, *pw, bufs=fb, fuse_gather=True)
        torch.cuda.synchronize()
        assert f["x_perm"] is None
        assert torch.equal(f["y_perm"][:m], g["y_perm"][:m]), "fused gather: y_perm"
        assert torch.equal(f["out"], g["out"]), "fused gather: out"
