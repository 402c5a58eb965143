"""The whole layer captured in a HIP graph and replayed (serving loops replay
one captured layer per step). Every launch of the path is a kernel (the FFN's
work counters are cleared by a kernel, not a memset) and nothing synchronises
with the host, so capture works; each replay must reproduce the eager result
bit for bit, with eager work and synchronisations between the replays.
"""
import numpy as np
import pytest
import torch

import paper_2606_00735_amd as moe
from synth import make_layer
import gpu_helpers as G

pytestmark = pytest.mark.gpu

CASES = [
    ("mixtral", 64, 1.0, True),       # E = 8 router (one pass), fused gather FFN
    ("qwen3", 256, 1.0, True),        # decode-sized router over K ranges
    ("dsv3_shard", 512, 0.0, False),  # 256-expert router over K ranges, permuted copy + FFN
]

KEYS = ("ids", "weights", "counts", "offsets", "perm_src", "dest", "out")


@pytest.mark.parametrize("name,T,alpha,fuse", CASES, ids=[f"{n}-T{t}-a{a}" for n, t, a, _ in CASES])
def test_layer_graph_replay(name, T, alpha, fuse):
    print("CASE graph", name, T, alpha, "fuse" if fuse else "copy", "seed 2", flush=True)
    li = make_layer(name, T, alpha, seed=2)
    d = G.upload_layer(li)
    k = li.shape.k
    args = (d["x"], d["w_router"], d["bias"], k, li.expert_map, d["w_gate"], d["w_up"], d["w_down"])
    bufs = {}
    moe.moe_layer(*args, bufs=bufs, fuse_gather=fuse)   # allocates every buffer, eager reference
    torch.cuda.synchronize()
    ref = {key: bufs[key].clone() for key in KEYS}
    m = int(ref["offsets"][-1].item())
    ref_y = bufs["y_perm"][:m].clone()

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        moe.moe_layer(*args, bufs=bufs, fuse_gather=fuse)
    for rep in range(3):
        # eager work between replays: poison the outputs the graph must rewrite
        bufs["out"].fill_(float("nan"))
        bufs["y_perm"].fill_(float("nan"))
        bufs["ids"].fill_(-7)
        bufs["dest"].fill_(-7)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for key in KEYS:
            assert torch.equal(bufs[key], ref[key]), (rep, key)
        assert torch.equal(bufs["y_perm"][:m], ref_y), (rep, "y_perm")
    print(f"  M_loc={m}: 3 replays bitwise equal to the eager layer", flush=True)
    assert np.isfinite(G.down(bufs["out"])).all()
