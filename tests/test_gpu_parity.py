"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Every case prints its name, shape and seed before touching the GPU. Sizes
are chosen so the oracle finishes in seconds while still spanning several
tiles and ragged per-expert tails; full-size cases (the bench's launch
configuration) are in test_gpu_fullsize.py.
"""
import dataclasses

import numpy as np
import pytest
import torch

import paper_2606_00735_amd as moe
from oracle import moe_oracle as O
from synth import CONFIGS, make_layer
from synth.moe_inputs import LayerInputs, expert_map_for, make_experts, make_router
import gpu_helpers as G

pytestmark = pytest.mark.gpu


def banner(*a):
    print("CASE", *a, flush=True)


def run_gpu(li, logits=True):
    d = G.upload_layer(li)
    bufs = G.poison_bufs(li.T, li.shape.k, li.shape.H, li.shape.E, len(li.local), d["dtype"])
    g = moe.moe_layer(d["x"], d["w_router"], d["bias"], li.shape.k, li.expert_map, d["w_gate"], d["w_up"],
                      d["w_down"], logits=logits, bufs=bufs)
    torch.cuda.synchronize()
    return g


REDUCED = [
    ("tiny", 64, 1.0),
    ("tiny", 37, 0.0),
    ("mixtral", 64, 0.0),
    ("mixtral", 96, 1.0),
    ("qwen3", 256, 0.0),
    ("qwen3", 200, 1.0),
    ("qwen3", 256, 1.5),
    ("dsv3_shard", 512, 0.0),
    ("dsv3_shard", 512, 1.0),
    ("dsv3_shard", 384, 1.5),
    ("maverick_shard", 1024, 0.0),
    ("maverick_shard", 1024, 1.0),
    ("maverick_shard", 1024, 1.5),
]


@pytest.mark.parametrize("name,T,alpha", REDUCED, ids=[f"{n}-T{t}-a{a}" for n, t, a in REDUCED])
def test_layer_parity(name, T, alpha):
    banner("layer", name, T, alpha, "seed 0")
    li = make_layer(name, T, alpha, seed=0)
    r = G.oracle_layer(li)
    g = run_gpu(li)
    stats = G.compare_layer(li, g, r, f"{name} T={T} a={alpha}")
    print("  stats", stats, "M_loc", int(r["offsets"][-1]), flush=True)


# The FFN's schedule (include/moe.h) depends on the host's bound on an
# expert's rows (M_cap; min(T, M_cap) for the gathering FFN) only through
# whether it is at most 128 (then no reduction launch follows), and otherwise
# on the rows and tiles, the same for both calls. Two calls give the same
# bits when they take the same schedule.
HOST_ROWS, PREF_ROWS = 128, 16


def _same_schedule(max_rows, bound_a, bound_b):
    return max_rows <= PREF_ROWS or ((bound_a <= HOST_ROWS) == (bound_b <= HOST_ROWS))


@pytest.mark.parametrize("name,T,alpha", [c for c in REDUCED if c[0] != "tiny"],
                         ids=[f"{n}-T{t}-a{a}" for n, t, a in REDUCED if n != "tiny"])
def test_layer_fused_gather(name, T, alpha):
    """moe_grouped_swiglu_ffn_gather in the layer: the oracle's tolerance, and
    the same bits as the layer that builds x_perm when both take the same
    schedule."""
    banner("layer fused gather", name, T, alpha, "seed 0")
    li = make_layer(name, T, alpha, seed=0)
    r = G.oracle_layer(li)
    g = run_gpu(li)
    d = G.upload_layer(li)
    bufs = G.poison_bufs(li.T, li.shape.k, li.shape.H, li.shape.E, len(li.local), d["dtype"])
    bufs.pop("x_perm")
    f = moe.moe_layer(d["x"], d["w_router"], d["bias"], li.shape.k, li.expert_map, d["w_gate"], d["w_up"],
                      d["w_down"], logits=True, bufs=bufs, fuse_gather=True)
    torch.cuda.synchronize()
    assert f["x_perm"] is None
    f["x_perm"] = g["x_perm"]  # not built; compare_layer checks the rest
    G.compare_layer(li, f, r, f"fused {name} T={T} a={alpha}")
    m = int(r["offsets"][-1])
    max_rows = int(np.diff(r["offsets"]).max()) if len(r["offsets"]) > 1 else 0
    M_cap = T * li.shape.k
    if _same_schedule(max_rows, min(T, M_cap), M_cap):
        assert torch.equal(f["y_perm"][:m], g["y_perm"][:m]) and torch.equal(f["out"], g["out"])
    else:
        print("  schedules differ (row bound min(T, M_cap) vs M_cap): each checked against the oracle", flush=True)


GATHER_CASES = [
    # (H, I, rows per local expert, T, k): perm_src a random injection of the
    # rows into the T*k flat assignments, so rows read scattered tokens
    (1024, 2048, [40] * 20, 800, 2),              # rounds: tail split gate/up, split-K down
    (1024, 2048, [1, 16, 0, 9], 64, 2),           # decode schedule in both
    (2048, 2048, [4608], 2400, 2),                # unsplit gate/up with a tail split
    (1024, 4096, [257, 300, 321, 576, 1], 400, 4),
]


@pytest.mark.parametrize("H,I,rows,T,k", GATHER_CASES, ids=["split", "decode", "tail", "ragged"])
def test_ffn_gather_matches_permuted_copy(H, I, rows, T, k):
    banner("stage ffn gather", H, I, rows, T, k, "seed 8")
    shape = dataclasses.replace(CONFIGS["qwen3"], name="gather", H=H, I=I, E=len(rows), k=k, E_local=len(rows))
    wg, wu, wd = make_experts(shape, list(range(len(rows))), seed=8)
    x, *_ = make_router(shape, T, 0.0, seed=8)
    m = sum(rows)
    M_cap = m + 5
    rng = np.random.default_rng(8)
    perm_src = np.full(M_cap, -1, np.int32)
    perm_src[:m] = rng.choice(T * k, size=m, replace=False)
    offsets = np.concatenate([[0], np.cumsum(rows)]).astype(np.int32)
    dx = G.up(x, torch.bfloat16)
    dps, doff = G.up_i32(perm_src), G.up_i32(offsets)
    dg, du, dd = (G.up(w, torch.bfloat16) for w in (wg, wu, wd))
    xp = torch.zeros((M_cap, H), dtype=torch.bfloat16, device="cuda")
    xp[:m] = dx[dps[:m].long() // k]
    y1, ws1 = moe.moe_grouped_swiglu_ffn(xp, dg, du, dd, doff)
    y2, ws2 = moe.moe_grouped_swiglu_ffn_gather(dx, dps, k, dg, du, dd, doff)
    torch.cuda.synchronize()
    assert _same_schedule(max(rows), min(T, M_cap), M_cap), "the case must keep one schedule"
    assert torch.equal(y2[:m], y1[:m])
    h1 = moe.ffn_hidden(ws1, M_cap, I, torch.bfloat16)[:m]
    h2 = moe.ffn_hidden(ws2, M_cap, I, torch.bfloat16)[:m]
    assert torch.equal(h1, h2)
    # and against the oracle on the gathered rows
    xr = x[perm_src[:m] // k]
    h_ref, y_ref = O.grouped_swiglu_ffn(xr, wg, wu, wd, offsets, bf16=True)
    G.check_bf16(G.down(h2), h_ref, "gather h")
    G.check_bf16(G.down(y2)[:m], y_ref, "gather y", scale=G.down_scale(h_ref, wd, offsets))


def test_layer_parity_seed1():
    banner("layer qwen3 T=128 a=1.0 seed 1")
    li = make_layer("qwen3", 128, 1.0, seed=1)
    G.compare_layer(li, run_gpu(li), G.oracle_layer(li), "qwen3 seed1")


def test_deterministic_bitwise():
    banner("determinism qwen3 T=512 a=1.0")
    li = make_layer("qwen3", 512, 1.0, seed=0)
    a = run_gpu(li)
    b = run_gpu(li)
    for key in ("logits", "ids", "weights", "counts", "offsets", "dest", "out"):
        assert torch.equal(a[key], b[key]), key
    m = int(a["offsets"][-1])
    for key in ("perm_src", "x_perm", "y_perm"):
        assert torch.equal(a[key][:m], b[key][:m]), key


def _custom(shape, T, alpha, seed=0, local=None, tie=False):
    x, w, b, rank = make_router(shape, T, alpha, seed)
    if tie:
        w = np.zeros_like(w)
        b = np.zeros_like(b)
    local = np.arange(shape.E) if local is None else np.sort(np.asarray(local))
    emap = expert_map_for(shape, local)
    wg, wu, wd = make_experts(shape, local, seed)
    return LayerInputs(shape, T, alpha, seed, x, w, b, rank, local, emap, wg, wu, wd)


def test_single_token():
    banner("edge T=1 qwen3")
    li = make_layer("qwen3", 1, 1.0, seed=2)
    G.compare_layer(li, run_gpu(li), G.oracle_layer(li), "T=1")


def test_top1_gather_exact():
    """k = 1: the weight is exactly 1, so out is y_perm gathered bit for bit."""
    banner("edge k=1 maverick-like small")
    shape = dataclasses.replace(CONFIGS["maverick_shard"], H=256, I=384, E=16, E_local=16)
    li = _custom(shape, 300, 1.0)
    r = G.oracle_layer(li)
    g = run_gpu(li)
    G.compare_layer(li, g, r, "k=1")
    assert torch.all(g["weights"] == 1.0)
    dest = g["dest"].long()
    assert torch.equal(g["out"], g["y_perm"][dest])


def test_k_equals_e():
    banner("edge k=E=8")
    shape = dataclasses.replace(CONFIGS["mixtral"], H=128, I=256, E=8, k=8, E_local=8)
    li = _custom(shape, 70, 0.5)
    G.compare_layer(li, run_gpu(li), G.oracle_layer(li), "k=E")


def test_all_tokens_on_one_expert():
    """A huge bias sends every token to the rank-1 expert: one expert with
    M = T rows (two full 128-row tiles and a ragged one), the rest idle."""
    banner("edge all tokens one expert")
    shape = dataclasses.replace(CONFIGS["qwen3"], H=256, I=384, E=16, k=1, E_local=16)
    li = _custom(shape, 300, 50.0)
    r = G.oracle_layer(li)
    assert r["counts"].max() == 300
    G.compare_layer(li, run_gpu(li), r, "one expert")


def test_ties_go_to_lower_ids():
    banner("edge all logits tie")
    shape = dataclasses.replace(CONFIGS["qwen3"], H=128, I=128, E=16, k=4, E_local=16)
    li = _custom(shape, 50, 0.0, tie=True)
    r = G.oracle_layer(li)
    assert np.all(r["ids"] == np.arange(4))
    G.compare_layer(li, run_gpu(li), r, "ties")


def test_shard_without_local_experts():
    banner("edge E_local=0")
    shape = dataclasses.replace(CONFIGS["dsv3_shard"], H=128, I=128, E=16, k=2, E_local=0)
    li = _custom(shape, 40, 1.0, local=[])
    r = G.oracle_layer(li)
    g = run_gpu(li)
    assert np.array_equal(G.down(g["counts"]), r["counts"])
    assert torch.all(g["dest"] == -1)
    assert torch.all(g["out"] == 0)
    assert G.down(g["offsets"]).tolist() == [0]


def test_mixed_small_and_large_experts():
    """Skewed loads: some experts take more than 128 rows, some fewer than 32,
    some none, with ragged tails everywhere, in one launch."""
    banner("edge mixed tiles")
    shape = dataclasses.replace(CONFIGS["qwen3"], H=384, I=256, E=24, k=3, E_local=24)
    li = _custom(shape, 400, 1.2, seed=5)
    r = G.oracle_layer(li)
    c = r["counts"]
    assert c.max() > 128 and ((c > 0) & (c <= 32)).any()
    G.compare_layer(li, run_gpu(li), r, "mixed")


ROUTER_WIDE = [
    # (H, E, k, T): which router runs follows the launcher's rule on 256 CUs
    (512, 256, 8, 4100),      # 8-wave router, 64-token blocks, E_pad 256, ragged last block
    (1024, 200, 16, 5000),    # 8-wave router, E = 200 of 256, k at its limit
    (256, 256, 8, 20000),     # 4-wave router, 128-token blocks, E_pad 256
    (256, 100, 6, 33000),     # 4-wave router, E_pad 128
    (256, 40, 4, 33000),      # 4-wave router, E = 40 of 64
    (2048, 128, 8, 9000),     # K-split router
    (1088, 8, 2, 40),         # K-split router: H/16 = 68 k-steps do not split evenly over 16 waves
    (4096, 8, 2, 1),          # small-batch router (16 waves, E_pad 32): one token
    (4096, 8, 2, 33),         # small-batch router, ragged second block
    (2048, 64, 4, 100),       # small-batch router, E_pad 64
    (2048, 96, 6, 65),        # small-batch router, E = 96 of 96
    (2048, 128, 8, 4096),     # small-batch router (8 waves, E_pad 128)
]


@pytest.mark.parametrize("H,E,k,T", ROUTER_WIDE, ids=[f"H{h}-E{e}-k{k}-T{t}" for h, e, k, t in ROUTER_WIDE])
def test_router_many_tokens(H, E, k, T):
    """Logits and ids bit-exact, weights to 1e-6, on the many-token router."""
    banner("router", H, E, k, T, "seed 3")
    shape = dataclasses.replace(CONFIGS["qwen3"], name="router", H=H, E=E, k=k, E_local=E)
    x, w, b, _ = make_router(shape, T, 1.0, seed=3)
    ids, wts, lg = moe.moe_gate_topk(G.up(x, torch.bfloat16), G.up(w, torch.bfloat16), G.up(b, torch.float32), k,
                                     logits=True)
    torch.cuda.synchronize()
    z = O.router_logits(x, w, b)
    assert np.array_equal(G.down(lg), z), "logits"
    rid = O.topk_select(z, k)
    assert np.array_equal(G.down(ids), rid), "ids"
    np.testing.assert_allclose(G.down(wts), O.topk_weights(z, rid), rtol=1e-6, atol=0)


ROUTER_SPLIT = [
    (7168, 256, 8, 3001),     # DSV3-shaped: 12 tiles x 8 K ranges, ragged last tile
    (5120, 128, 1, 1030),     # Maverick-shaped, top-1: 5 tiles x 8 ranges of 10 chunks
    (5120, 128, 1, 3000),     # Maverick-shaped: 12 tiles x 8 ranges, ragged last tile
    (256, 256, 8, 66000),     # 258 tiles: one K range
    (2048, 128, 8, 4096),     # Qwen3-shaped, the largest E = 128 batch it takes at H < 4096
    (5120, 128, 1, 6000),     # Maverick-shaped, ragged tile
    (5120, 128, 1, 12000),    # rows of 5120: batches whose 128-token blocks half-fill the CUs (ragged tile)
    (7168, 256, 8, 77),       # decode-sized DSV3-shaped batch
    # decode-sized batches over <= 128 experts: 32-token blocks x K ranges
    (4096, 8, 2, 32),         # Mixtral-shaped decode: 8 ranges of 32 k-steps
    (4096, 8, 2, 16),         # (16 + 8) rows of 8 KB: the smallest batch it takes at E = 8
    (2048, 128, 8, 1),        # Qwen3-shaped, one token: 8 ranges of 16 k-steps
    (2048, 128, 8, 200),      # Qwen3-shaped, ragged last block
    (5120, 128, 1, 100),      # Maverick-shaped: 5 ranges of 64 k-steps
    (2048, 96, 6, 256),       # E = 96 (padded to 128 columns)
    (1536, 40, 4, 33),        # E = 40 of 64 columns, 6 ranges of 16 k-steps
]


@pytest.mark.parametrize("H,E,k,T", ROUTER_SPLIT, ids=[f"H{h}-E{e}-k{k}-T{t}" for h, e, k, t in ROUTER_SPLIT])
def test_router_split_matches_one_pass(H, E, k, T):
    """The router with its workspace (logits summed over K ranges of
    256-token tiles) gives the one-pass router's logits, ids and weights bit
    for bit, and the oracle's."""
    banner("router split", H, E, k, T, "seed 6")
    shape = dataclasses.replace(CONFIGS["qwen3"], name="router", H=H, E=E, k=k, E_local=E)
    x, w, b, _ = make_router(shape, T, 1.0, seed=6)
    assert moe.gate_ws_bytes(T, H, E, torch.bfloat16) > 0
    dx, dw, db = G.up(x, torch.bfloat16), G.up(w, torch.bfloat16), G.up(b, torch.float32)
    i1, w1, l1 = moe.moe_gate_topk(dx, dw, db, k, logits=True)
    i2, w2, l2 = moe.moe_gate_topk(dx, dw, db, k, logits=True, use_ws=False)
    i3, w3, _ = moe.moe_gate_topk(dx, dw, None, k)   # no bias, no logits
    torch.cuda.synchronize()
    assert torch.equal(l1, l2) and torch.equal(i1, i2) and torch.equal(w1, w2)
    z = O.router_logits(x, w, b)
    assert np.array_equal(G.down(l1), z), "logits"
    rid = O.topk_select(z, k)
    assert np.array_equal(G.down(i1), rid), "ids"
    np.testing.assert_allclose(G.down(w1), O.topk_weights(z, rid), rtol=1e-6, atol=0)
    z0 = O.router_logits(x, w, np.zeros_like(b))
    assert np.array_equal(G.down(i3), O.topk_select(z0, k)), "ids without bias"


def test_router_many_tokens_ties():
    """All logits equal: every token takes experts 0..k-1 in order."""
    banner("router ties E=256 T=4096")
    shape = dataclasses.replace(CONFIGS["dsv3_shard"], name="router", H=256, E=256, k=8, E_local=256)
    x, w, b, _ = make_router(shape, 4096, 0.0, seed=1)
    ids, wts, _ = moe.moe_gate_topk(G.up(x, torch.bfloat16), torch.zeros((256, 256), dtype=torch.bfloat16,
                                    device="cuda"), torch.zeros(256, dtype=torch.float32, device="cuda"), 8)
    torch.cuda.synchronize()
    assert np.all(G.down(ids) == np.arange(8)) and np.allclose(G.down(wts), 1.0 / 8, rtol=1e-6)


def test_empty_batch():
    banner("edge T=0")
    d = G.upload_layer(make_layer("tiny", 1, 1.0))
    x = d["x"][:0]
    ids, w, _ = moe.moe_gate_topk(x, d["w_router"], d["bias"], 2)
    counts, offsets, ws = moe.moe_expert_histogram_scan(ids, 8, np.arange(8))
    torch.cuda.synchronize()
    assert torch.all(counts == 0) and torch.all(offsets == 0)


HIST_CASES = [
    # (T, E, k, local experts): count tables of n_blk = ceil(T / 256) rows x E
    (20000, 256, 8, 32),    # 20224 counts: the scan reads the table from L2
    (16384, 256, 8, 32),    # 16384 counts: the largest table the scan stages in LDS
    (32768, 128, 1, 16),    # 16384 counts, top-1
    (40000, 128, 2, 128),   # 20096 counts, every expert local
    (300, 64, 4, 64),       # two count blocks
    (1000, 8, 2, 8),        # four count blocks, few experts
]


@pytest.mark.parametrize("T,E,k,n_local", HIST_CASES, ids=[f"T{t}-E{e}-k{k}-L{l}" for t, e, k, l in HIST_CASES])
def test_histogram_and_positions(T, E, k, n_local):
    """Counts, offsets, perm_src and dest bit-exact against the oracle on
    skewed synthetic ids, on both sides of the scan's LDS staging limit."""
    banner("histogram/positions", T, E, k, n_local, "seed 9")
    rng = np.random.default_rng(9)
    score = rng.random((T, E)) - 0.7 * np.log(np.arange(1, E + 1))[None, :] * rng.random((T, 1))
    ids = np.argsort(-score, axis=1, kind="stable")[:, :k].astype(np.int32)
    emap = np.full(E, -1, np.int32)
    local = np.sort(rng.choice(E, n_local, replace=False))
    emap[local] = np.arange(n_local, dtype=np.int32)
    d_ids = G.up_i32(ids)
    counts, offsets, ws = moe.moe_expert_histogram_scan(d_ids, E, emap)
    x = torch.zeros((T, 64), dtype=torch.bfloat16, device="cuda")
    _, perm_src, dest = moe.moe_permute(x, d_ids, emap, ws, gather=False)
    torch.cuda.synchronize()
    c_ref = O.expert_histogram(ids, E)
    o_ref = O.local_offsets(c_ref, emap)
    _, p_ref, d_ref = O.permute(np.zeros((T, 1), np.float32), ids, emap, o_ref)
    assert np.array_equal(G.down(counts), c_ref), "counts"
    assert np.array_equal(G.down(offsets), o_ref), "offsets"
    m = int(o_ref[-1])
    assert np.array_equal(G.down(perm_src)[:m], p_ref), "perm_src"
    assert np.array_equal(G.down(dest), d_ref), "dest"


def test_ffn_stage_on_oracle_inputs():
    """The FFN alone, fed the oracle's x_perm and offsets."""
    banner("stage ffn dsv3-like")
    li = make_layer("dsv3_shard", 256, 0.0, seed=3)
    r = G.oracle_layer(li)
    m = int(r["offsets"][-1])
    M_cap = m + 5
    xp = np.zeros((M_cap, li.shape.H), np.float32)
    xp[:m] = r["x_perm"]
    d = G.upload_layer(li)
    y, ws = moe.moe_grouped_swiglu_ffn(G.up(xp, torch.bfloat16), d["w_gate"], d["w_up"], d["w_down"],
                                       G.up_i32(r["offsets"]))
    torch.cuda.synchronize()
    h = G.down(moe.ffn_hidden(ws, M_cap, li.shape.I, torch.bfloat16))[:m]
    G.check_bf16(h, r["h"], "stage h")
    G.check_bf16(G.down(y)[:m], r["y_perm"], "stage y")


SPLIT_CASES = [
    # (H, I, rows per local expert, S of the down GEMM's split-K plan).
    # Each GEMM launch takes the decode schedule (equal shares of (tile, K
    # chunk) units per CU, split tiles finished in the GEMM; the plan then
    # says 1) when no expert exceeds 16 rows, or 64 rows when no reduction
    # launch follows (M_cap <= 128), or 128 rows when it has no more 128-column
    # tiles than half its blocks (256 CUs here); other launches run tiles in
    # rounds, split along K (S from the split rule) when they have fewer
    # tiles than CUs and a reduction launch follows.
    (1024, 2048, [40] * 20, 3),            # 160 down tiles: split-K, S = 3 (32 chunks)
    (4096, 14336, [64], 1),                # one Mixtral-shaped expert of 64 rows, M_cap 67: 32 down tiles, decode
    (4096, 14336, [1], 1),                 # decode schedule
    (4096, 14336, [16, 7, 0, 11], 1),      # decode schedule at its preferred 16-row bound
    (4096, 14336, [32, 7, 0, 19], 1),      # 32 rows, M_cap 61: no reduction launch, decode schedule
    (4096, 14336, [40, 7, 0, 19, 30, 25], 1),  # M_cap 124: no reduction launch, decode schedule
    (4096, 14336, [40, 7, 0, 19, 30, 25, 10], 4),  # M_cap 134, 192 down tiles: split-K, S = 4 (224 chunks)
    (1024, 2048, [65, 3, 0, 1], 1),        # a 65-row expert, M_cap 72, 24 down tiles: decode schedule
    (4096, 14336, [128], 1),               # a 128-row expert, M_cap 131, 32 down tiles: decode schedule
    (7168, 2048, [256], 4),                # a 256-row DSV3-shaped expert: gate/up S = 8, down S = 4
    (5120, 8192, [400, 100, 32], 3),       # Maverick-shaped experts of mixed size: down S = 3
    (7168, 2048, [1, 33], 1),              # DSV3-shaped experts, M_cap 37: decode schedule
    (7168, 2048, [1, 33, 40, 60, 5], 1),   # M_cap 142, 280 down tiles: rounds, last one split along K (plan S = 1)
    (7168, 2048, [1], 1),                  # one DSV3-shaped expert: decode schedule
    (5120, 8192, [1], 1),                  # one Maverick-shaped expert: decode schedule
    (2048, 768, [5], 1),                   # one Qwen3-shaped expert: decode schedule
    (2048, 768, [128, 1, 60, 0, 127], 1),  # 64 down tiles: decode schedule
]


def _down_split_factor(ws, M_cap, I):
    """S of the last (down) GEMM, from the split-K plan that follows h in the
    workspace (white-box: shows which path a case exercised; 1 also for the
    decode schedule, whose split tiles are finished inside the GEMM)."""
    off = moe.FFN_COUNTER_BYTES + ((M_cap * I * 2 + 255) // 256) * 256
    return int(ws[off:off + 4].view(torch.int32).item())


def _counters_zero(ws):
    """The workspace's counters are left zero by every call."""
    return bool(torch.all(ws[:moe.FFN_COUNTER_BYTES] == 0).item())


@pytest.mark.parametrize("H,I,rows,S_down", SPLIT_CASES,
                         ids=[f"H{h}-I{i}-rows{'_'.join(map(str, r))}" for h, i, r, _ in SPLIT_CASES])
def test_ffn_split_k(H, I, rows, S_down):
    banner("stage ffn split-K", H, I, rows, "seed 5")
    shape = dataclasses.replace(CONFIGS["qwen3"], name="split", H=H, I=I, E=len(rows), k=1,
                                E_local=len(rows))
    wg, wu, wd = make_experts(shape, list(range(len(rows))), seed=5)
    m = sum(rows)
    x, *_ = make_router(shape, m, 0.0, seed=5)
    offsets = np.concatenate([[0], np.cumsum(rows)]).astype(np.int32)
    M_cap = m + 3
    xp = np.zeros((M_cap, H), np.float32)
    xp[:m] = x
    h_ref, y_ref = O.grouped_swiglu_ffn(x, wg, wu, wd, offsets, bf16=True)
    dg, du, dd = (G.up(w, torch.bfloat16) for w in (wg, wu, wd))
    dx, doff = G.up(xp, torch.bfloat16), G.up_i32(offsets)
    y, ws = moe.moe_grouped_swiglu_ffn(dx, dg, du, dd, doff)
    torch.cuda.synchronize()
    assert _down_split_factor(ws, M_cap, I) == S_down
    assert _counters_zero(ws)
    h = G.down(moe.ffn_hidden(ws, M_cap, I, torch.bfloat16))[:m]
    G.check_bf16(h, h_ref, "split h")
    G.check_bf16(G.down(y)[:m], y_ref, "split y", scale=G.down_scale(h_ref, wd, offsets))
    # the split partials are summed in a fixed order: a second call is bitwise equal
    y2, _ = moe.moe_grouped_swiglu_ffn(dx, dg, du, dd, doff, ws=ws)
    torch.cuda.synchronize()
    assert torch.equal(y2[:m], y[:m])
    assert _counters_zero(ws)


TAIL_CASES = [
    # (H, I, rows of one expert, (S, St, rem, cols) of the down GEMM) worked out
    # by hand from the tail rule on 256 CUs: an unsplit launch whose last round
    # holds rem <= 128 tiles cuts each into St = min(8, 256 // rem) K ranges,
    # fewer if a range would hold under 8 chunks or the partials would not fit
    (2048, 2048, [4608], (1, 4, 32, 128)),   # 288 tiles of 128 columns: 32 left over, K = 32 chunks
    (4096, 2048, [8448], (1, 4, 16, 256)),   # 528 tiles of 256 columns: 16 left over
]


@pytest.mark.parametrize("H,I,rows,plan", TAIL_CASES,
                         ids=[f"H{h}-I{i}-rows{r[0]}" for h, i, r, _ in TAIL_CASES])
def test_ffn_tail_split(H, I, rows, plan):
    """The last, partly filled round of an unsplit launch split along K over
    the idle CUs; the gate/up GEMM of these shapes takes the same path."""
    banner("stage ffn tail split", H, I, rows, "seed 6")
    shape = dataclasses.replace(CONFIGS["qwen3"], name="tail", H=H, I=I, E=1, k=1, E_local=1)
    wg, wu, wd = make_experts(shape, [0], seed=6)
    m = sum(rows)
    x, *_ = make_router(shape, m, 0.0, seed=6)
    offsets = np.array([0, m], np.int32)
    M_cap = m + 3
    xp = np.zeros((M_cap, H), np.float32)
    xp[:m] = x
    h_ref, y_ref = O.grouped_swiglu_ffn(x, wg, wu, wd, offsets, bf16=True)
    y, ws = moe.moe_grouped_swiglu_ffn(G.up(xp, torch.bfloat16), G.up(wg, torch.bfloat16),
                                       G.up(wu, torch.bfloat16), G.up(wd, torch.bfloat16), G.up_i32(offsets))
    torch.cuda.synchronize()
    off = moe.FFN_COUNTER_BYTES + ((M_cap * I * 2 + 255) // 256) * 256
    got = ws[off:off + 20].view(torch.int32).cpu().numpy()
    assert (got[0], got[2], got[3], got[4]) == plan, got[:5]
    h = G.down(moe.ffn_hidden(ws, M_cap, I, torch.bfloat16))[:m]
    G.check_bf16(h, h_ref, "tail h")
    G.check_bf16(G.down(y)[:m], y_ref, "tail y", scale=G.down_scale(h_ref, wd, offsets))
    # tiles taken from the work queues in whatever order: still bitwise equal
    y2, _ = moe.moe_grouped_swiglu_ffn(G.up(xp, torch.bfloat16), G.up(wg, torch.bfloat16),
                                       G.up(wu, torch.bfloat16), G.up(wd, torch.bfloat16), G.up_i32(offsets), ws=ws)
    torch.cuda.synchronize()
    assert torch.equal(y2[:m], y[:m])


RAGGED_CASES = [
    # (H, I, rows per local expert, (S, cols) of the down GEMM): experts of
    # 256 q + t rows end in a 64-, 128- or 256-row tile (t = 1, 44, 64, 65, 4).
    # Case 1: the gate/up GEMM runs 320 tiles unsplit and splits its last 64
    # (among them 64-row remainders and one-row experts) along K over the idle
    # CUs; the down GEMM runs split-K. Case 2: the down GEMM in 256-column
    # tiles over 29 ragged experts.
    (1024, 4096, [257, 300, 321, 576, 1], (3, 128)),
    (4096, 512, [300] * 28 + [64, 260, 576, 1], (1, 256)),
]


@pytest.mark.parametrize("H,I,rows,plan", RAGGED_CASES, ids=["tail-split", "wide-down"])
def test_ffn_ragged_tails(H, I, rows, plan):
    """Experts with short row remainders after full 256-row tiles."""
    banner("stage ffn ragged tails", H, I, len(rows), "experts seed 7")
    shape = dataclasses.replace(CONFIGS["qwen3"], name="ragged", H=H, I=I, E=len(rows), k=1, E_local=len(rows))
    wg, wu, wd = make_experts(shape, list(range(len(rows))), seed=7)
    m = sum(rows)
    x, *_ = make_router(shape, m, 0.0, seed=7)
    offsets = np.concatenate([[0], np.cumsum(rows)]).astype(np.int32)
    M_cap = m + 2
    xp = np.zeros((M_cap, H), np.float32)
    xp[:m] = x
    h_ref, y_ref = O.grouped_swiglu_ffn(x, wg, wu, wd, offsets, bf16=True)
    dg, du, dd = (G.up(w, torch.bfloat16) for w in (wg, wu, wd))
    dx, doff = G.up(xp, torch.bfloat16), G.up_i32(offsets)
    y, ws = moe.moe_grouped_swiglu_ffn(dx, dg, du, dd, doff)
    torch.cuda.synchronize()
    off = moe.FFN_COUNTER_BYTES + ((M_cap * I * 2 + 255) // 256) * 256
    got = ws[off:off + 20].view(torch.int32).cpu().numpy()
    assert (got[0], got[4]) == plan, got[:5]
    h = G.down(moe.ffn_hidden(ws, M_cap, I, torch.bfloat16))[:m]
    G.check_bf16(h, h_ref, "ragged h")
    G.check_bf16(G.down(y)[:m], y_ref, "ragged y", scale=G.down_scale(h_ref, wd, offsets))
    y2, _ = moe.moe_grouped_swiglu_ffn(dx, dg, du, dd, doff, ws=ws)
    torch.cuda.synchronize()
    assert torch.equal(y2[:m], y[:m])


def test_combine_stage_on_oracle_inputs():
    banner("stage combine qwen3")
    li = make_layer("qwen3", 64, 1.0, seed=4)
    r = G.oracle_layer(li)
    yp = G.up(r["y_perm"], torch.bfloat16)
    out = moe.moe_unpermute_combine(yp, G.up(r["weights"], torch.float32), G.up_i32(r["dest"]), li.T)
    torch.cuda.synchronize()
    G.check_bf16(G.down(out), r["out"], "stage out")


def test_load_sweep_output_and_timing():
    """The sweep's last run leaves y for the largest M; it must match the
    oracle's single-expert FFN, and every median must be positive."""
    banner("sweep qwen3 expert")
    shape = CONFIGS["qwen3"]
    wg, wu, wd = make_experts(shape, [5], seed=0)
    x, *_ = make_router(shape, 300, 0.0, seed=0)
    Ms = [1, 7, 33, 128, 300]
    rot = 3
    dg = G.up(np.repeat(wg, rot, 0), torch.bfloat16)
    du = G.up(np.repeat(wu, rot, 0), torch.bfloat16)
    dd = G.up(np.repeat(wd, rot, 0), torch.bfloat16)
    y = torch.full((300, shape.H), float("nan"), dtype=torch.bfloat16, device="cuda")
    us, allus = moe.moe_load_sweep(G.up(x, torch.bfloat16), dg, du, dd, Ms, warmup=2, iters=5, y_scratch=y,
                                   keep_all=True)
    print("  sweep us", us.tolist(), flush=True)
    assert np.all(us > 0) and allus.shape == (5, 5)
    _, yref = O.swiglu_rows(x, wg[0], wu[0], wd[0], bf16=True)
    G.check_bf16(G.down(y), yref, "sweep y")


def _padded(w, pad, dtype):
    """Device copy of weights [B, R, K] as the columns [:, :, :K] of a
    [B, R, K + pad] buffer whose padding holds NaN (read, it would poison
    the outputs)."""
    B, R, K = w.shape
    buf = torch.full((B, R, K + pad), float("nan"), dtype=dtype, device="cuda")
    buf[:, :, :K] = G.up(w, dtype)
    return buf[:, :, :K]


PAD_CASES = [
    # (H, I, rows per expert, pad of W_gate/W_up rows, pad of W_down rows, dtype)
    (1024, 2048, [40] * 20, 64, 8, "bf16"),                   # tail split gate/up, split-K down
    (1024, 1024, [257, 300, 321, 576, 1], 64, 64, "bf16"),    # every tile class, ragged tails
    (2048, 2048, [4608], 128, 8, "bf16"),                     # unsplit gate/up with a tail split
    (128, 256, [3, 40, 0, 77], 4, 12, "f32"),
]


@pytest.mark.parametrize("H,I,rows,pg,pd,dt", PAD_CASES, ids=["split", "ragged", "tail", "f32"])
def test_ffn_padded_weight_rows(H, I, rows, pg, pd, dt):
    """Weights whose rows are padded (row stride H + pg, I + pd) give the
    dense call's results bit for bit, through the permuted and the gathering
    FFN, and never read the padding."""
    banner("stage ffn padded rows", H, I, rows, pg, pd, dt, "seed 9")
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    k = 2
    shape = dataclasses.replace(CONFIGS["qwen3"], name="pad", H=H, I=I, E=len(rows), k=k, E_local=len(rows))
    wg, wu, wd = make_experts(shape, list(range(len(rows))), seed=9)
    m = sum(rows)
    T = m
    x, *_ = make_router(shape, T, 0.0, seed=9)
    M_cap = m + 3
    rng = np.random.default_rng(9)
    perm_src = np.full(M_cap, -1, np.int32)
    perm_src[:m] = rng.choice(T * k, size=m, replace=False)
    offsets = np.concatenate([[0], np.cumsum(rows)]).astype(np.int32)
    xr = x[perm_src[:m] // k]
    xp = np.zeros((M_cap, H), np.float32)
    xp[:m] = xr
    dxp, doff = G.up(xp, tdt), G.up_i32(offsets)
    dense = [G.up(w, tdt) for w in (wg, wu, wd)]
    padded = [_padded(wg, pg, tdt), _padded(wu, pg, tdt), _padded(wd, pd, tdt)]
    assert padded[0].stride(1) == H + pg and padded[2].stride(1) == I + pd
    y1, _ = moe.moe_grouped_swiglu_ffn(dxp, *dense, doff)
    y2, ws2 = moe.moe_grouped_swiglu_ffn(dxp, *padded, doff)
    torch.cuda.synchronize()
    assert torch.equal(y2[:m], y1[:m])
    h_ref, y_ref = O.grouped_swiglu_ffn(xr, wg, wu, wd, offsets, bf16=dt == "bf16")
    if dt == "bf16":
        G.check_bf16(G.down(y2)[:m], y_ref, "padded y", scale=G.down_scale(h_ref, wd, offsets))
        dx, dps = G.up(x, tdt), G.up_i32(perm_src)
        y3, _ = moe.moe_grouped_swiglu_ffn_gather(dx, dps, k, *padded, doff)
        torch.cuda.synchronize()
        assert torch.equal(y3[:m], y1[:m])
    else:
        G.check_f32(G.down(y2)[:m], y_ref, "padded y")


def test_load_sweep_padded_weight_rows():
    """The sweep over weight copies with padded rows leaves the same y as
    over dense copies."""
    banner("sweep qwen3 expert padded rows")
    shape = CONFIGS["qwen3"]
    wg, wu, wd = make_experts(shape, [5], seed=0)
    x, *_ = make_router(shape, 96, 0.0, seed=0)
    rot = 3
    dx = G.up(x, torch.bfloat16)
    ys = []
    for pad in (0, 64):
        w = [_padded(np.repeat(a, rot, 0), pad, torch.bfloat16) for a in (wg, wu, wd)]
        y = torch.full((96, shape.H), float("nan"), dtype=torch.bfloat16, device="cuda")
        moe.moe_load_sweep(dx, *w, [1, 96], warmup=1, iters=2, y_scratch=y)
        ys.append(y)
    torch.cuda.synchronize()
    assert torch.equal(ys[0], ys[1])
    _, yref = O.swiglu_rows(x, wg[0], wu[0], wd[0], bf16=True)
    G.check_bf16(G.down(ys[1]), yref, "padded sweep y")
