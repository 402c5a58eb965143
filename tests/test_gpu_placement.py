"""GPU parity of the placement control path (latency-aware greedy placement,
incremental swap solver, window sums and drift distance) against the
placement oracle, through the C ABI. Decisions are exact: assignments, swap
counts and loads must match bit for bit.
"""
import numpy as np
import pytest
import torch

import paper_2606_00735_amd as moe
from oracle import placement_oracle as P

pytestmark = pytest.mark.gpu
DEV = "cuda"


def banner(*a):
    print("CASE", *a, flush=True)


def sweep_like_models(G, seed, nk=8):
    """Per-GPU curves shaped like a load sweep (a flat weight-streaming floor,
    then linear growth), scaled by up to 7 % per GPU."""
    rng = np.random.default_rng(seed)
    n = np.array([2.0 ** i for i in range(nk)]) * 8
    base = np.maximum(90.0, 0.35 * n) + rng.uniform(0, 3, nk)
    base = np.maximum.accumulate(base)
    scale = 1.0 + 0.07 * rng.random(G)
    kn = np.tile(n, (G, 1))
    kt = np.outer(scale, base)
    return kn, kt


def loads(Lyr, E, seed, integer=True, alpha=1.2):
    rng = np.random.default_rng(seed)
    if integer:
        w = np.stack([rng.zipf(1 + alpha, E).clip(max=5000) + rng.integers(0, 30, E) for _ in range(Lyr)])
        w[:, rng.integers(0, E)] = 0                    # an idle expert
        return w.astype(np.float64)
    return rng.gamma(0.7, 50.0, (Lyr, E))


def dev(a, dt=torch.float64):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV).to(dt).contiguous()


GREEDY = [
    (12, 256, 8, 32, True), (12, 256, 8, 0, True), (6, 64, 3, 0, True), (6, 1000, 64, 16, True),
    (4, 7, 2, 4, False), (3, 1, 1, 0, True), (8, 256, 8, 32, False), (5, 1024, 16, 64, True),
]


@pytest.mark.parametrize("Lyr,E,G,cap,integer", GREEDY, ids=[f"L{a}-E{b}-G{c}-cap{d}-{'int' if e else 'frac'}"
                                                             for a, b, c, d, e in GREEDY])
def test_greedy_matches_oracle(Lyr, E, G, cap, integer):
    banner("greedy", Lyr, E, G, cap, integer)
    W = loads(Lyr, E, seed=E + G, integer=integer)
    kn, kt = sweep_like_models(G, seed=G)
    a, n, tau = moe.moe_place_greedy(dev(W), dev(kn), dev(kt), cap=cap)
    torch.cuda.synchronize()
    a, n, tau = a.cpu().numpy(), n.cpu().numpy(), tau.cpu().numpy()
    for l in range(Lyr):
        ra, rn, rt = P.greedy_placement(W[l], kn, kt, cap=cap)
        assert np.array_equal(a[l], ra), f"layer {l}"
        assert np.array_equal(n[l], rn) and np.array_equal(tau[l], rt), f"layer {l}"


def test_greedy_ties_and_equal_models():
    banner("greedy ties")
    G, E = 4, 64
    W = np.tile(np.repeat([7.0, 3.0, 3.0, 0.0], 16), (3, 1))    # many equal loads
    kn, kt = P.eplb_models(G)
    a, _, _ = moe.moe_place_greedy(dev(W), dev(kn), dev(kt), cap=16)
    for l in range(3):
        assert np.array_equal(a.cpu().numpy()[l], P.greedy_placement(W[l], kn, kt, cap=16)[0])


INCR = [(8, 256, 8, 0.03, 1 << 16), (8, 256, 8, 0.0, 1 << 16), (6, 64, 4, 0.03, 1), (6, 64, 4, 0.03, 0),
        (4, 33, 3, 0.01, 1 << 16), (2, 1, 1, 0.03, 10)]


@pytest.mark.parametrize("Lyr,E,G,eps,max_swaps", INCR, ids=[f"L{a}-E{b}-G{c}-eps{d}-max{e}"
                                                             for a, b, c, d, e in INCR])
def test_incremental_matches_oracle(Lyr, E, G, eps, max_swaps):
    banner("incremental", Lyr, E, G, eps, max_swaps)
    W1 = loads(Lyr, E, seed=1)
    W2 = W1 * np.random.default_rng(2).uniform(0.5, 2.0, W1.shape).round(2)   # drifted loads
    kn, kt = sweep_like_models(G, seed=3)
    start = np.stack([P.greedy_placement(W1[l], kn, kt, cap=(E // G if E % G == 0 else 0))[0]
                      for l in range(Lyr)])
    a = dev(start, torch.int32)
    ns = moe.moe_place_incremental(dev(W2), dev(kn), dev(kt), a, eps=eps, max_swaps=max_swaps)
    torch.cuda.synchronize()
    a, ns = a.cpu().numpy(), ns.cpu().numpy()
    for l in range(Lyr):
        ra, rs = P.incremental_update(start[l], W2[l], kn, kt, eps=eps, max_swaps=max_swaps)
        assert np.array_equal(a[l], ra) and ns[l] == rs, f"layer {l}: {ns[l]} vs {rs} swaps"


def test_drift_distance_and_window():
    banner("drift window")
    Lyr, E, win = 5, 64, 100
    rng = np.random.default_rng(9)
    ring = torch.zeros((win, Lyr, E), dtype=torch.int32, device=DEV)
    sums = torch.zeros((Lyr, E), dtype=torch.float64, device=DEV)
    samples = []
    for i in range(130):
        c = rng.integers(0, 4000, (Lyr, E)).astype(np.int32)
        samples.append(c)
        moe.moe_window_push(dev(c, torch.int32), ring, sums, i % win)
    torch.cuda.synchronize()
    ref = P.window_sum(samples, win)
    assert np.array_equal(sums.cpu().numpy(), ref.astype(np.float64))
    cur = ref.astype(np.float64)
    refv = cur.copy()
    refv[1] = refv[1][::-1]                      # one layer drifts
    refv[2] = 0.0                                # a zero reference
    refv[3] = 3.0 * cur[3]                       # the same direction
    d, trig = moe.moe_drift_distance(dev(cur), dev(refv), delta=0.05)
    torch.cuda.synchronize()
    d = d.cpu().numpy()
    for l in range(Lyr):
        assert d[l] == P.cosine_distance(cur[l], refv[l]), f"layer {l}"
    assert int(trig.item()) == int(max(d) > 0.05) == 1
    d2, trig2 = moe.moe_drift_distance(dev(cur), dev(cur), delta=0.05)
    torch.cuda.synchronize()
    assert int(trig2.item()) == 0 and np.all(np.abs(d2.cpu().numpy()) < 1e-12)


def test_full_size_dsv3_like():
    """58 MoE layers, 256 experts on 8 GPUs with 32 slots each: a greedy solve,
    then the incremental update after a few experts heat up."""
    banner("placement dsv3-like L58 E256 G8")
    Lyr, E, G = 58, 256, 8
    W = loads(Lyr, E, seed=58)
    kn, kt = sweep_like_models(G, seed=8)
    a, n, _ = moe.moe_place_greedy(dev(W), dev(kn), dev(kt), cap=32)
    torch.cuda.synchronize()
    a = a.cpu().numpy()
    for l in range(Lyr):
        assert np.array_equal(a[l], P.greedy_placement(W[l], kn, kt, cap=32)[0]), f"layer {l}"
    W2 = W.copy()
    rng = np.random.default_rng(59)
    for l in range(Lyr):
        W2[l, rng.choice(E, 5, replace=False)] *= 3.0
    ad = dev(a, torch.int32)
    ns = moe.moe_place_incremental(dev(W2), dev(kn), dev(kt), ad, eps=0.03)
    torch.cuda.synchronize()
    ad, ns = ad.cpu().numpy(), ns.cpu().numpy()
    for l in range(0, Lyr, 6):
        ra, rs = P.incremental_update(a[l], W2[l], kn, kt, eps=0.03)
        assert np.array_equal(ad[l], ra) and ns[l] == rs, f"layer {l}"
    print("  swaps per layer: max", int(ns.max()), "mean", float(ns.mean()), flush=True)


def test_placement_cost_matches_oracle():
    banner("placement cost")
    Lyr, E, G = 10, 256, 8
    W = loads(Lyr, E, seed=4, integer=False)
    kn, kt = sweep_like_models(G, seed=5)
    rng = np.random.default_rng(6)
    A = rng.integers(0, G, (Lyr, E)).astype(np.int32)
    n, lat, latg = moe.moe_placement_cost(dev(W), dev(A, torch.int32), dev(kn), dev(kt))
    torch.cuda.synchronize()
    n, lat, latg = n.cpu().numpy(), lat.cpu().numpy(), latg.cpu().numpy()
    for l in range(Lyr):
        rn = P.gpu_loads(A[l], W[l], G)
        assert np.array_equal(n[l], rn)
        assert np.array_equal(lat[l], [P.latency(kn[g], kt[g], rn[g]) for g in range(G)])
        assert lat[l].max() == P.layer_latency(A[l], W[l], kn, kt)
        assert latg[l].max() == P.layer_latency(A[l], W[l], kn, kt, grouped=True)
