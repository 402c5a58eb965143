"""Pins of the placement oracle (latency model, Algorithm 1 Phase 2, drift
detector, Algorithm 2) against facts fixed by the definitions and by
scheduling theory: closed forms, LPT list scheduling, Graham's bound against a
brute-force optimum, invariants and stopping rules.
"""
import heapq
import itertools
import math

import numpy as np
import pytest

from oracle import placement_oracle as P


def line_models(cs, a=0.0):
    """f_g(n) = a + c_g n for n >= 1 (knots on that line)."""
    kn = np.tile(np.array([1.0, 2.0, 4.0, 64.0]), (len(cs), 1))
    kt = np.array([[a + c * n for n in kn[0]] for c in cs])
    return kn, kt


# ---------------------------------------------------------------- f_g(n)
def test_latency_model_knots_interpolation_and_ends():
    kn = np.array([1.0, 4.0, 16.0])
    kt = np.array([10.0, 13.0, 40.0])
    assert P.latency(kn, kt, 0) == 0.0 and P.latency(kn, kt, -3) == 0.0
    assert P.latency(kn, kt, 0.5) == 10.0                      # floor below the first knot
    for n, t in zip(kn, kt):
        assert P.latency(kn, kt, n) == t
    assert P.latency(kn, kt, 2.5) == pytest.approx(11.5, abs=1e-12)   # midpoint of a segment
    assert P.latency(kn, kt, 10.0) == pytest.approx(26.5, abs=1e-12)
    assert P.latency(kn, kt, 28.0) == pytest.approx(40.0 + 27.0, abs=1e-12)  # last slope continued
    one = (np.array([8.0]), np.array([3.0]))
    assert P.latency(*one, 4.0) == 3.0 and P.latency(*one, 16.0) == pytest.approx(6.0)


def test_latency_model_on_a_line_is_the_line():
    kn, kt = line_models([2.5], a=7.0)
    for n in np.linspace(1.0, 200.0, 57):
        assert P.latency(kn[0], kt[0], n) == pytest.approx(7.0 + 2.5 * n, rel=1e-13)


def test_fit_is_monotone_and_keeps_monotone_data():
    n, t = P.fit_latency_model([64, 1, 8, 2], [90.0, 91.0, 89.0, 93.0])
    assert list(n) == [1, 2, 8, 64]
    assert list(t) == [91.0, 93.0, 93.0, 93.0]               # running maximum in load order
    n2, t2 = P.fit_latency_model([1, 2, 3], [1.0, 2.0, 5.0])
    assert list(t2) == [1.0, 2.0, 5.0]
    grid = np.linspace(0.1, 100, 400)
    vals = [P.latency(n, t, x) for x in grid]
    assert all(b >= a for a, b in zip(vals, vals[1:]))
    with pytest.raises(ValueError):
        P.fit_latency_model([1, 1], [1.0, 2.0])


# ---------------------------------------------------------------- Algorithm 1
def lpt(w, G):
    """Textbook LPT list scheduling: jobs in descending size, each to the
    least-loaded machine (lowest index on ties)."""
    heap = [(0.0, g) for g in range(G)]
    out = np.zeros(len(w), np.int32)
    for e in sorted(range(len(w)), key=lambda e: (-w[e], e)):
        load, g = heapq.heappop(heap)
        out[e] = g
        heapq.heappush(heap, (load + w[e], g))
    return out


@pytest.mark.parametrize("seed", range(6))
def test_equal_models_reduce_to_lpt(seed):
    rng = np.random.default_rng(seed)
    E, G = 48, 5
    w = rng.integers(0, 500, E).astype(float)
    kn, kt = line_models([1.3] * G, a=4.0)
    a, n, tau = P.greedy_placement(w, kn, kt)
    assert np.array_equal(a, lpt(list(w), G))
    assert np.allclose(tau, w.sum() / G, rtol=1e-14)
    kn, kt = P.eplb_models(G)                                 # EPLB's f(n) = n: the same placement
    assert np.array_equal(P.greedy_placement(w, kn, kt)[0], a)


def brute_force_makespan(w, G):
    best = math.inf
    for assign in itertools.product(range(G), repeat=len(w)):
        loads = [0.0] * G
        for e, g in enumerate(assign):
            loads[g] += w[e]
        best = min(best, max(loads))
    return best


@pytest.mark.parametrize("seed", range(12))
def test_graham_bound_against_brute_force(seed):
    rng = np.random.default_rng(100 + seed)
    E, G = 8, 3
    w = rng.integers(1, 60, E).astype(float)
    kn, kt = P.eplb_models(G)
    a, n, _ = P.greedy_placement(w, kn, kt)
    opt = brute_force_makespan(list(w), G)
    assert max(n) <= (4.0 / 3.0 - 1.0 / (3 * G)) * opt + 1e-9
    assert np.allclose(n, P.gpu_loads(a, w, G))


def test_speed_targets_closed_form():
    cs = [1.0, 1.07, 0.95, 1.02]
    kn, kt = line_models(cs)
    rng = np.random.default_rng(7)
    w = rng.integers(1, 100, 64).astype(float)
    _, n, tau = P.greedy_placement(w, kn, kt)
    inv = np.array([1.0 / c for c in cs])
    assert np.allclose(tau, w.sum() * inv / inv.sum(), rtol=1e-12)
    # every GPU ends within one expert's load of its target
    assert np.all(np.abs(n - tau) <= w.max() + 1e-9)
    # faster GPUs (smaller c) receive more tokens
    order = np.argsort(cs)
    assert np.all(np.diff(n[order]) <= w.max())
    # affine models: the speed is taken at the mean per-expert load N / E
    kn, kt = line_models(cs, a=25.0)
    _, _, tau = P.greedy_placement(w, kn, kt)
    inv = np.array([1.0 / (25.0 + c * w.sum() / len(w)) for c in cs])
    assert np.allclose(tau, w.sum() * inv / inv.sum(), rtol=1e-12)


def test_capacity_keeps_equal_expert_counts():
    rng = np.random.default_rng(3)
    E, G = 64, 8
    w = rng.zipf(1.5, E).astype(float)
    kn, kt = line_models([1.0 + 0.01 * g for g in range(G)])
    a, _, _ = P.greedy_placement(w, kn, kt, cap=E // G)
    assert np.all(np.bincount(a, minlength=G) == E // G)
    with pytest.raises(ValueError):
        P.greedy_placement(w, kn, kt, cap=E // G - 1)


def test_zero_load_layer_and_contiguous():
    kn, kt = line_models([1.0, 2.0])
    a, n, tau = P.greedy_placement(np.zeros(6), kn, kt, cap=3)
    assert list(a) == [0, 0, 0, 1, 1, 1] and list(n) == [0, 0] and list(tau) == [0, 0]
    assert list(P.contiguous_placement(8, 4)) == [0, 0, 1, 1, 2, 2, 3, 3]


def test_layer_latency_readings():
    kn, kt = line_models([1.0, 2.0], a=10.0)
    w = [3.0, 5.0]
    a = [0, 1]                                   # one expert per GPU: the readings agree
    assert P.layer_latency(a, w, kn, kt) == P.layer_latency(a, w, kn, kt, grouped=True) == 20.0
    a = [1, 1]                                   # two experts on GPU 1: f(8) vs f(3) + f(5)
    assert P.layer_latency(a, w, kn, kt) == pytest.approx(26.0)
    assert P.layer_latency(a, w, kn, kt, grouped=True) == pytest.approx(16.0 + 20.0)


# ---------------------------------------------------------------- drift detector
def test_cosine_distance_closed_forms():
    assert P.cosine_distance([1, 2, 3], [1, 2, 3]) == pytest.approx(0.0, abs=1e-15)
    assert P.cosine_distance([1, 2, 3], [10, 20, 30]) == pytest.approx(0.0, abs=1e-15)
    assert P.cosine_distance([1, 0], [0, 5]) == 1.0
    assert P.cosine_distance([1, 0], [1, 1]) == pytest.approx(1.0 - 1.0 / math.sqrt(2.0), rel=1e-14)
    assert P.cosine_distance([0, 0], [0, 0]) == 0.0 and P.cosine_distance([0, 0], [1, 0]) == 1.0
    rng = np.random.default_rng(0)
    u, v = rng.random(50), rng.random(50)
    assert P.cosine_distance(u, v) == pytest.approx(P.cosine_distance(v, u), rel=1e-14)


def test_window_sum():
    samples = [np.full(4, i) for i in range(150)]
    assert list(P.window_sum(samples, 100)) == [sum(range(50, 150))] * 4


# ---------------------------------------------------------------- Algorithm 2
def check_stop(a, w, kn, kt, eps, swaps, max_swaps):
    G = len(kn)
    n = P.gpu_loads(a, w, G)
    lat = [P.latency(kn[g], kt[g], n[g]) for g in range(G)]
    if max(lat) <= (1 + eps) * sum(lat) / G or swaps == max_swaps:
        return
    hi = max(range(G), key=lambda g: (lat[g], -g))
    lo = min(range(G), key=lambda g: (lat[g], g))
    for ei in np.flatnonzero(a == hi):
        for ej in np.flatnonzero(a == lo):
            nh, nl = n[hi] - w[ei] + w[ej], n[lo] - w[ej] + w[ei]
            assert max(P.latency(kn[hi], kt[hi], nh), P.latency(kn[lo], kt[lo], nl)) >= lat[hi]


@pytest.mark.parametrize("seed", range(8))
def test_incremental_update_stops_where_the_rule_says(seed):
    rng = np.random.default_rng(seed)
    E, G = 32, 4
    kn, kt = line_models([1.0, 1.04, 0.97, 1.07], a=30.0)
    w = rng.zipf(1.4, E).clip(max=400).astype(float)
    a0 = P.contiguous_placement(E, G)
    a, swaps = P.incremental_update(a0, w, kn, kt, eps=0.03)
    assert np.array_equal(np.bincount(a, minlength=G), np.bincount(a0, minlength=G))  # swaps only
    assert P.layer_latency(a, w, kn, kt) <= P.layer_latency(a0, w, kn, kt)
    check_stop(a, w, kn, kt, 0.03, swaps, 1 << 30)
    a1, s1 = P.incremental_update(a0, w, kn, kt, eps=0.03, max_swaps=1)
    assert s1 <= 1


def test_incremental_update_within_tolerance_does_nothing():
    # loads 100 / 98 / 99 / 97: max f = 130 <= 1.03 * mean 128.5, although the
    # swap 40 <-> 39 between GPUs 0 and 3 would still lower the maximum
    kn, kt = line_models([1.0] * 4, a=30.0)
    w = np.array([60, 40, 50, 48, 60, 39, 58, 39], float)
    a0 = np.array([0, 0, 1, 1, 2, 2, 3, 3], np.int32)
    a, swaps = P.incremental_update(a0, w, kn, kt, eps=0.03)
    assert swaps == 0 and np.array_equal(a, a0)
    a, swaps = P.incremental_update(a0, w, kn, kt, eps=0.0)
    assert swaps >= 1 and P.layer_latency(a, w, kn, kt) < 130.0


def test_incremental_update_moves_few_experts_under_drift():
    """Section 4.2.4: after a drift, a few swaps restore balance where a fresh
    greedy solve reassigns most experts."""
    rng = np.random.default_rng(11)
    E, G = 256, 8
    kn, kt = line_models([1.0 + 0.01 * g for g in range(G)], a=50.0)
    w1 = rng.zipf(1.3, E).clip(max=3000).astype(float) + rng.integers(0, 40, E)
    a1, _, _ = P.greedy_placement(w1, kn, kt, cap=E // G)
    w2 = w1.copy()
    hot = rng.choice(E, 6, replace=False)
    w2[hot] *= 3.0                                            # a few experts heat up
    a2, swaps = P.incremental_update(a1, w2, kn, kt, eps=0.03)
    fresh, _, _ = P.greedy_placement(w2, kn, kt, cap=E // G)
    moved_fresh = int((fresh != a1).sum())
    assert 0 < swaps <= 30
    assert 2 * swaps < moved_fresh
    assert P.layer_latency(a2, w2, kn, kt) < P.layer_latency(a1, w2, kn, kt)


# ---------------------------------------------------------------- planted mistakes
# Each mutant edits one line of the oracle's source; some pin above must fail.
PLACEMENT_MUTANTS = {
    "ascending_expert_order": ("key=lambda e: (-float(w[e]), e)", "key=lambda e: (float(w[e]), e)"),
    "argmin_instead_of_argmax": ("if gap > best_gap:", "if -gap > best_gap:"),
    "speed_not_inverted": ("s = [1.0 / latency(kn[g], kt[g], n_ref) for g in range(G)]",
                           "s = [latency(kn[g], kt[g], n_ref) for g in range(G)]"),
    "reference_load_is_total": ("n_ref = N / E", "n_ref = N"),
    "interpolation_wrong_segment": ("return lo_t + (hi_t - lo_t) * ((n - lo_n) / (hi_n - lo_n))",
                                    "return lo_t + (hi_t - lo_t) * ((n - lo_n) / (hi_n - lo_n + 1.0))"),
    "no_running_max": ("run = max(run, float(latencies[i]))", "run = float(latencies[i])"),
    "cosine_without_norm": ("return 1.0 - dot / (math.sqrt(na) * math.sqrt(nb))", "return 1.0 - dot"),
    "swap_gain_sign": ("gain = lat[hi] - new", "gain = new - lat[hi]"),
    "no_tolerance_stop": ("if lat[hi] <= (1.0 + eps) * fbar or hi == lo:", "if hi == lo:"),
    "capacity_ignored": ("if cap > 0 and cnt[g] >= cap:", "if False:"),
}


def _mutant_module(old, new):
    import types
    src = open(P.__file__).read()
    assert src.count(old) == 1, old
    mod = types.ModuleType("placement_mutant")
    mod.__file__ = P.__file__
    exec(compile(src.replace(old, new), P.__file__, "exec"), mod.__dict__)
    return mod


def _pin_calls():
    calls = [test_latency_model_knots_interpolation_and_ends, test_latency_model_on_a_line_is_the_line,
             test_fit_is_monotone_and_keeps_monotone_data, test_speed_targets_closed_form,
             test_capacity_keeps_equal_expert_counts, test_zero_load_layer_and_contiguous,
             test_layer_latency_readings, test_cosine_distance_closed_forms, test_window_sum,
             test_incremental_update_moves_few_experts_under_drift,
             test_incremental_update_within_tolerance_does_nothing]
    calls += [lambda s=s: test_equal_models_reduce_to_lpt(s) for s in range(6)]
    calls += [lambda s=s: test_graham_bound_against_brute_force(s) for s in range(12)]
    calls += [lambda s=s: test_incremental_update_stops_where_the_rule_says(s) for s in range(8)]
    return calls


@pytest.mark.parametrize("mname", sorted(PLACEMENT_MUTANTS))
def test_placement_mutant_is_caught(mname):
    global P
    orig = P
    P = _mutant_module(*PLACEMENT_MUTANTS[mname])
    failures = 0
    try:
        for call in _pin_calls():
            try:
                call()
            except Exception:
                failures += 1
    finally:
        P = orig
    assert failures, f"no pin caught mutant {mname}"
