"""CPU oracle for ViBE's placement control path. TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this module. The product path never imports it.

What is computed (Section 4.2 "Framework Design", Algorithm 1 "ViBE End-to-End
Flow" and Algorithm 2 "Incremental Placement Update"):

* f_g(n): a per-GPU latency model, token load -> kernel latency (Section
  4.2.1). It is built from measured (load, latency) points of the load sweep
  as a monotone piecewise-linear function (the paper does not give its form;
  reading below).
* Latency-aware greedy placement (Section 4.2.3, Algorithm 1 Phase 2), per
  layer: N = sum_e w_e; speed s_g = 1 / f_g(N / E); token target
  tau_g = N s_g / sum_h s_h; experts in descending w_e order each go to the
  GPU with the largest tau_g - n_g, which then gains w_e.
* EPLB's special case f_g(n) = n (all speeds equal, targets N / G) and the
  contiguous placement (GPU g holds experts [g E/G, (g+1) E/G)).
* Layer latency T = max_g f_g(n_g) with n_g = sum_{e in S_g} w_e (Section
  4.2.3), and the grouped reading max_g sum_{e in S_g} f_g(w_e).
* Drift detector (Section 4.2.4): cosine distance d = 1 - w.w_ref /
  (|w| |w_ref|) between the current and the reference load vector of a layer.
* Incremental placement update (Algorithm 2), per layer: while the slowest
  GPU's f_g(n_g) exceeds (1 + eps) times the mean over GPUs, take the slowest
  GPU g+ and the fastest g-, and apply the expert swap between them that
  lowers max(f_g+(n_g+), f_g-(n_g-)) the most; stop when no swap lowers it.

Readings where the paper is silent (the same choices are made by the GPU path):

* latency model: knots (n_k, t_k), n strictly increasing and positive, t the
  running maximum of the measured latencies (monotone); f(n) = 0 for n <= 0,
  t_0 for 0 < n <= n_0, linear between knots, and beyond the last knot the
  last segment's slope (t_0 n / n_0 with one knot). Evaluated as
  t_k + (t_{k+1} - t_k) * ((n - n_k) / (n_{k+1} - n_k)), each operation an
  IEEE fp64 operation in that order.
* ties: experts of equal load in ascending id; equal tau_g - n_g, equal
  latencies (g+, g-) and equal swap gains go to the lowest GPU index, the
  lowest pair (e_i, e_j) in ascending id order.
* capacity: Algorithm 1 has no per-GPU expert count; the paper's evaluation
  keeps E/G experts per GPU. ``cap`` > 0 excludes full GPUs from the argmax;
  cap = 0 is the unconstrained algorithm.
* N = 0 (a layer with no tokens): every speed is taken as 1.
* swaps only (Algorithm 2 exchanges two experts, so expert counts per GPU are
  kept); if g+ = g- or no swap gains, the loop ends; ``max_swaps`` bounds it.
* cosine distance of a zero vector: 0 if both are zero, else 1.
* loads are sums in ascending expert id, in fp64 (exact for integer counts).

Every function works on plain Python floats/ints or NumPy arrays in fp64 and
shares no code with the GPU path.
"""
from __future__ import annotations

import math

import numpy as np


# --------------------------------------------------------------------------
# Latency model f_g (Section 4.2.1)
# --------------------------------------------------------------------------
def fit_latency_model(loads, latencies):
    """Knots (n, t) from measured points: loads ascending, latencies made
    non-decreasing by a running maximum (the model must be monotone)."""
    order = sorted(range(len(loads)), key=lambda i: loads[i])
    n = [float(loads[i]) for i in order]
    for a, b in zip(n, n[1:]):
        if not b > a:
            raise ValueError("loads must be distinct")
    if n[0] <= 0:
        raise ValueError("loads must be positive")
    t, run = [], -math.inf
    for i in order:
        run = max(run, float(latencies[i]))
        t.append(run)
    return np.array(n, np.float64), np.array(t, np.float64)


def latency(kn, kt, n):
    """f(n) of one GPU's model with knots kn, kt (fp64)."""
    n = float(n)
    m = len(kn)
    if n <= 0.0:
        return 0.0
    if n <= kn[0]:
        return float(kt[0])
    if m == 1:
        return float(kt[0]) * (n / float(kn[0]))
    for k in range(m - 1):
        if n <= kn[k + 1]:
            lo_n, hi_n, lo_t, hi_t = float(kn[k]), float(kn[k + 1]), float(kt[k]), float(kt[k + 1])
            return lo_t + (hi_t - lo_t) * ((n - lo_n) / (hi_n - lo_n))
    lo_n, hi_n, lo_t, hi_t = float(kn[m - 2]), float(kn[m - 1]), float(kt[m - 2]), float(kt[m - 1])
    return hi_t + (hi_t - lo_t) * ((n - hi_n) / (hi_n - lo_n))


def gpu_loads(assign, w, G):
    """n_g = sum_{e in S_g} w_e, summed in ascending expert id."""
    n = [0.0] * G
    for e in range(len(w)):
        n[int(assign[e])] += float(w[e])
    return n


def layer_latency(assign, w, kn, kt, grouped=False):
    """T = max_g f_g(n_g) (Section 4.2.3); grouped: max_g sum_{e in S_g} f_g(w_e)."""
    G = len(kn)
    if not grouped:
        n = gpu_loads(assign, w, G)
        return max(latency(kn[g], kt[g], n[g]) for g in range(G))
    tot = [0.0] * G
    for e in range(len(w)):
        g = int(assign[e])
        tot[g] += latency(kn[g], kt[g], w[e])
    return max(tot)


# --------------------------------------------------------------------------
# Initial placement (Algorithm 1, Phase 2)
# --------------------------------------------------------------------------
def greedy_placement(w, kn, kt, cap=0):
    """One layer: returns (assign[E] int32, n[G] fp64 loads, tau[G])."""
    E, G = len(w), len(kn)
    if cap > 0 and cap * G < E:
        raise ValueError("capacity too small")
    N = 0.0
    for e in range(E):
        N += float(w[e])
    if N > 0.0:
        n_ref = N / E
        s = [1.0 / latency(kn[g], kt[g], n_ref) for g in range(G)]
    else:
        s = [1.0] * G
    S = 0.0
    for g in range(G):
        S += s[g]
    tau = [N * s[g] / S for g in range(G)]
    order = sorted(range(E), key=lambda e: (-float(w[e]), e))
    n = [0.0] * G
    cnt = [0] * G
    assign = np.zeros(E, np.int32)
    for e in order:
        best, best_gap = -1, -math.inf
        for g in range(G):
            if cap > 0 and cnt[g] >= cap:
                continue
            gap = tau[g] - n[g]
            if gap > best_gap:
                best, best_gap = g, gap
        assign[e] = best
        n[best] += float(w[e])
        cnt[best] += 1
    return assign, np.array(n), np.array(tau)


def eplb_models(G):
    """f_g(n) = n for every GPU (EPLB's implicit model, Section 4.2.3)."""
    kn = np.tile(np.array([1.0, 2.0]), (G, 1))
    return kn, kn.copy()


def contiguous_placement(E, G):
    """GPU g holds experts [g E/G, (g+1) E/G) (the default EP layout)."""
    if E % G:
        raise ValueError("E must be a multiple of G")
    return (np.arange(E) // (E // G)).astype(np.int32)


# --------------------------------------------------------------------------
# Drift detection (Section 4.2.4)
# --------------------------------------------------------------------------
def cosine_distance(w, w_ref):
    dot = na = nb = 0.0
    for a, b in zip(w, w_ref):
        a, b = float(a), float(b)
        dot += a * b
        na += a * a
        nb += b * b
    if na == 0.0 or nb == 0.0:
        return 0.0 if na == nb else 1.0
    return 1.0 - dot / (math.sqrt(na) * math.sqrt(nb))


def window_sum(samples, window):
    """Sum of the last `window` per-pass load vectors (integer counts)."""
    s = np.asarray(samples[-window:], np.int64)
    return s.sum(axis=0)


# --------------------------------------------------------------------------
# Incremental placement update (Algorithm 2)
# --------------------------------------------------------------------------
def incremental_update(assign, w, kn, kt, eps=0.03, max_swaps=1 << 30):
    """One layer: returns (new assign, number of swaps)."""
    assign = np.array(assign, np.int32).copy()
    E, G = len(w), len(kn)
    n = gpu_loads(assign, w, G)

    def mean_latency():
        tot = 0.0
        for g in range(G):
            tot += latency(kn[g], kt[g], n[g])
        return tot / G

    fbar = mean_latency()
    swaps = 0
    while swaps < max_swaps:
        lat = [latency(kn[g], kt[g], n[g]) for g in range(G)]
        hi = max(range(G), key=lambda g: (lat[g], -g))
        lo = min(range(G), key=lambda g: (lat[g], g))
        if lat[hi] <= (1.0 + eps) * fbar or hi == lo:
            break
        best, best_gain = None, 0.0
        for ei in range(E):
            if assign[ei] != hi:
                continue
            for ej in range(E):
                if assign[ej] != lo:
                    continue
                nh = n[hi] - float(w[ei]) + float(w[ej])
                nl = n[lo] - float(w[ej]) + float(w[ei])
                new = max(latency(kn[hi], kt[hi], nh), latency(kn[lo], kt[lo], nl))
                gain = lat[hi] - new
                if gain > best_gain:
                    best, best_gain = (ei, ej, nh, nl), gain
        if best is None:
            break
        ei, ej, nh, nl = best
        assign[ei], assign[ej] = lo, hi
        n[hi], n[lo] = nh, nl
        fbar = mean_latency()
        swaps += 1
    return assign, swaps
