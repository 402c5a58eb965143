"""CPU tests of the oracle against its pins (no GPU).

The pins live in ``oracle_pins``; the planted-mistake tests below replace one
oracle function by a plausible slip and check that some pin catches it.
"""
import types

import numpy as np
import pytest

from oracle import moe_oracle as O
from oracle import bruteforce as bf
import oracle_pins as P


@pytest.mark.parametrize("name,pin", P.ALL_PINS, ids=[n for n, _ in P.ALL_PINS])
def test_pin(name, pin):
    pin(O)


def test_bf16_rne_matches_torch():
    """The oracle's bf16 rounding equals torch's float32 -> bfloat16 cast."""
    import torch
    g = np.random.default_rng(0)
    vals = [g.standard_normal(20000).astype(np.float32) * s for s in (1e-3, 1.0, 1e4)]
    # exact halfway cases with even and odd kept bits, both signs
    base = g.integers(0, 0x7F7F, 4000, dtype=np.uint32) << 16  # finite patterns
    ties = (base | np.uint32(0x8000)).view(np.float32)
    ties = np.concatenate([ties, -ties])
    special = np.array([0.0, -0.0, 1e-40, -1e-40, 3.4e38, -3.4e38, np.inf, -np.inf,
                        1.0 + 2 ** -8, 1.0 + 3 * 2 ** -9], np.float32)
    a = np.concatenate(vals + [ties, special]).astype(np.float32)
    ref = torch.from_numpy(a).to(torch.bfloat16).float().numpy()
    got = O.bf16_rne(a)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))
    # and the brute force's independent rounding agrees on finite values
    fin = a[np.isfinite(a)][:3000]
    bb = np.array([bf.bf16(float(v)) for v in fin], np.float32)
    assert np.array_equal(bb, O.bf16_rne(fin))


def test_bf16_rne_nan():
    a = np.array([np.nan, 1.0], np.float32)
    r = O.bf16_rne(a)
    assert np.isnan(r[0]) and r[1] == 1.0


def test_closed_form_example():
    """Hand-derivable 2-token example: every value follows from the definitions.

    x = I_2, router rows (0.5,0), (0,0.5), (0.25,0.25), no bias, top-2, all
    experts local, I = 1. Token 0 picks experts 0 then 2, token 1 picks 1 then 2.
    """
    import math
    x = np.eye(2, dtype=np.float32)
    wr = np.array([[0.5, 0], [0, 0.5], [0.25, 0.25]], np.float32)
    b = np.zeros(3, np.float32)
    wg = np.array([[[2.0, 0.0]], [[0.0, 1.0]], [[1.0, -1.0]]], np.float32)   # [E, I=1, H]
    wu = np.array([[[1.0, 1.0]], [[2.0, 0.0]], [[0.5, 0.5]]], np.float32)
    wd = np.array([[[1.0], [-1.0]], [[0.5], [0.5]], [[2.0], [0.0]]], np.float32)  # [E, H, I]
    r = O.moe_layer(x, wr, b, 2, np.arange(3, dtype=np.int32), wg, wu, wd, bf16=False)
    assert r["ids"].tolist() == [[0, 2], [1, 2]]
    assert r["counts"].tolist() == [1, 1, 2]
    assert r["offsets"].tolist() == [0, 1, 2, 4]
    assert r["perm_src"].tolist() == [0, 2, 1, 3]
    assert r["dest"].tolist() == [0, 2, 1, 3]
    silu = lambda g: g / (1 + math.exp(-g))
    w0 = 1 / (1 + math.exp(-0.25))
    # token 0: expert 0 -> G=2, U=1, h=silu(2), y=(h,-h); expert 2 -> G=1, U=0.5
    h00 = silu(2.0)
    h02 = silu(1.0) * 0.5
    out0 = [w0 * h00 + (1 - w0) * 2 * h02, w0 * -h00 + 0.0]
    # token 1: expert 1 -> G=1, U=0, h=0; expert 2 -> G=-1, U=0.5
    h12 = silu(-1.0) * 0.5
    out1 = [w0 * 0.0 + (1 - w0) * 2 * h12, 0.0]
    np.testing.assert_allclose(r["out"], np.array([out0, out1]), rtol=2e-7, atol=1e-7)


def test_order_floor_small():
    """fp32 vs fp64 accumulation with identical rounding points stays close."""
    inp = P.tiny_inputs(seed=12, T=64, H=64, I=96, E=8, k=2, bf16=True)
    args = (inp["x"], inp["w_router"], inp["bias"], inp["k"], inp["expert_map"],
            inp["w_gate"], inp["w_up"], inp["w_down"])
    a = O.moe_layer(*args, bf16=True, acc="f32")["out"]
    b = O.moe_layer(*args, bf16=True, acc="f64")["out"]
    rms = float(np.sqrt(np.mean(b.astype(np.float64) ** 2)))
    d = float(np.max(np.abs(a - b))) / rms
    assert d < 0.05


def test_rows_form_matches_layer():
    """The per-token form used for full-size sampling equals the whole layer."""
    inp = P.tiny_inputs(seed=13, T=30, E=7, k=2, n_local=4, bf16=True)
    args = (inp["x"], inp["w_router"], inp["bias"], inp["k"], inp["expert_map"],
            inp["w_gate"], inp["w_up"], inp["w_down"])
    full = O.moe_layer(*args, bf16=True)
    rows = np.array([0, 3, 7, 29, 11])
    part = O.moe_layer_rows(*args, bf16=True, rows=rows)
    assert np.array_equal(part["ids"], full["ids"][rows])
    ulp = 2.0 ** (np.floor(np.log2(np.maximum(np.abs(full["out"][rows]), 1e-30))) - 7)
    assert np.all(np.abs(part["out"] - full["out"][rows]) <= 2 * ulp)


# --------------------------------------------------------------------------
# Planted mistakes: each replaces one oracle function; some pin must fail.
# --------------------------------------------------------------------------
def _mutant(**repl):
    ns = types.SimpleNamespace(**{k: getattr(O, k) for k in dir(O) if not k.startswith("__")})
    for k, v in repl.items():
        setattr(ns, k, v)

    # moe_layer must call the namespace's (possibly mutated) functions
    def moe_layer(x, w_router, bias, k, expert_map, w_gate, w_up, w_down, bf16, acc="f32"):
        z = ns.router_logits(x, w_router, bias)
        ids = ns.topk_select(z, k)
        w = ns.topk_weights(z, ids)
        counts = ns.expert_histogram(ids, z.shape[1])
        offsets = ns.local_offsets(counts, expert_map)
        x_perm, perm_src, dest = ns.permute(x, ids, expert_map, offsets)
        h, y = ns.grouped_swiglu_ffn(x_perm, w_gate, w_up, w_down, offsets, bf16, acc)
        out = ns.unpermute_combine(y, w, dest, np.shape(x)[0], k, bf16)
        return dict(logits=z, ids=ids, weights=w, counts=counts, offsets=offsets,
                    x_perm=x_perm, perm_src=perm_src, dest=dest, h=h, y_perm=y, out=out)
    ns.moe_layer = moe_layer
    return ns


def _no_bias(x, w, b):
    return np.matmul(np.asarray(x, np.float32), np.asarray(w, np.float32).T).astype(np.float32)


def _ties_high(z, k):
    z = np.asarray(z, np.float32)
    E = z.shape[1]
    order = np.argsort(-z[:, ::-1].astype(np.float64), axis=1, kind="stable")
    return (E - 1 - order[:, :k]).astype(np.int32)


def _softmax_over_all(z, ids):
    z = np.asarray(z, np.float32)
    p = np.exp(z - z.max(1, keepdims=True))
    p = p / p.sum(1, keepdims=True)
    return np.take_along_axis(p, np.asarray(ids, np.int64), 1).astype(np.float32)


def _hist_off_by_one(ids, E):
    c = O.expert_histogram(ids, E)
    return np.roll(c, 1)


def _unstable_permute(x, ids, expert_map, offsets):
    xp, ps, dest = O.permute(x, ids, expert_map, offsets)
    k = np.shape(ids)[1]
    offsets = np.asarray(offsets)
    for s in range(len(offsets) - 1):
        a, b = offsets[s], offsets[s + 1]
        ps[a:b] = ps[a:b][::-1].copy()
    dest = np.full_like(dest, -1)
    dest[ps] = np.arange(len(ps))
    return np.asarray(x, np.float32)[ps // k], ps, dest


def _ffn_swap(x_perm, wg, wu, wd, off, bf16, acc="f32"):
    return O.grouped_swiglu_ffn(x_perm, wu, wg, wd, off, bf16, acc)


def _ffn_sigmoid(x_perm, wg, wu, wd, off, bf16, acc="f32"):
    off = np.asarray(off)
    I, H = np.shape(wg)[1], np.shape(wg)[2]
    h_all = np.zeros((off[-1], I), np.float32)
    y_all = np.zeros((off[-1], H), np.float32)
    for s in range(len(off) - 1):
        X = np.asarray(x_perm)[off[s]:off[s + 1]]
        G, U = X @ wg[s].T, X @ wu[s].T
        h = (1 / (1 + np.exp(-G))) * U
        h_all[off[s]:off[s + 1]] = h
        y_all[off[s]:off[s + 1]] = h @ wd[s].T
    return h_all, y_all


def _ffn_wrong_expert(x_perm, wg, wu, wd, off, bf16, acc="f32"):
    n = np.shape(wg)[0]
    perm = np.roll(np.arange(n), 1)
    return O.grouped_swiglu_ffn(x_perm, wg[perm], wu[perm], wd[perm], off, bf16, acc)


def _ffn_down_not_transposed(x_perm, wg, wu, wd, off, bf16, acc="f32"):
    # reinterpret the [H, I] down matrix as [I, H] (a reshape instead of a transpose)
    n, H, I = np.shape(wd)
    return O.grouped_swiglu_ffn(x_perm, wg, wu, np.asarray(wd).reshape(n, I, H)
                                .transpose(0, 2, 1), off, bf16, acc)


def _combine_unweighted(y, w, dest, T, k, bf16):
    return O.unpermute_combine(y, np.ones_like(np.asarray(w)), dest, T, k, bf16)


def _combine_first_only(y, w, dest, T, k, bf16):
    d = np.asarray(dest).reshape(T, k).copy()
    d[:, 1:] = -1
    return O.unpermute_combine(y, w, d.ravel(), T, k, bf16)


def _no_round(a):
    return np.asarray(a, np.float32)


MUTANTS = {
    "router_drops_bias": dict(router_logits=_no_bias),
    "ties_to_higher_id": dict(topk_select=_ties_high),
    "softmax_not_renormalised": dict(topk_weights=_softmax_over_all),
    "histogram_shifted": dict(expert_histogram=_hist_off_by_one),
    "unstable_permutation": dict(permute=_unstable_permute),
    "gate_up_swapped": dict(grouped_swiglu_ffn=_ffn_swap),
    "sigmoid_for_silu": dict(grouped_swiglu_ffn=_ffn_sigmoid),
    "wrong_expert_weights": dict(grouped_swiglu_ffn=_ffn_wrong_expert),
    "down_not_transposed": dict(grouped_swiglu_ffn=_ffn_down_not_transposed),
    "combine_ignores_weights": dict(unpermute_combine=_combine_unweighted),
    "combine_drops_slots": dict(unpermute_combine=_combine_first_only),
    "bf16_rounding_skipped": dict(bf16_rne=_no_round),
}


@pytest.mark.parametrize("mname", sorted(MUTANTS))
def test_planted_mistake_is_caught(mname):
    ns = _mutant(**MUTANTS[mname])
    if mname == "bf16_rounding_skipped":
        # bf16_rne is looked up through the module, so patch it there
        orig = O.bf16_rne
        O.bf16_rne = _no_round
        try:
            failures = _count_failures(_mutant())
        finally:
            O.bf16_rne = orig
    else:
        failures = _count_failures(ns)
    assert failures, f"no pin caught mutant {mname}"


def _count_failures(ns):
    failed = []
    for name, pin in P.ALL_PINS:
        try:
            pin(ns)
        except (AssertionError, ValueError, IndexError):
            failed.append(name)
    return failed


@pytest.mark.parametrize("name,T,alpha", [("dsv3_shard", 512, 0.0), ("maverick_shard", 1024, 1.0),
                                          ("qwen3", 256, 1.0)])
def test_tolerance_rule_accepts_two_correct_oracles(name, T, alpha):
    """The bf16 comparison rule used on the GPU must accept the fp32-accumulate
    oracle against the fp64-accumulate oracle (same rounding points): both are
    correct, so any rule that rejects one of them is too tight."""
    import gpu_helpers as G
    from synth import make_layer
    li = make_layer(name, T, alpha, seed=0)
    a = G.oracle_layer(li, "f32")
    b = G.oracle_layer(li, "f64")
    G.check_bf16(a["y_perm"], b["y_perm"], "y", scale=G.down_scale(b["h"], li.w_down, b["offsets"]))
    G.check_bf16(a["out"], b["out"], "out",
                 scale=G.combine_scale(b["weights"], b["y_perm"], b["dest"], T, li.shape.k))
