"""Pins of the MXFP8 oracle: the E4M3 encoding against torch's float8_e4m3fn,
the OCP MX block-scale rule, hand-derived blocks, round trips of values
already on the grid, the FFN's wiring against a torch restatement, and
planted mistakes.
"""
import numpy as np
import pytest
import torch

from oracle import mx_oracle as X


def torch_e4m3(v):
    """torch's RNE cast to float8_e4m3fn, as codes (inputs within +-448)."""
    return torch.tensor(np.asarray(v, np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_decode_table_matches_torch():
    t = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).float().numpy().astype(np.float64)
    mine = X.e4m3_decode(np.arange(256))
    nan = np.isnan(mine)
    assert np.array_equal(nan, np.isnan(t)) and nan.sum() == 2
    assert np.array_equal(mine[~nan], t[~nan])
    assert X.e4m3_decode(0x7E) == 448.0 and X.e4m3_decode(0x01) == 2.0 ** -9


def test_encode_round_trips_every_finite_code():
    codes = np.array([c for c in range(256) if (c & 0x7F) != 0x7F])
    assert np.array_equal(X.e4m3_encode(X.e4m3_decode(codes)), codes)           # -0 included
    assert X.e4m3_encode(-2.0 ** -12) == 0x80 and X.e4m3_encode(2.0 ** -12) == 0  # signed zero


def test_encode_matches_torch_including_ties():
    rng = np.random.default_rng(0)
    v = np.concatenate([rng.uniform(-448, 448, 20000), rng.uniform(-1, 1, 20000), rng.uniform(-0.02, 0.02, 5000)])
    vals = X.e4m3_decode(np.arange(0, 127))
    mids = (vals[:-1] + vals[1:]) / 2                        # exact midpoints: ties to even
    v = np.concatenate([v, mids, -mids]).astype(np.float32)
    mine, ref = X.e4m3_encode(v.astype(np.float64)), torch_e4m3(v)
    assert np.array_equal(mine, ref)


def test_block_scale_rule_hand_derived():
    v = np.arange(1, 33, dtype=np.float64)[None, :]          # max 32: s = 5 - 8 = -3, elements 8 .. 256
    q, s = X.mx_quantize(v)
    assert s[0, 0] == 127 - 3
    d = X.mx_dequantize(q, s)[0]
    assert list(d[:8]) == [1, 2, 3, 4, 5, 6, 7, 8]           # 8k exactly representable up to 64
    # 17 * 8 = 136 sits halfway between 128 (mantissa 0) and 144 (mantissa 1): even wins, 128;
    # 19 * 8 = 152 halfway between 144 (mantissa 1) and 160 (mantissa 2): 160; 18 * 8 = 144 exact
    assert d[16] == 16.0 and d[17] == 18.0 and d[18] == 20.0
    assert X.e4m3_decode(q[0, 16]) == 128.0 and X.e4m3_decode(q[0, 31]) == 256.0
    z, zs = X.mx_quantize(np.zeros((1, 32)))
    assert np.all(z == 0) and zs[0, 0] == 0                  # all-zero block: s = -127
    big = np.full((1, 32), 500.0)                            # 500: s = 8 - 8 = 0 ... clamp to 448
    q, s = X.mx_quantize(big)
    assert s[0, 0] == 127 and np.all(X.e4m3_decode(q) == 448.0)


@pytest.mark.parametrize("seed", range(4))
def test_block_properties_and_error_bound(seed):
    rng = np.random.default_rng(seed)
    v = rng.standard_normal((64, 256)) * np.exp2(rng.integers(-20, 20, (64, 1)))
    q, s = X.mx_quantize(v)
    vals = np.abs(X.e4m3_decode(q)).reshape(64, 8, 32)
    assert np.all(vals.max(axis=-1) >= 256) and np.all(vals.max(axis=-1) <= 448)
    d = X.mx_dequantize(q, s).reshape(64, 8, 32)
    vb = v.reshape(64, 8, 32)
    scale = np.exp2(s.astype(np.float64) - 127)[..., None]
    # RNE: within half a step; the step at E4M3 value |u| is 2^(floor(log2|u|) - 3), >= 2^-9
    u = np.abs(vb) / scale
    step = np.exp2(np.maximum(np.floor(np.log2(np.maximum(u, 2.0 ** -9))), -6) - 3)
    clamped = u > 448
    err = np.abs(d - vb) / scale
    assert np.all(err[~clamped] <= step[~clamped] / 2 + 1e-12)


def test_values_on_the_grid_round_trip():
    rng = np.random.default_rng(5)
    codes = rng.integers(0, 127, (16, 128)).astype(np.uint8)
    codes[:, ::32] = 0x7E                                    # each block holds 448 = 1.75 * 2^8
    scales = rng.integers(100, 150, (16, 4)).astype(np.uint8)
    v = X.mx_dequantize(codes, scales)
    q, s = X.mx_quantize(v)
    assert np.array_equal(s, scales) and np.array_equal(X.mx_dequantize(q, s), v)


def test_ffn_wiring_against_torch():
    """One expert: the oracle's FFN equals a torch restatement on the
    dequantised operands (fp64 matmuls, fp32 SiLU, the pinned quantiser)."""
    rng = np.random.default_rng(9)
    M, H, I = 5, 64, 96
    x, wg, wu, wd = (rng.standard_normal(s) for s in ((M, H), (1, I, H), (1, I, H), (1, H, I)))
    xq, xs = X.mx_quantize(x)
    (gq, gs), (uq, us), (dq, ds) = X.mx_quantize(wg), X.mx_quantize(wu), X.mx_quantize(wd)
    hq, hs, h32, y, mag = X.grouped_swiglu_ffn_mx(xq, xs, gq, gs, uq, us, dq, ds, [0, M])
    T = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    xd = T(X.mx_dequantize(xq, xs))
    G = (xd @ T(X.mx_dequantize(gq, gs))[0].T).float()
    U = (xd @ T(X.mx_dequantize(uq, us))[0].T).float()
    h = torch.nn.functional.silu(G) * U
    assert np.allclose(h.numpy(), h32, rtol=2e-6, atol=1e-7)
    q2, s2 = X.mx_quantize(h32)
    assert np.array_equal(q2, hq) and np.array_equal(s2, hs)
    yref = (T(X.mx_dequantize(hq, hs)) @ T(X.mx_dequantize(dq, ds))[0].T).float().bfloat16().float().numpy()
    assert np.array_equal(yref, y)


# ---------------------------------------------------------------- planted mistakes
MX_MUTANTS = {
    "scale_exponent_off_by_one": ("ex - 1.0 - 8.0", "ex - 1.0 - 7.0"),
    "truncate_not_round": ("pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (_CODES[hi] % 2 == 0))", "pick_hi = d_hi < 0"),
    "ties_away_from_zero": ("((d_hi == d_lo) & (_CODES[hi] % 2 == 0))", "(d_hi == d_lo)"),
    "no_clamp": ("scaled = np.clip(xb / np.exp2(e)[..., None], -E4M3_MAX, E4M3_MAX)",
                 "scaled = xb / np.exp2(e)[..., None]"),
    "gate_up_swapped": ("h = ((G * sig).astype(F32) * U).astype(F32)",
                        "h = ((U * (F32(1.0) / (F32(1.0) + np.exp(-U)))).astype(F32) * G).astype(F32)"),
    "h_not_requantised": ("Hd = mx_dequantize(hq[r0:r1], hs[r0:r1])", "Hd = h.astype(np.float64)"),
    "decode_bias_8": ("np.exp2(e - 7.0)", "np.exp2(e - 8.0)"),
}


def _mx_mutant(old, new):
    import types
    src = open(X.__file__).read()
    assert src.count(old) == 1, old
    mod = types.ModuleType("oracle.mx_mutant")
    mod.__file__ = X.__file__
    mod.__package__ = "oracle"
    exec(compile(src.replace(old, new), X.__file__, "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("mname", sorted(MX_MUTANTS))
def test_mx_mutant_is_caught(mname):
    global X
    orig = X
    X = _mx_mutant(*MX_MUTANTS[mname])
    failures = 0
    calls = [test_decode_table_matches_torch, test_encode_round_trips_every_finite_code,
             test_encode_matches_torch_including_ties, test_block_scale_rule_hand_derived,
             test_values_on_the_grid_round_trip, test_ffn_wiring_against_torch]
    calls += [lambda s=s: test_block_properties_and_error_bound(s) for s in range(4)]
    try:
        for c in calls:
            try:
                c()
            except Exception:
                failures += 1
    finally:
        X = orig
    assert failures, f"no pin caught mutant {mname}"
