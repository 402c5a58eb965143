"""CPU oracle for the MXFP8 expert FFN. TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this module. The product path never imports it.

The paper runs its models in FP8 (Table 2a) without stating a scaling
scheme. Reading: OCP Microscaling (MX) FP8 -- elements in FP8 E4M3 (the OCP
"E4M3FN" encoding: bias 7, no infinities, S.1111.111 is NaN, largest finite
448) sharing one E8M0 scale X = 2^(e - 127) per block of 32 consecutive
elements along the reduction dimension. Quantising a block (OCP MX v1.0,
conversion from higher precision):
    shared exponent  s = floor(log2(max_i |v_i|)) - 8   (8 = exponent of
                     E4M3's largest power of two), clamped to [-127, 127];
                     an all-zero block takes s = -127
    element          q_i = RNE_E4M3( clamp(v_i / 2^s, -448, 448) )
(round to nearest, ties to even; E4M3 has a signed zero, and a value that
rounds to zero keeps its sign, as in IEEE 754 rounding). Dequantised value =
E4M3(q_i) * 2^s.

The expert FFN in MXFP8 (the bf16 layer of ``moe_oracle`` with FP8
operands): x rows and weights quantised per block of 32 along H (gate/up)
and I (down); G = X W_gate^T and U = X W_up^T from the dequantised values;
h = silu(G) * U in fp32 (as in ``moe_oracle``), quantised per block of 32
along I; y = bf16( h W_down^T ) from the dequantised values. The matmuls are
taken in fp64 here: the hardware's FP8 dot products are only accurate to
about 2^-12 of the summed term magnitudes, so the parity rule is stated
against |a| |b| sums, not against a particular fp32 order.

Scales are returned as [rows, K / 32] uint8 (E8M0 codes); the GPU path keeps
them in its own layout. Shares no code with the GPU path or ``synth``.
"""
from __future__ import annotations

import numpy as np

from .moe_oracle import bf16_rne, F32

E4M3_MAX = 448.0


def e4m3_decode(codes) -> np.ndarray:
    """float64 values of E4M3 codes (NaN for S.1111.111)."""
    c = np.asarray(codes, np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = (c & 7).astype(np.float64)
    v = np.where(e == 0, m * 2.0 ** -9, (1.0 + m / 8.0) * np.exp2(e - 7.0))
    v = np.where((e == 15) & ((c & 7) == 7), np.nan, v)
    return sign * v


def _finite_table():
    codes = np.arange(128)
    vals = e4m3_decode(codes)
    ok = ~np.isnan(vals)
    return codes[ok], vals[ok]                      # non-negative codes 0..126, ascending values


_CODES, _VALS = _finite_table()


def e4m3_encode(v) -> np.ndarray:
    """RNE to E4M3 of values already clamped to [-448, 448] (float64 in)."""
    v = np.asarray(v, np.float64)
    a = np.abs(v)
    if np.any(a > E4M3_MAX) or np.any(np.isnan(a)):
        raise ValueError("e4m3_encode takes finite values within +-448")
    hi = np.searchsorted(_VALS, a, side="left").clip(0, len(_VALS) - 1)   # first value >= a
    lo = (hi - 1).clip(0)
    d_lo, d_hi = a - _VALS[lo], _VALS[hi] - a
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (_CODES[hi] % 2 == 0))
    pick_hi = np.where(_VALS[hi] == a, True, pick_hi)
    idx = np.where(pick_hi, hi, lo)
    code = _CODES[idx].astype(np.int64)
    code = np.where(np.signbit(v), code | 0x80, code)
    return code.astype(np.uint8)


def mx_quantize(x, block: int = 32):
    """Rows of x [.., K] (K % 32 == 0) -> (codes [.., K] uint8, scales [.., K/32] uint8)."""
    x = np.asarray(x, np.float64)
    K = x.shape[-1]
    if K % block:
        raise ValueError("K must be a multiple of the block size")
    xb = x.reshape(x.shape[:-1] + (K // block, block))
    amax = np.abs(xb).max(axis=-1)
    _, ex = np.frexp(np.where(amax > 0, amax, 1.0))     # amax = f 2^ex, f in [0.5, 1)
    e = np.where(amax > 0, ex - 1.0 - 8.0, -127.0).clip(-127.0, 127.0)   # floor(log2 amax) - 8
    scaled = np.clip(xb / np.exp2(e)[..., None], -E4M3_MAX, E4M3_MAX)
    codes = e4m3_encode(scaled).reshape(x.shape)
    return codes, (e + 127.0).astype(np.uint8)


def mx_dequantize(codes, scales, block: int = 32) -> np.ndarray:
    c = np.asarray(codes)
    K = c.shape[-1]
    v = e4m3_decode(c).reshape(c.shape[:-1] + (K // block, block))
    v = v * np.exp2(np.asarray(scales, np.float64) - 127.0)[..., None]
    return v.reshape(c.shape)


def grouped_swiglu_ffn_mx(xq, xs, wgq, wgs, wuq, wus, wdq, wds, offsets, parts=False):
    """Per local expert l, rows [offsets[l], offsets[l+1]) of the MX-quantised
    x_perm. Returns (h codes [M,I], h scales [M,I/32], h fp32 before
    quantisation [M,I], y [M,H] fp32 holding bf16 values, |h||W_down|^T [M,H]);
    with parts=True also a dict of the fp64 G, U and their term magnitudes
    |X||W_gate|^T, |X||W_up|^T (for error bounds).
    """
    offsets = np.asarray(offsets, np.int64)
    m = int(offsets[-1])
    I, H = wgq.shape[1], wgq.shape[2]
    hq = np.zeros((m, I), np.uint8)
    hs = np.zeros((m, I // 32), np.uint8)
    h32 = np.zeros((m, I), F32)
    y = np.zeros((m, H), F32)
    mag = np.zeros((m, H))
    P = {k: np.zeros((m, I)) for k in ("G", "U", "magG", "magU")}
    for s in range(len(offsets) - 1):
        r0, r1 = int(offsets[s]), int(offsets[s + 1])
        if r1 == r0:
            continue
        X = mx_dequantize(xq[r0:r1], xs[r0:r1])
        Wg, Wu = mx_dequantize(wgq[s], wgs[s]), mx_dequantize(wuq[s], wus[s])
        G64, U64 = X @ Wg.T, X @ Wu.T
        if parts:
            P["G"][r0:r1], P["U"][r0:r1] = G64, U64
            P["magG"][r0:r1], P["magU"][r0:r1] = np.abs(X) @ np.abs(Wg).T, np.abs(X) @ np.abs(Wu).T
        G, U = G64.astype(F32), U64.astype(F32)
        with np.errstate(over="ignore"):
            sig = (F32(1.0) / (F32(1.0) + np.exp(-G))).astype(F32)
        h = ((G * sig).astype(F32) * U).astype(F32)
        h32[r0:r1] = h
        hq[r0:r1], hs[r0:r1] = mx_quantize(h)
        Hd = mx_dequantize(hq[r0:r1], hs[r0:r1])
        Wd = mx_dequantize(wdq[s], wds[s])
        y[r0:r1] = bf16_rne((Hd @ Wd.T).astype(F32))
        mag[r0:r1] = np.abs(Hd) @ np.abs(Wd).T
    if parts:
        return hq, hs, h32, y, mag, P
    return hq, hs, h32, y, mag
