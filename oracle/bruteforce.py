"""Pure-Python brute force of the MoE layer for tiny inputs.

TEST INFRASTRUCTURE ONLY (same import rule as ``moe_oracle``). It exists to
pin the NumPy oracle: every step is re-derived with Python floats (fp64) and
plain loops, with its own bf16 rounding (exponent/ulp arithmetic rather than
bit patterns), so a slip in the oracle's vectorised indexing, transposes or
rounding shows up as a mismatch.

Definitions are the ones listed in ``moe_oracle`` (top-k routed MoE layer of
Section 2; activation profile of Section 4.2.2; per-GPU token load of
Section 4.2.3). Only use it on inputs of a few thousand multiply-adds.
"""
from __future__ import annotations

import math
import struct


def f32(v: float) -> float:
    """Round a Python float to the nearest binary32 value (RNE)."""
    return struct.unpack("<f", struct.pack("<f", v))[0]


def bf16(v: float) -> float:
    """Round a Python float to the nearest bf16 value, ties to even.

    bf16 has an 8-bit significand: for |v| in [2^e, 2^(e+1)) the spacing is
    2^(e-7). Python's round() on v / spacing (an exact scaling) rounds half to
    even.
    """
    if v == 0.0 or math.isnan(v) or math.isinf(v):
        return v
    e = math.floor(math.log2(abs(v)))
    # guard log2 rounding at exact powers of two
    if 2.0 ** e > abs(v):
        e -= 1
    elif 2.0 ** (e + 1) <= abs(v):
        e += 1
    e = max(e, -126)
    ulp = 2.0 ** (e - 7)
    return round(v / ulp) * ulp


def layer(x, w_router, bias, k, expert_map, w_gate, w_up, w_down, use_bf16):
    """Every intermediate of the layer, from nested lists / arrays of floats.

    x [T][H], w_router [E][H], bias [E], expert_map [E] (slot or -1),
    w_gate/w_up [E_local][I][H], w_down [E_local][H][I].
    """
    T = len(x)
    H = len(x[0]) if T else len(w_router[0])
    E = len(w_router)
    rnd = bf16 if use_bf16 else (lambda v: f32(v))

    # logits: the exact dot product (grid inputs make it exact in fp32 too),
    # then one fp32 rounding of the sum with the bias
    z = []
    for t in range(T):
        row = []
        for e in range(E):
            s = 0.0
            for h in range(H):
                s += float(x[t][h]) * float(w_router[e][h])
            row.append(f32(f32(s) + float(bias[e])))
        z.append(row)

    ids, wts = [], []
    for t in range(T):
        order = sorted(range(E), key=lambda e: (-z[t][e], e))[:k]
        ids.append(order)
        p = [math.exp(z[t][e] - z[t][order[0]]) for e in order]
        s = sum(p)
        wts.append([v / s for v in p])

    counts = [0] * E
    for t in range(T):
        for e in ids[t]:
            counts[e] += 1

    n_local = sum(1 for s in expert_map if s >= 0)
    slot_expert = [None] * n_local
    for e, s in enumerate(expert_map):
        if s >= 0:
            slot_expert[s] = e
    rows_of = {s: [] for s in range(n_local)}
    for t in range(T):
        for j in range(k):
            s = expert_map[ids[t][j]]
            if s >= 0:
                rows_of[s].append(t * k + j)
    offsets = [0]
    for s in range(n_local):
        offsets.append(offsets[-1] + counts[slot_expert[s]])
    perm_src = [i for s in range(n_local) for i in rows_of[s]]
    dest = [-1] * (T * k)
    for pos, i in enumerate(perm_src):
        dest[i] = pos

    def expert(s, xrow):
        I = len(w_gate[s])
        h = []
        for i in range(I):
            g = sum(float(xrow[c]) * float(w_gate[s][i][c]) for c in range(H))
            u = sum(float(xrow[c]) * float(w_up[s][i][c]) for c in range(H))
            h.append(rnd(g / (1.0 + math.exp(-g)) * u) if g > -700 else rnd(0.0 * u))
        y = [rnd(sum(h[i] * float(w_down[s][c][i]) for i in range(I))) for c in range(H)]
        return h, y

    y_perm = []
    h_perm = []
    for pos, i in enumerate(perm_src):
        t = i // k
        s = expert_map[ids[t][i % k]]
        h, y = expert(s, x[t])
        h_perm.append(h)
        y_perm.append(y)

    out = []
    for t in range(T):
        acc = [0.0] * H
        for j in range(k):
            d = dest[t * k + j]
            if d >= 0:
                for c in range(H):
                    acc[c] += wts[t][j] * y_perm[d][c]
        out.append([rnd(v) for v in acc])

    return dict(logits=z, ids=ids, weights=wts, counts=counts, offsets=offsets,
                perm_src=perm_src, dest=dest, h=h_perm, y_perm=y_perm, out=out)
