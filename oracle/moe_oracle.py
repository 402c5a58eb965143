"""CPU oracle for one GPU's share of an expert-parallel MoE layer.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module. The product path
(``paper_2606_00735_amd``) never imports it and has no CPU fallback.

What is computed (the paper treats the fused MoE kernel as a black box it
profiles, Sections 4.2.1 and 5.1; the layer itself is the standard top-k
routed MoE of Section 2, "Mixture-of-Experts and Expert Parallelism"):

1. router logits  z[t,e] = fl32( fl32(sum_h x[t,h] * w_router[e,h]) + b[e] )
2. top-k selection per token by (z descending, expert id ascending)
3. gate weights   w_j = p_j / sum_j' p_j',  p_j = exp(z_j - z_max) over the k
   selected logits (softmax over all E then renormalising over the k selected
   gives the same value: the full-softmax denominator cancels)
4. expert histogram counts[e] over all E experts: the per-layer activation
   profile, one row of the activation matrix W of Section 4.2.2
5. local offsets: exclusive prefix sum of counts over the local slots; their
   total is the GPU's token load n_g = sum_{e in S_g} w_e of Section 4.2.3
6. stable permutation of the flat assignment index i = t*k + j by local slot
7. per local expert: h = bf16( silu(G) * U ), G = X W_gate^T, U = X W_up^T
   (fp32 accumulation, silu(g) = g * 1/(1+exp(-g)) in fp32), then
   y = bf16( fp32(h W_down^T) )
8. combine: out[t] = bf16( sum_{j ascending, assignment local} w[t,j] y[dest] )
   with an fp32 accumulator; rows with no local assignment are exactly 0.

Precision: fp32 accumulation, bf16 round-to-nearest-even at inputs, h, y and
out (bf16 configs); the fp32 config rounds nothing. ``acc="f64"`` accumulates
the three matmuls in fp64 (then rounds to fp32) with identical rounding points,
which measures how much two correct accumulation orders disagree.

The oracle is written from the definition above, loops per expert and per
assignment, and shares no code with the HIP path or with ``synth``.
"""
from __future__ import annotations

import numpy as np

F32 = np.float32


# --------------------------------------------------------------------------
# bf16 rounding (round to nearest, ties to even) of float32 values.
# --------------------------------------------------------------------------
def bf16_rne(a) -> np.ndarray:
    """Round float32 values to bf16 precision (RNE), returned as float32.

    bf16 keeps the top 16 bits of the IEEE binary32 pattern; rounding adds
    0x7FFF plus the lowest kept bit before truncating the low 16 bits. NaN is
    kept as a quiet NaN.
    """
    a = np.ascontiguousarray(a, dtype=F32)
    bits = a.view(np.uint32).astype(np.uint64)
    keep_lsb = (bits >> 16) & 1
    rounded = ((bits + 0x7FFF + keep_lsb) & 0xFFFF0000).astype(np.uint32)
    out = rounded.view(F32).copy()
    nan = np.isnan(a)
    if nan.any():
        out[nan] = np.nan
    return out


# --------------------------------------------------------------------------
# Steps 1-3: gating.
# --------------------------------------------------------------------------
def router_logits(x, w_router, bias) -> np.ndarray:
    """z[t,e] = fl32(fl32(x[t,:] . w_router[e,:]) + bias[e]), shape [T,E]."""
    x = np.asarray(x, F32)
    w = np.asarray(w_router, F32)
    acc = np.matmul(x, w.T).astype(F32)
    return (acc + np.asarray(bias, F32)[None, :]).astype(F32)


def topk_select(z, k: int) -> np.ndarray:
    """ids[t, 0..k-1]: experts ordered by (z descending, expert id ascending)."""
    z = np.asarray(z, F32)
    # A stable ascending sort of -z keeps equal logits in expert-id order.
    order = np.argsort(-z.astype(np.float64), axis=1, kind="stable")
    return order[:, :k].astype(np.int32)


def topk_weights(z, ids) -> np.ndarray:
    """w[t,j] = exp(z_j - z_0) / sum_j' exp(z_j' - z_0) in fp32, j ascending."""
    z = np.asarray(z, F32)
    zs = np.take_along_axis(z, np.asarray(ids, np.int64), axis=1).astype(F32)
    p = np.exp((zs - zs[:, :1]).astype(F32)).astype(F32)
    s = np.zeros(zs.shape[0], F32)
    for j in range(zs.shape[1]):
        s = (s + p[:, j]).astype(F32)
    return (p / s[:, None]).astype(F32)


# --------------------------------------------------------------------------
# Steps 4-6: activation profile, offsets, permutation.
# --------------------------------------------------------------------------
def expert_histogram(ids, E: int) -> np.ndarray:
    """counts[e] = number of (t, j) with ids[t, j] == e, for all E experts."""
    counts = np.zeros(E, np.int64)
    for e in np.asarray(ids).ravel():
        counts[int(e)] += 1
    return counts.astype(np.int32)


def local_experts_of(expert_map) -> np.ndarray:
    """Global expert id of each local slot (slot order)."""
    expert_map = np.asarray(expert_map)
    n_local = int((expert_map >= 0).sum())
    local = np.full(n_local, -1, np.int64)
    for e, slot in enumerate(expert_map):
        if slot >= 0:
            local[int(slot)] = e
    return local


def local_offsets(counts, expert_map) -> np.ndarray:
    """offsets[0] = 0, offsets[l+1] = offsets[l] + counts[expert in slot l]."""
    local = local_experts_of(expert_map)
    off = np.zeros(len(local) + 1, np.int64)
    for slot, e in enumerate(local):
        off[slot + 1] = off[slot] + int(counts[e])
    return off.astype(np.int32)


def permute(x, ids, expert_map, offsets):
    """Stable counting sort of flat assignments i = t*k + j by local slot.

    Returns x_perm [M_loc, H], perm_src [M_loc] (flat index i of each row) and
    dest [T*k] (row of assignment i, or -1 when its expert is remote).
    """
    ids = np.asarray(ids)
    T, k = ids.shape
    expert_map = np.asarray(expert_map)
    offsets = np.asarray(offsets, np.int64)
    m_loc = int(offsets[-1])
    cursor = offsets[:-1].copy()
    perm_src = np.full(m_loc, -1, np.int64)
    dest = np.full(T * k, -1, np.int64)
    flat = ids.ravel()
    for i in range(T * k):
        slot = int(expert_map[int(flat[i])])
        if slot < 0:
            continue
        pos = int(cursor[slot])
        cursor[slot] += 1
        perm_src[pos] = i
        dest[i] = pos
    x_perm = np.asarray(x, F32)[perm_src // k] if m_loc else np.zeros((0, np.shape(x)[1]), F32)
    return x_perm, perm_src.astype(np.int32), dest.astype(np.int32)


# --------------------------------------------------------------------------
# Step 7: grouped SwiGLU expert FFN.
# --------------------------------------------------------------------------
def _matmul_t(a, b, acc: str) -> np.ndarray:
    """a @ b.T with fp32 (BLAS sgemm) or fp64 accumulation, result in fp32."""
    if acc == "f32":
        return np.matmul(np.asarray(a, F32), np.asarray(b, F32).T).astype(F32)
    if acc == "f64":
        return np.matmul(np.asarray(a, np.float64), np.asarray(b, np.float64).T).astype(F32)
    raise ValueError(acc)


def swiglu_rows(X, w_gate, w_up, w_down, bf16: bool, acc: str = "f32"):
    """One expert on rows X [M,H]: returns (h [M,I], y [M,H]) in fp32 arrays."""
    G = _matmul_t(X, w_gate, acc)
    U = _matmul_t(X, w_up, acc)
    with np.errstate(over="ignore"):
        sig = (F32(1.0) / (F32(1.0) + np.exp(-G))).astype(F32)
    h = ((G * sig).astype(F32) * U).astype(F32)
    if bf16:
        h = bf16_rne(h)
    y = _matmul_t(h, w_down, acc)
    if bf16:
        y = bf16_rne(y)
    return h, y


def grouped_swiglu_ffn(x_perm, w_gate, w_up, w_down, offsets, bf16: bool,
                       acc: str = "f32"):
    """Per local expert l, rows [offsets[l], offsets[l+1]) of x_perm.

    Returns (h [M_loc, I], y_perm [M_loc, H]). Experts with no rows are skipped.
    """
    offsets = np.asarray(offsets, np.int64)
    m_loc = int(offsets[-1])
    I = np.shape(w_gate)[1]
    H = np.shape(w_gate)[2]
    h_all = np.zeros((m_loc, I), F32)
    y_all = np.zeros((m_loc, H), F32)
    for slot in range(len(offsets) - 1):
        r0, r1 = int(offsets[slot]), int(offsets[slot + 1])
        if r1 == r0:
            continue
        h, y = swiglu_rows(np.asarray(x_perm)[r0:r1], w_gate[slot], w_up[slot],
                           w_down[slot], bf16, acc)
        h_all[r0:r1] = h
        y_all[r0:r1] = y
    return h_all, y_all


# --------------------------------------------------------------------------
# Step 8: combine.
# --------------------------------------------------------------------------
def unpermute_combine(y_perm, w, dest, T: int, k: int, bf16: bool) -> np.ndarray:
    """out[t] = sum over ascending j with dest >= 0 of w[t,j] * y_perm[dest]."""
    y_perm = np.asarray(y_perm, F32)
    H = y_perm.shape[1]
    dest = np.asarray(dest, np.int64).reshape(T, k)
    w = np.asarray(w, F32).reshape(T, k)
    out = np.zeros((T, H), F32)
    for j in range(k):
        d = dest[:, j]
        m = d >= 0
        if m.any():
            out[m] = (out[m] + (w[m, j][:, None] * y_perm[d[m]]).astype(F32)).astype(F32)
    return bf16_rne(out) if bf16 else out


# --------------------------------------------------------------------------
# The whole layer, and the per-token form used to sample full-size outputs.
# --------------------------------------------------------------------------
def moe_layer(x, w_router, bias, k, expert_map, w_gate, w_up, w_down,
              bf16: bool, acc: str = "f32") -> dict:
    """All steps in order; returns every intermediate by name."""
    z = router_logits(x, w_router, bias)
    ids = topk_select(z, k)
    w = topk_weights(z, ids)
    counts = expert_histogram(ids, z.shape[1])
    offsets = local_offsets(counts, expert_map)
    x_perm, perm_src, dest = permute(x, ids, expert_map, offsets)
    h, y_perm = grouped_swiglu_ffn(x_perm, w_gate, w_up, w_down, offsets, bf16, acc)
    out = unpermute_combine(y_perm, w, dest, np.shape(x)[0], k, bf16)
    return dict(logits=z, ids=ids, weights=w, counts=counts, offsets=offsets,
                x_perm=x_perm, perm_src=perm_src, dest=dest, h=h, y_perm=y_perm,
                out=out)


def moe_layer_rows(x, w_router, bias, k, expert_map, w_gate, w_up, w_down,
                   bf16: bool, rows) -> dict:
    """Outputs of the layer for the selected tokens only (definition per token).

    Routing and FFN rows are independent per token, so each sampled token is
    routed on its own and sent through its local experts; tokens that share an
    expert are stacked into one matmul for speed.
    """
    rows = np.asarray(rows, np.int64)
    xr = np.asarray(x, F32)[rows]
    z = router_logits(xr, w_router, bias)
    ids = topk_select(z, k)
    w = topk_weights(z, ids)
    H = xr.shape[1]
    n = len(rows)
    y = np.zeros((n, k, H), F32)
    local = np.full((n, k), False)
    local_ids = local_experts_of(expert_map)
    for slot, e in enumerate(local_ids):
        sel = np.argwhere(ids == e)
        if len(sel) == 0:
            continue
        _, ys = swiglu_rows(xr[sel[:, 0]], w_gate[slot], w_up[slot], w_down[slot], bf16)
        y[sel[:, 0], sel[:, 1]] = ys
        local[sel[:, 0], sel[:, 1]] = True
    out = np.zeros((n, H), F32)
    abs_terms = np.zeros((n, H))
    for j in range(k):
        m = local[:, j]
        out[m] = (out[m] + (w[m, j][:, None] * y[m, j]).astype(F32)).astype(F32)
        abs_terms[m] += np.abs(w[m, j].astype(np.float64))[:, None] * np.abs(y[m, j].astype(np.float64))
    if bf16:
        out = bf16_rne(out)
    # abs_terms = sum_j |w_j y_j|: the magnitude of what was summed into out
    return dict(logits=z, ids=ids, weights=w, out=out, abs_terms=abs_terms)
