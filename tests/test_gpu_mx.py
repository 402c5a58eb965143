"""GPU parity of the MXFP8 expert FFN (quantiser, gate/up, down, whole FFN)
against the MXFP8 oracle, through the C ABI.

Rules (fixed before any GPU run):
* quantisation (codes and scale codes): bit-exact.
* GEMM outputs: each product of two E4M3 codes and their power-of-two
  scales is exact in fp32, so an output differs from the exact sum only by
  its fp32 summation, in whatever order the hardware and the split schedule
  take: K - 1 additions, each rounded to nearest (or kept exact) with a
  relative error of at most 2^-24, bound the error by about (K - 1) 2^-24 sum |a_i b_i| (the standard
  recursive-summation bound), 2^-10.2 sum |a_i b_i| at the largest K here
  (14336). Each output may therefore differ from the fp64 result by
  MFMA_F8_REL = 2^-10 of sum |a_i b_i|, plus one bf16 rounding on each side.
* h (quantised in the gate/up epilogue from fp32 G, U that differ from the
  oracle's within the rule above): the scale code of each block must be one
  the oracle allows for some h within the error bound of its block, and each
  code must lie between the codes of h - bound and h + bound under that
  scale (quantisation at a fixed scale is monotone). The whole FFN then
  allows y the effect of every such code difference on top of the GEMM rule.

Inputs: each side quantises the same seeded synthetic values with its own
code; the tests first check that the codes agree bit for bit.
"""
import dataclasses

import numpy as np
import pytest
import torch

import paper_2606_00735_amd as moe
from oracle import mx_oracle as X
from oracle import moe_oracle as O
from synth import CONFIGS, make_layer
from synth.moe_inputs import make_experts, make_router

pytestmark = pytest.mark.gpu
DEV = "cuda"
MFMA_F8_REL = 2.0 ** -10


def banner(*a):
    print("CASE", *a, flush=True)


def up(a, dtype=torch.bfloat16):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(DEV).to(dtype).contiguous()


def gpu_scales(scales, R, K):
    """Scale dwords [.., K/128, R] -> E8M0 codes [.., R, K/32] (the oracle's layout)."""
    s = scales.cpu().numpy().view(np.uint8)
    s = s.reshape(s.shape[:-2] + (K // 128, R, 4))
    s = np.swapaxes(s, -3, -2)
    return np.ascontiguousarray(s.reshape(s.shape[:-3] + (R, K // 32)))


def oracle_quant(a, chunk=256):
    """Row-chunked oracle quantisation (the MX blocks lie within rows)."""
    a = np.asarray(a)
    q = np.empty(a.shape, np.uint8)
    s = np.empty(a.shape[:-1] + (a.shape[-1] // 32,), np.uint8)
    flat_a, flat_q, flat_s = a.reshape(-1, a.shape[-1]), q.reshape(-1, a.shape[-1]), s.reshape(-1, s.shape[-1])
    for r in range(0, flat_a.shape[0], chunk):
        flat_q[r:r + chunk], flat_s[r:r + chunk] = X.mx_quantize(flat_a[r:r + chunk])
    return q, s


def check_quant(t, a, what):
    """GPU MxTensor t == oracle quantisation of a, bit for bit. Returns the oracle's (codes, scales)."""
    torch.cuda.synchronize()
    K = a.shape[-1]
    R = a.shape[-2]
    q, s = oracle_quant(a)
    gq = t.codes.cpu().numpy()
    gs = gpu_scales(t.scales, R, K)
    bad_s = gs != s
    assert not bad_s.any(), f"{what}: {bad_s.sum()} scale codes differ, first at {np.argwhere(bad_s)[0]}"
    bad = gq != q
    if bad.any():
        i = tuple(np.argwhere(bad)[0])
        raise AssertionError(f"{what}: {bad.sum()} codes differ; first {i}: value {a[i]!r} "
                             f"gpu {gq[i]:#04x} oracle {q[i]:#04x}")
    return q, s


def check_gemm(got, ref, mag, what, extra=0.0):
    """GEMM rule; `extra` is a further allowance per element (h code differences)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert np.all(np.isfinite(got)), what
    tol = MFMA_F8_REL * mag + extra + 2.0 ** -7 * np.maximum(np.abs(ref), np.abs(got)) + 1e-30
    err = np.abs(got - ref)
    bad = err > tol
    if bad.any():
        i = tuple(np.argwhere(bad)[0])
        raise AssertionError(f"{what}: {bad.sum()} of {bad.size} outside; first {i}: gpu {got[i]} "
                             f"oracle {ref[i]} mag {mag[i]} tol {tol[i]}")
    rel = float(np.max(err / np.maximum(mag, 1e-30)))
    print(f"  {what}: max |err|/mag = {rel:.2e}", flush=True)


def h_bounds(P, h32):
    """Per-element bound on |h_gpu - h_oracle| before quantisation."""
    G, U = P["G"], P["U"]
    dG = MFMA_F8_REL * P["magG"] + 2.0 ** -23 * np.abs(G)
    dU = MFMA_F8_REL * P["magU"] + 2.0 ** -23 * np.abs(U)
    with np.errstate(over="ignore"):
        silu = G / (1.0 + np.exp(-G))
    return 1.1 * dG * (np.abs(U) + dU) + np.abs(silu) * dU + 2.0 ** -20 * np.abs(h32.astype(np.float64)) + 1e-38


def q_at(v, code):
    """Dequantised value of v quantised at scale code `code` (per element)."""
    sc = np.exp2(code.astype(np.float64) - 127.0)
    return X.e4m3_decode(X.e4m3_encode(np.clip(v / sc, -X.E4M3_MAX, X.E4M3_MAX))) * sc


def scale_code(amax):
    _, ex = np.frexp(np.where(amax > 0, amax, 1.0))
    return np.where(amax > 0, ex - 1.0 - 8.0, -127.0).clip(-127.0, 127.0) + 127.0


def allowed_h(h32, P):
    """Interval [lo, hi] around the oracle's h that holds the GPU's h before
    quantisation, and the range [s_lo, s_hi] of block scale codes it allows."""
    m, I = h32.shape
    tol = h_bounds(P, h32)
    h = h32.astype(np.float64)
    lo, hi = h - tol, h + tol
    blk = lambda a: a.reshape(m, I // 32, 32)
    mag_lo = np.where((lo > 0) | (hi < 0), np.minimum(np.abs(lo), np.abs(hi)), 0.0)
    s_lo = scale_code(blk(mag_lo).max(-1))
    s_hi = scale_code(blk(np.maximum(np.abs(lo), np.abs(hi))).max(-1))
    return lo, hi, s_lo, s_hi


def h_deviation(lo, hi, s_lo, s_hi, hq, hs):
    """Largest |dequantised h_gpu - oracle Hd| any allowed code can give."""
    Hd = X.mx_dequantize(hq, hs)
    dev = np.zeros_like(Hd)
    for s in (s_lo, s_hi):
        sc = np.repeat(s, 32, axis=1)
        dev = np.maximum(dev, np.maximum(np.abs(q_at(lo, sc) - Hd), np.abs(q_at(hi, sc) - Hd)))
    return dev


def check_h(ghq, ghs, hq, hs, h32, P, what):
    """The h rule of the module docstring. Returns per-element |h_gpu - Hd| bound (fp64)."""
    lo, hi, s_lo, s_hi = allowed_h(h32, P)
    gs = ghs.astype(np.float64)
    assert np.all((gs >= s_lo) & (gs <= s_hi)), f"{what}: scale codes outside the allowed range"
    gsc = np.repeat(gs, 32, axis=1)
    gv = X.mx_dequantize(ghq, ghs)
    qlo, qhi = q_at(lo, gsc), q_at(hi, gsc)
    bad = (gv < qlo) | (gv > qhi)
    assert not bad.any(), f"{what}: {bad.sum()} h codes outside the bound"
    diff = float(np.mean(ghq != hq))
    print(f"  {what}: {diff:.2e} of h codes differ from the oracle's (all within the bound), "
          f"{float(np.mean(ghs != hs)):.1e} of scales", flush=True)
    assert diff < 0.02
    return h_deviation(lo, hi, s_lo, s_hi, hq, hs)


# ---------------------------------------------------------------- quantiser
def all_bf16_values():
    u = np.arange(65536, dtype=np.uint32)
    u = u[((u >> 7) & 0xFF) != 0xFF]           # finite values only: 65024 of them
    return (u << 16).view(np.float32)


def test_quantize_every_bf16_value():
    banner("mx quantize: every finite bf16 value, sorted and shuffled blocks")
    v = all_bf16_values()
    for name, arr in (("sorted", v), ("shuffled", np.random.default_rng(0).permutation(v))):
        a = arr.reshape(-1, 256)
        t = moe.moe_mx_quantize(up(a))
        check_quant(t, a, f"bf16 {name}")


def test_quantize_f32_ties_clamp_and_zeros():
    banner("mx quantize fp32: ties, clamp band, zeros, tiny blocks")
    rng = np.random.default_rng(1)
    R, K = 96, 384
    a = (rng.standard_normal((R, K)) * np.exp2(rng.integers(-30, 30, (R, 1)))).astype(np.float32)
    vals = X.e4m3_decode(np.arange(1, 127))
    mids = ((vals[:-1] + vals[1:]) / 2)
    for r in range(0, 32):                      # exact ties after scaling: blocks with amax 448 * 2^s
        s = float(r - 10)
        blk = rng.choice(mids, 31) * rng.choice([-1, 1], 31)
        a[r, :32] = np.concatenate([[448.0], blk]).astype(np.float64) * 2.0 ** s
    a[32, :] = 0.0
    a[33, :64] = -0.0
    a[34, :32] = np.float32(2.0 ** -140)         # fp32 denormals
    a[35, :32] = 1.9 * 2.0 ** np.arange(32)[::-1] / 2.0 ** 20   # amax mantissa 1.9: the clamp band
    a[36, :32] = -(2.0 ** -10) * rng.random(32)  # tiny negatives: signed zeros
    t = moe.moe_mx_quantize(up(a, torch.float32))
    check_quant(t, a, "f32")


def test_quantize_batched_weights_layout():
    banner("mx quantize batched [3, 256, 384]")
    a = np.random.default_rng(2).standard_normal((3, 256, 384)).astype(np.float32)
    a = (torch.from_numpy(a).bfloat16().float()).numpy()
    t = moe.moe_mx_quantize(up(a))
    assert tuple(t.scales.shape) == (3, 3, 256)
    check_quant(t, a, "batched")


def test_quantize_device_row_count():
    """With a device row count only the first rows are quantised; the rest of
    the output keeps what it held."""
    banner("mx quantize with a device row count")
    a = (torch.from_numpy(np.random.default_rng(3).standard_normal((300, 256)).astype(np.float32))
         .bfloat16().float().numpy())
    out = moe.MxTensor(torch.full((300, 256), 0x5A, dtype=torch.uint8, device=DEV),
                       torch.full((2, 300), 0x11111111, dtype=torch.int32, device=DEV))
    n = torch.tensor([171], dtype=torch.int32, device=DEV)
    moe.moe_mx_quantize(up(a), out=out, row_count=n)
    torch.cuda.synchronize()
    check_quant(_Sub(out, np.arange(171)), a[:171], "first rows")
    assert torch.all(out.codes[171:] == 0x5A) and torch.all(out.scales[:, 171:] == 0x11111111)


# ---------------------------------------------------------------- GEMMs
def _shape(H, I, n):
    return dataclasses.replace(CONFIGS["qwen3"], name="mx", H=H, I=I, E=n, k=1, E_local=n)


def _inputs(H, I, rows, seed, pad=3):
    shape = _shape(H, I, len(rows))
    wg, wu, wd = make_experts(shape, list(range(len(rows))), seed=seed)
    m = sum(rows)
    x, *_ = make_router(shape, max(m, 1), 0.0, seed=seed)
    M_cap = m + pad
    xp = np.zeros((M_cap, H), np.float32)
    xp[:m] = x[:m]
    offsets = np.concatenate([[0], np.cumsum(rows)]).astype(np.int32)
    return xp, wg, wu, wd, offsets, m


GEMM_CASES = [
    # (N, K, rows per expert): ragged tails of every tile class, empty experts
    (768, 2048, [300, 0, 1, 65, 129]),
    (2048, 7168, [40, 257]),
    (1024, 512, [8192]),          # 32 row tiles x 8 column tiles
    (4096, 512, [8192]),          # >= 4 tiles per CU: 256-column tiles
]


@pytest.mark.parametrize("N,K,rows", GEMM_CASES, ids=[f"N{n}-K{k}-rows{'_'.join(map(str, r))}"
                                                     for n, k, r in GEMM_CASES])
def test_grouped_gemm_mx(N, K, rows):
    banner("mx gemm", N, K, rows, "seed 7")
    _, _, b = make_experts(_shape(N, K, len(rows)), list(range(len(rows))), seed=7)   # [E, N, K]
    m = sum(rows)
    offsets = np.concatenate([[0], np.cumsum(rows)]).astype(np.int32)
    xa, *_ = make_router(_shape(K, N, len(rows)), max(m, 1), 0.0, seed=8)             # rows of K
    a = np.zeros((m + 3, K), np.float32)
    a[:m] = xa[:m]
    ta, tb = moe.moe_mx_quantize(up(a)), moe.moe_mx_quantize(up(b))
    aq, as_ = check_quant(ta, a, "a")
    bq, bs = check_quant(tb, b, "b")
    c = moe.moe_grouped_gemm_mx(ta, tb, torch.from_numpy(offsets).to(DEV))
    torch.cuda.synchronize()
    got = c.float().cpu().numpy()[:m]
    sample = np.arange(m) if m <= 2048 else np.random.default_rng(0).choice(m, 512, replace=False)
    ad = X.mx_dequantize(aq[sample], as_[sample])
    eid = np.searchsorted(offsets, sample, side="right") - 1
    ref = np.zeros((len(sample), N))
    mag = np.zeros((len(sample), N))
    for e in np.unique(eid):
        sel = eid == e
        bd = X.mx_dequantize(bq[e], bs[e])
        ref[sel] = ad[sel] @ bd.T
        mag[sel] = np.abs(ad[sel]) @ np.abs(bd).T
    ref = O.bf16_rne(ref.astype(np.float32))
    check_gemm(got[sample], ref, mag, f"gemm N={N} K={K}")


FFN_CASES = [
    (2048, 768, [300, 0, 1, 65, 129]),
    (7168, 2048, [40, 257]),
    (1024, 1024, [600, 5]),
]


def _ffn_case(H, I, rows, seed, rerun=False):
    """The MXFP8 FFN on one case under the rules of the module docstring
    (rerun: a second call must be bitwise equal). Returns the FFN's workspace."""
    xp, wg, wu, wd, offsets, m = _inputs(H, I, rows, seed=seed)
    tx = moe.moe_mx_quantize(up(xp))
    tg, tu, td = (moe.moe_mx_quantize(up(w)) for w in (wg, wu, wd))
    xq, xs = check_quant(tx, xp, "x")
    (gq, gs), (uq, us), (dq, ds) = (check_quant(t, w, n) for t, w, n in ((tg, wg, "wg"), (tu, wu, "wu"),
                                                                         (td, wd, "wd")))
    doff = torch.from_numpy(offsets).to(DEV)
    y, ws = moe.moe_grouped_swiglu_ffn_mx(tx, tg, tu, td, doff)
    torch.cuda.synchronize()
    M_cap = xp.shape[0]
    wsn = ws.cpu().numpy()
    hq_off = moe.FFN_COUNTER_BYTES
    hs_off = hq_off + ((M_cap * I + 255) // 256) * 256
    ghq = wsn[hq_off:hq_off + M_cap * I].reshape(M_cap, I)[:m]
    assert not wsn[:hq_off].any(), "the workspace's counters must be left zero"
    ghs_dw = torch.from_numpy(wsn[hs_off:hs_off + (I // 128) * M_cap * 4].view(np.int32).reshape(I // 128, M_cap))
    ghs = gpu_scales(ghs_dw, M_cap, I)[:m]
    hq, hs, h32, y_ref, mag, P = X.grouped_swiglu_ffn_mx(xq[:m], xs[:m], gq, gs, uq, us, dq, ds, offsets, parts=True)
    dev = check_h(ghq, ghs, hq, hs, h32, P, f"h H={H} I={I}")
    got = y.float().cpu().numpy()[:m]
    # y: GEMM rule on the oracle's h, plus the effect of every allowed h code difference
    allow = np.zeros_like(mag)
    for e in range(len(rows)):
        r0, r1 = offsets[e], offsets[e + 1]
        if r1 > r0:
            Wd = np.abs(X.mx_dequantize(dq[e], ds[e]))
            allow[r0:r1] = dev[r0:r1] @ Wd.T
    # the GPU's down GEMM sums |h_gpu| |W_down| <= mag + allow
    check_gemm(got, y_ref, mag + allow, f"ffn y H={H} I={I}", extra=allow)
    if rerun:
        y2, _ = moe.moe_grouped_swiglu_ffn_mx(tx, tg, tu, td, doff)
        torch.cuda.synchronize()
        assert torch.equal(y2[:m], y[:m]), "a second call differs"
    # the gate/up entry point alone writes the same h
    h = moe.moe_grouped_swiglu_mx(tx, tg, tu, doff)
    torch.cuda.synchronize()
    same = np.array_equal(h.codes.cpu().numpy()[:m], ghq)
    return ws, M_cap, same


@pytest.mark.parametrize("H,I,rows", FFN_CASES, ids=[f"H{h}-I{i}-rows{'_'.join(map(str, r))}"
                                                   for h, i, r in FFN_CASES])
def test_ffn_mx(H, I, rows):
    banner("mx ffn", H, I, rows, "seed 9")
    _, _, same = _ffn_case(H, I, rows, seed=9)
    assert same, "moe_grouped_swiglu_mx and the FFN's h differ"


MX_DECODE_CASES = [
    # the decode schedule (equal shares of (tile, K chunk) units per CU,
    # split tiles finished inside the GEMMs) when no expert exceeds 16 rows,
    # or 64 rows when no reduction launch follows (M_cap at most 128), or 128
    # rows in launches with no more tiles than half the CUs
    (4096, 14336, [9, 3, 0, 11]),     # Mixtral-shaped experts, M_cap 26
    (7168, 2048, [1, 16, 16]),        # DSV3-shaped experts, M_cap 36
    (2048, 768, [3, 0, 7, 1]),        # Qwen3-shaped experts, M_cap 14
    (4096, 2048, [20, 30]),           # 30 rows, M_cap 53
    (4096, 2048, [20, 30, 40]),       # 40 rows, M_cap 93, 48 gate/up and 96 down tiles: decode
    (4096, 2048, [100, 30, 120]),     # 120 rows, M_cap 253, tile-starved: decode
]


@pytest.mark.parametrize("H,I,rows", MX_DECODE_CASES, ids=[f"H{h}-I{i}-rows{'_'.join(map(str, r))}"
                                                           for h, i, r in MX_DECODE_CASES])
def test_ffn_mx_decode_schedule(H, I, rows):
    """The rules of the module docstring, a bitwise rerun, and the plan
    showing that nothing was left for a reduction launch."""
    banner("mx ffn decode schedule", H, I, rows, "seed 13")
    ws, M_cap, _ = _ffn_case(H, I, rows, seed=13, rerun=True)
    hs_off = moe.FFN_COUNTER_BYTES + ((M_cap * I + 255) // 256) * 256
    plan_off = hs_off + (((I // 128) * M_cap * 4 + 255) // 256) * 256
    got = ws[plan_off:plan_off + 12].view(torch.int32).cpu().numpy()
    assert got[0] == 1 and got[2] == 1, got  # every case here takes the decode schedule


MX_SPLIT_CASES = [
    # (H, I, rows per expert, S of the down GEMM), worked out by hand from the
    # split rule on 256 CUs (K chunks of 128): Mixtral-shaped experts of up to
    # 40 rows, M_cap 134, 192 down tiles (down S = 4 over 112 chunks); one 256-row
    # DSV3-shaped expert (gate/up S = 7, down S = 2: partial bytes equal to the
    # weight bytes are still allowed); Qwen3-shaped, 5 rows (decode schedule);
    # Maverick-shaped experts of 400, 100 and 32 rows (down S = 3)
    (4096, 14336, [40, 7, 0, 19, 30, 25, 10], 4),
    (7168, 2048, [256], 2),
    (2048, 768, [5], 1),
    (5120, 8192, [400, 100, 32], 3),
]


@pytest.mark.parametrize("H,I,rows,S_down", MX_SPLIT_CASES,
                         ids=[f"H{h}-I{i}-rows{'_'.join(map(str, r))}" for h, i, r, _ in MX_SPLIT_CASES])
def test_ffn_mx_split_k(H, I, rows, S_down):
    banner("mx ffn split-K", H, I, rows, "seed 5")
    ws, M_cap, _ = _ffn_case(H, I, rows, seed=5)
    hs_off = moe.FFN_COUNTER_BYTES + ((M_cap * I + 255) // 256) * 256
    plan_off = hs_off + (((I // 128) * M_cap * 4 + 255) // 256) * 256
    assert int(ws[plan_off:plan_off + 4].view(torch.int32).item()) == S_down


MX_TAIL_CASES = [
    # (H, I, rows of one expert, (S, St, rem, cols) of the down GEMM) from the
    # tail rule on 256 CUs with K chunks of 128: St is held to 2 by K = 16 chunks
    (2048, 2048, [4608], (1, 2, 32, 128)),
    (4096, 2048, [8448], (1, 2, 16, 256)),
]


@pytest.mark.parametrize("H,I,rows,plan", MX_TAIL_CASES,
                         ids=[f"H{h}-I{i}-rows{r[0]}" for h, i, r, _ in MX_TAIL_CASES])
def test_ffn_mx_tail_split(H, I, rows, plan):
    banner("mx ffn tail split", H, I, rows, "seed 4")
    ws, M_cap, _ = _ffn_case(H, I, rows, seed=4, rerun=True)
    hs_off = moe.FFN_COUNTER_BYTES + ((M_cap * I + 255) // 256) * 256
    plan_off = hs_off + (((I // 128) * M_cap * 4 + 255) // 256) * 256
    got = ws[plan_off:plan_off + 20].view(torch.int32).cpu().numpy()
    assert (got[0], got[2], got[3], got[4]) == plan, got[:5]


def test_load_sweep_mx_output_and_timing():
    """The MXFP8 sweep's last run leaves y for the largest M (rows checked
    under the FFN rule) and every median is positive."""
    banner("mx sweep qwen3-shaped expert")
    H, I = 2048, 768
    _, wg, wu, wd, _, _ = _inputs(H, I, [1], seed=12)
    x, *_ = make_router(_shape(H, I, 1), 300, 0.0, seed=12)
    Ms = [1, 7, 33, 128, 300]
    rot = 3
    tx = moe.moe_mx_quantize(up(x))
    tg, tu, td = (moe.moe_mx_quantize(up(np.repeat(w, rot, 0))) for w in (wg, wu, wd))
    y = torch.full((300, H), float("nan"), dtype=torch.bfloat16, device=DEV)
    us, allus = moe.moe_load_sweep_mx(tx, tg, tu, td, Ms, warmup=2, iters=5, y_scratch=y, keep_all=True)
    print("  sweep us", us.tolist(), flush=True)
    assert np.all(us > 0) and allus.shape == (5, 5)
    xq, xs = check_quant(tx, x, "x")
    (gq, gs), (uq, us_), (dq, ds) = (oracle_quant(w) for w in (wg, wu, wd))
    hq, hs, h32, y_ref, mag, P = X.grouped_swiglu_ffn_mx(xq, xs, gq, gs, uq, us_, dq, ds, [0, 300], parts=True)
    dev = h_deviation(*allowed_h(h32, P), hq, hs)
    allow = dev @ np.abs(X.mx_dequantize(dq[0], ds[0])).T
    check_gemm(y.float().cpu().numpy(), y_ref, mag + allow, "sweep y", extra=allow)


def test_ffn_mx_rows_of_empty_experts_untouched():
    banner("mx ffn: rows past offsets[-1] are not written")
    xp, wg, wu, wd, offsets, m = _inputs(1024, 1024, [0, 70, 0], seed=11, pad=40)
    tx = moe.moe_mx_quantize(up(xp))
    tg, tu, td = (moe.moe_mx_quantize(up(w)) for w in (wg, wu, wd))
    y = torch.full((xp.shape[0], 1024), 7.0, dtype=torch.bfloat16, device=DEV)
    moe.moe_grouped_swiglu_ffn_mx(tx, tg, tu, td, torch.from_numpy(offsets).to(DEV), y_perm=y)
    torch.cuda.synchronize()
    assert torch.all(y[m:] == 7.0)
    assert torch.all(torch.isfinite(y[:m].float()))


# ---------------------------------------------------------------- full size
MX_FULL = [("mixtral", 4096, 1.0), ("qwen3", 8192, 1.0), ("dsv3_shard", 16384, 0.0), ("maverick_shard", 32768, 0.0)]


@pytest.mark.parametrize("name,T,alpha", MX_FULL, ids=[f"{n}-T{t}-a{a}" for n, t, a in MX_FULL])
def test_ffn_mx_fullsize(name, T, alpha):
    """Every bf16 workload at full size: routing from the oracle, the MXFP8
    FFN in the bench's launch configuration (x_perm of M_cap = T k rows),
    sampled rows of the hottest and the coldest local expert checked."""
    banner("mx ffn fullsize", name, T, alpha, "seed 0")
    li = make_layer(name, T, alpha, seed=0)
    H, I = li.shape.H, li.shape.I
    z = O.router_logits(li.x, li.w_router, li.bias)
    ids = O.topk_select(z, li.shape.k)
    counts = O.expert_histogram(ids, li.shape.E)
    offsets = O.local_offsets(counts, li.expert_map)
    x_perm, _, _ = O.permute(li.x, ids, li.expert_map, offsets)
    m = int(offsets[-1])
    M_cap = T * li.shape.k
    xp_full = np.zeros((M_cap, H), np.float32)
    xp_full[:m] = x_perm
    tx = moe.moe_mx_quantize(up(xp_full))
    # weight code rows padded to weight_row_stride: the padded path at full size
    tg, tu, td = (moe.moe_mx_quantize(up(w), ld=moe.weight_row_stride(w.shape[-1], 1))
                  for w in (li.w_gate, li.w_up, li.w_down))
    y, _ = moe.moe_grouped_swiglu_ffn_mx(tx, tg, tu, td, torch.from_numpy(offsets.astype(np.int32)).to(DEV))
    torch.cuda.synchronize()
    got = y.float().cpu().numpy()
    rows_e = np.diff(offsets)
    hot, cold = int(np.argmax(rows_e)), int(np.argmin(np.where(rows_e > 0, rows_e, 1 << 30)))
    print(f"  M_loc={m} rows per expert {rows_e.tolist()}", flush=True)
    for e in (hot, cold):
        r0, r1 = int(offsets[e]), int(offsets[e + 1])
        cand = np.unique(np.clip([r0, r0 + 1, r0 + 255, r0 + 256, (r0 + r1) // 2, r1 - 2, r1 - 1], r0, r1 - 1))
        print(f"  expert {e}: rows {cand.tolist()}: oracle quantisation of its weights", flush=True)
        xq, xs = check_quant(_Sub(tx, cand), x_perm[cand], f"x rows of expert {e}")
        wq = [check_quant(_Sub(t, e), w[e], f"{n}[{e}]")
              for t, w, n in ((tg, li.w_gate, "wg"), (tu, li.w_up, "wu"), (td, li.w_down, "wd"))]
        (gq, gs), (uq, us), (dq, ds) = wq
        print(f"  expert {e}: weights bit-exact; oracle FFN rows", flush=True)
        off1 = np.array([0, len(cand)], np.int32)
        hq, hs, h32, y_ref, mag, P = X.grouped_swiglu_ffn_mx(xq, xs, gq[None], gs[None], uq[None], us[None],
                                                             dq[None], ds[None], off1, parts=True)
        # the GPU's h is not checked here: allow every code the bound permits
        dev = h_deviation(*allowed_h(h32, P), hq, hs)
        allow = dev @ np.abs(X.mx_dequantize(dq, ds)).T
        check_gemm(got[cand], y_ref, mag + allow, f"fullsize y expert {e}", extra=allow)


class _Sub:
    """Rows (or one expert) of a GPU MxTensor, for check_quant."""

    def __init__(self, t, sel):
        if np.isscalar(sel):
            self.codes, self.scales = t.codes[sel], t.scales[sel]
        else:
            idx = torch.from_numpy(np.asarray(sel, np.int64)).to(DEV)
            self.codes = t.codes[idx]
            self.scales = t.scales[:, idx]


def _quant_padded(w, pad):
    """MXFP8 codes of weights [B, R, K] written into rows padded by `pad`
    bytes, the padding pre-filled with 0x7F (an E4M3 NaN: read, it would
    poison the output)."""
    B, R, K = w.shape
    codes = torch.full((B, R, K + pad), 0x7F, dtype=torch.uint8, device=DEV)[:, :, :K]
    scales = torch.empty((B, K // 128, R), dtype=torch.int32, device=DEV)
    return moe.moe_mx_quantize(up(w), out=moe.MxTensor(codes, scales))


MX_PAD_CASES = [
    # (H, I, rows per expert, pad of gate/up code rows, pad of down code rows)
    (4096, 1024, [1, 64, 0, 30], 128, 16),        # split-K in both GEMMs
    (1024, 1024, [257, 300, 321, 576, 1], 128, 128),
    (2048, 2048, [4608], 16, 128),                # tail split
]


@pytest.mark.parametrize("H,I,rows,pg,pd", MX_PAD_CASES, ids=["split", "ragged", "tail"])
def test_ffn_mx_padded_weight_rows(H, I, rows, pg, pd):
    """MXFP8 weights quantised into padded code rows: the same codes and
    scales as dense ones, the padding untouched, and the FFN, its gate/up
    half and the down GEMM give the dense operands' results bit for bit."""
    banner("mx ffn padded rows", H, I, rows, pg, pd, "seed 13")
    xp, wg, wu, wd, offsets, m = _inputs(H, I, rows, seed=13)
    doff = torch.from_numpy(offsets).to(DEV)
    tx = moe.moe_mx_quantize(up(xp))
    dense = [moe.moe_mx_quantize(up(w)) for w in (wg, wu, wd)]
    padded = [_quant_padded(wg, pg), _quant_padded(wu, pg), _quant_padded(wd, pd)]
    torch.cuda.synchronize()
    for d, p, pad in zip(dense, padded, (pg, pg, pd)):
        assert p.ld == d.ld + pad
        assert torch.equal(p.codes, d.codes) and torch.equal(p.scales, d.scales)
        assert bool((p.codes.as_strided((p.codes.shape[0], p.codes.shape[1], pad),
                                        p.codes.stride(), p.codes.shape[2]) == 0x7F).all()), "padding written"
    y1, _ = moe.moe_grouped_swiglu_ffn_mx(tx, *dense, doff)
    y2, _ = moe.moe_grouped_swiglu_ffn_mx(tx, *padded, doff)
    h1 = moe.moe_grouped_swiglu_mx(tx, dense[0], dense[1], doff)
    h2 = moe.moe_grouped_swiglu_mx(tx, padded[0], padded[1], doff)
    c1 = moe.moe_grouped_gemm_mx(h1, dense[2], doff)
    c2 = moe.moe_grouped_gemm_mx(h1, padded[2], doff)
    torch.cuda.synchronize()
    assert torch.equal(y2[:m], y1[:m]), "FFN output"
    assert torch.equal(h2.codes[:m], h1.codes[:m]) and torch.equal(h2.scales[:, :m], h1.scales[:, :m]), "h"
    assert torch.equal(c2[:m], c1[:m]), "down GEMM"
    assert bool(torch.isfinite(y2[:m].float()).all())


def test_load_sweep_mx_padded_weight_rows():
    """The MXFP8 sweep over weight copies with padded code rows leaves the
    same y as over dense copies."""
    banner("mx sweep padded rows")
    H, I = 2048, 768
    _, wg, wu, wd, _, _ = _inputs(H, I, [1], seed=12)
    x, *_ = make_router(_shape(H, I, 1), 96, 0.0, seed=12)
    tx = moe.moe_mx_quantize(up(x))
    rot = 3
    ys = []
    for pad in (0, 128):
        w = [_quant_padded(np.repeat(a, rot, 0), pad) for a in (wg, wu, wd)]
        y = torch.full((96, H), float("nan"), dtype=torch.bfloat16, device=DEV)
        moe.moe_load_sweep_mx(tx, *w, [1, 96], warmup=1, iters=2, y_scratch=y)
        ys.append(y)
    torch.cuda.synchronize()
    assert torch.equal(ys[0], ys[1])
