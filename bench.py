#!/usr/bin/env python3
"""Benchmark: one GPU's share of an expert-parallel MoE layer on MI355X.

    python bench.py [--steps K] [--warmup W] [--config mixtral --T 4096 --alpha 1.0]

A step is one pass of the whole layer -- top-k gating, expert histogram and
offsets, dispatch permutation, grouped SwiGLU FFN, weighted combine -- over
one batch of seeded synthetic tokens already resident in HBM. The default
workload is the Mixtral-8x7B-shaped layer (H=4096, I=14336, 8 experts all on
this GPU, top-2, bf16) at T=4096 tokens with rank-bias skew alpha=1.0.

Prints ONE JSON line: whole-layer throughput (algorithmic TFLOP/s), per-stage
HIP-event times, the roofline of the dominant step (the grouped SwiGLU FFN
call: two GEMM launches, each followed by its split-K reduction), a skew table, the per-expert latency-vs-load sweep,
and the CPU oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MoE layer µs + TFLOP/s / HBM GB/s (% roofline) on one GPU's expert shard vs skew"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3       # MI355X fp32 vector
PEAK_FP8_TFLOPS = 5000.0       # MI355X dense fp8 MFMA
PEAK_HBM_GBPS = 8000.0         # MI355X HBM3E
SWEEP_MS = [1, 2, 4, 8, 16, 32, 64, 128, 256, 512, 1024, 2048, 4096, 8192]
MALL_BYTES = 256 << 20


def parse():
    p = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--config", default="mixtral")
    p.add_argument("--T", type=int, default=4096)
    p.add_argument("--alpha", type=float, default=1.0)
    p.add_argument("--seed", type=int, default=0)
    p.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    p.add_argument("--no-extras", action="store_true", help="skip the skew table and load sweep")
    p.add_argument("--mx", action="store_true", help="time the MXFP8 FFN even with --no-extras")
    p.add_argument("--sweep-iters", type=int, default=10)
    p.add_argument("--cpu-seconds", type=float, default=12.0, help="target CPU oracle time")
    p.add_argument("--calib-copy-mib", type=int, default=0,
                   help="first run three device-to-device copies of this many MiB (a plain copy kernel of "
                        "known size, to calibrate HBM byte counters)")
    return p.parse_args()


def layer_work(shape, T, counts, local):
    """Algorithmic flops and HBM bytes of one layer pass and of its FFN step."""
    s = 2 if shape.dtype == "bf16" else 4
    H, I, E, k = shape.H, shape.I, shape.E, shape.k
    loc = [int(counts[e]) for e in local]
    m_loc = sum(loc)
    active = sum(1 for c in loc if c > 0)
    ffn_flops = 6.0 * H * I * m_loc
    router_flops = 2.0 * T * H * E
    w_bytes = 3.0 * H * I * s * active
    ffn_bytes = w_bytes + 2.0 * m_loc * H * s
    layer_bytes = w_bytes + 2.0 * T * H * s + H * E * s + 16.0 * T * k
    return dict(m_loc=m_loc, active=active, ffn_flops=ffn_flops, ffn_bytes=ffn_bytes,
                layer_flops=ffn_flops + router_flops, layer_bytes=layer_bytes)


def source_sha():
    h = hashlib.sha256()
    for f in ("ffn_kernels.hip", "common.hpp", "mx.hpp"):
        with open(os.path.join(ROOT, "paper_2606_00735_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_from_profile(workload_key):
    """HBM bytes per FFN call from committed rocprofv3 counters, if they were
    taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", "ffn_traffic.json")
    try:
        with open(path) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None
    ent = rec.get(workload_key)
    if not ent or ent.get("source_sha") != source_sha():
        return None
    return ent.get("bytes_per_call")


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU's share of the expert-parallel layer and runs on one GPU "
              "only (--gpus 1).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2606_00735_amd as moe
    from synth import CONFIGS, make_layer
    from synth.moe_inputs import make_experts, make_router

    if not torch.cuda.is_available():
        print("bench.py needs an MI355X GPU", file=sys.stderr)
        sys.exit(1)
    moe.load_library()
    dev = "cuda"
    shape = CONFIGS[args.config]
    dt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    T, k, H, I, E = args.T, shape.k, shape.H, shape.I, shape.E

    t_gen = time.time()
    li = make_layer(shape, T, args.alpha, seed=args.seed)

    def up(a, dtype=dt):
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(dtype).contiguous()

    x, wr, bias = up(li.x), up(li.w_router), up(li.bias, torch.float32)
    # expert weights in HBM with rows padded off multiples of 4 KiB
    # (moe.weight_row_stride), the layout the FFN streams fastest
    wg, wu, wd = (moe.pad_weight_rows(up(a)) for a in (li.w_gate, li.w_up, li.w_down))
    t_gen = time.time() - t_gen
    emap = li.expert_map
    E_local = len(li.local)

    def make_bufs(Tb, xb):
        b = {}
        moe.moe_layer(xb, wr, bias, k, emap, wg, wu, wd, bufs=b)
        return b

    # bf16: the FFN reads the routed rows of x itself (moe_grouped_swiglu_ffn_gather),
    # so the permute stage only computes positions
    fuse = dt == torch.bfloat16

    def run_timed(xb, bb, Tb, steps, warmup):
        """Warmup, then `steps` timed layer passes with per-stage HIP events."""
        names = ["gate_topk", "histogram_scan", "permute", "grouped_swiglu_ffn", "combine"]
        for _ in range(warmup):
            moe.moe_layer(xb, wr, bb["bias"], k, emap, wg, wu, wd, bufs=bb, fuse_gather=fuse)
        torch.cuda.synchronize()
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)] for _ in range(steps)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for s in range(steps):
            ev = evs[s]
            ev[0].record()
            ids, wts, _ = moe.moe_gate_topk(xb, wr, bb["bias"], k, ids=bb["ids"], weights=bb["weights"],
                                            ws=bb["gate_ws"])
            ev[1].record()
            counts, offsets, hws = moe.moe_expert_histogram_scan(ids, E, emap, ws=bb["hist_ws"],
                                                                 counts=bb["counts"], offsets=bb["offsets"])
            ev[2].record()
            xp, ps, dest = moe.moe_permute(xb, ids, emap, hws, x_perm=bb["x_perm"], perm_src=bb["perm_src"],
                                           dest=bb["dest"], gather=not fuse)
            ev[3].record()
            if fuse:
                yp, _ = moe.moe_grouped_swiglu_ffn_gather(xb, ps, k, wg, wu, wd, offsets, ws=bb["ffn_ws"],
                                                          y_perm=bb["y_perm"])
            else:
                yp, _ = moe.moe_grouped_swiglu_ffn(xp, wg, wu, wd, offsets, ws=bb["ffn_ws"], y_perm=bb["y_perm"])
            ev[4].record()
            moe.moe_unpermute_combine(yp, wts, dest, Tb, out=bb["out"])
            ev[5].record()
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        per = {n: np.array([evs[s][i].elapsed_time(evs[s][i + 1]) for s in range(steps)]) * 1e3
               for i, n in enumerate(names)}
        stage = {n: float(v.mean()) for n, v in per.items()}
        spread = {n: [round(float(np.percentile(v, q)), 2) for q in (10, 50, 90)] for n, v in per.items()}
        run_timed.spread = spread
        return (t1 - t0) * 1e3 / steps, stage

    if args.calib_copy_mib > 0:
        n = args.calib_copy_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    bufs = make_bufs(T, x)
    bufs["bias"] = bias
    ms, stage = run_timed(x, bufs, T, args.steps, args.warmup)
    counts = bufs["counts"].cpu().numpy()
    w = layer_work(shape, T, counts, li.local)
    us = ms * 1e3
    ffn_us = stage["grouped_swiglu_ffn"]
    peak_f = PEAK_BF16_TFLOPS if dt == torch.bfloat16 else PEAK_FP32_TFLOPS
    ffn_tflops = w["ffn_flops"] / (ffn_us * 1e-6) / 1e12
    ffn_gbps = w["ffn_bytes"] / (ffn_us * 1e-6) / 1e9
    mfma_bound = w["ffn_flops"] / (peak_f * 1e12) >= w["ffn_bytes"] / (PEAK_HBM_GBPS * 1e9)
    wkey = f"{args.config}-T{T}-a{args.alpha:g}-s{args.seed}"
    roofline = {
        "kernel": ("moe_grouped_swiglu_ffn_gather (gate/up GEMM reading the routed rows of x, down GEMM, "
                   "split-K reductions)" if fuse else "moe_grouped_swiglu_ffn (gate/up and down GEMMs + split-K reductions)"),
        "bound": "mfma" if mfma_bound else "hbm",
        "achieved": round(ffn_tflops if mfma_bound else ffn_gbps, 3),
        "peak": peak_f if mfma_bound else PEAK_HBM_GBPS,
        "unit": "TFLOP/s" if mfma_bound else "GB/s",
        "frac": round((ffn_tflops / peak_f) if mfma_bound else (ffn_gbps / PEAK_HBM_GBPS), 4),
        "traffic": traffic_from_profile(wkey),
        "algorithmic_flops": w["ffn_flops"],
        "algorithmic_bytes": w["ffn_bytes"],
        "avg_us": round(ffn_us, 2),
    }

    result = {
        "metric": METRIC,
        "value": round(w["layer_flops"] / (us * 1e-6) / 1e12, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if dt == torch.bfloat16 else "f32",
        "data": "synthetic (seeded; grid-quantised router inputs, rank-bias skew)",
        "config": {"workload": f"{args.config}-shaped MoE layer, {E_local}/{E} experts local, top-{k}, "
                               f"T={T}, alpha={args.alpha:g}",
                   "T": T, "H": H, "I": I, "E": E, "k": k, "E_local": E_local, "alpha": args.alpha,
                   "seed": args.seed, "M_loc": w["m_loc"], "active_local_experts": w["active"],
                   "weight_row_stride": {"gate_up": wg.stride(1), "down": wd.stride(1)}},
        "us_per_layer": round(us, 2),
        "layer_gbps": round(w["layer_bytes"] / (us * 1e-6) / 1e9, 1),
        "stages_us": {n: round(v, 2) for n, v in stage.items()},
        "stages_us_p10_p50_p90": run_timed.spread,
        "roofline": roofline,
        "gen_s": round(t_gen, 1),
    }

    # MXFP8 FFN on this batch's routed rows (before the skew table, which
    # reuses these buffers for its other token counts and skews)
    if (args.mx or not args.no_extras) and dt == torch.bfloat16:
        cases = [(T, args.alpha, bufs, stage["grouped_swiglu_ffn"])]
        for Tb, a in (((min(shape.Ts), 0.0),) if not args.no_extras else ()):
            if Tb != T:
                xs, _, bs, _ = make_router(shape, Tb, a, seed=args.seed)
                bb = make_bufs(Tb, up(xs))
                bb["bias"] = up(bs, torch.float32)
                _, st_b = run_timed(up(xs), bb, Tb, max(5, args.steps // 2), 3)
                cases.append((Tb, a, bb, st_b["grouped_swiglu_ffn"]))
        result["mx_ffn"] = mx_section(moe, torch, np, shape, li, wg, wu, wd, cases, args.steps,
                                      key=lambda Tb, a: f"{args.config}-T{Tb}-a{a:g}-s{args.seed}-mx")
    if not args.no_extras:
        # skew table: same weights, other token counts and skews of this config
        table = []
        for Tb in shape.Ts:
            for a in shape.alphas:
                xs, _, bs, _ = make_router(shape, Tb, a, seed=args.seed)
                xb = up(xs)
                bb = make_bufs(Tb, xb) if (Tb != T) else dict(bufs)
                bb["bias"] = up(bs, torch.float32)
                ms_b, st_b = run_timed(xb, bb, Tb, max(5, args.steps // 2), 3)
                wb = layer_work(shape, Tb, bb["counts"].cpu().numpy(), li.local)
                fu = st_b["grouped_swiglu_ffn"]
                table.append({"T": Tb, "alpha": a, "us_per_layer": round(ms_b * 1e3, 2),
                              "layer_tflops": round(wb["layer_flops"] / (ms_b * 1e-3) / 1e12, 2),
                              "ffn_us": round(fu, 2), "M_loc": wb["m_loc"], "active": wb["active"],
                              "ffn_tflops": round(wb["ffn_flops"] / (fu * 1e-6) / 1e12, 2),
                              "ffn_gbps": round(wb["ffn_bytes"] / (fu * 1e-6) / 1e9, 1),
                              "ffn_frac_mfma": round(wb["ffn_flops"] / (fu * 1e-6) / 1e12 / peak_f, 4),
                              "ffn_frac_hbm": round(wb["ffn_bytes"] / (fu * 1e-6) / 1e9 / PEAK_HBM_GBPS, 4)})
        result["skew_table"] = table
        # latency vs load on one expert, weight copies rotated past the 256 MB cache
        e_bytes = 3 * H * I * (2 if dt == torch.bfloat16 else 4)
        n_rot = max(1, -(-2 * MALL_BYTES // e_bytes))
        g1, u1, d1 = make_experts(shape, [int(li.local[0])], seed=args.seed)
        rep = lambda a: moe.pad_weight_rows(up(a).repeat(n_rot, 1, 1))
        xs = up(make_router(shape, max(SWEEP_MS), 0.0, seed=args.seed)[0])
        med, _ = moe.moe_load_sweep(xs, rep(g1), rep(u1), rep(d1), SWEEP_MS, warmup=3, iters=args.sweep_iters)
        med = [float(v) for v in med]
        result["load_sweep"] = {"M": SWEEP_MS, "us": [round(float(v), 2) for v in med], "n_rot": n_rot,
                                "tflops": [round(6.0 * H * I * m / (u * 1e-6) / 1e12, 2) for m, u in
                                           zip(SWEEP_MS, med)],
                                "gbps": [round((e_bytes + 2.0 * m * H * 2) / (u * 1e-6) / 1e9, 1) for m, u in
                                         zip(SWEEP_MS, med)]}
        if dt == torch.bfloat16:
            # the same expert in MXFP8 (weights 1 byte + a scale byte per 32)
            mx_bytes = 3 * H * I * (1 + 1 / 32)
            n_rot_mx = max(1, -(-2 * MALL_BYTES // int(mx_bytes)))
            rep_mx = lambda a: moe.moe_mx_quantize(up(a).repeat(n_rot_mx, 1, 1).contiguous())
            tg, tu, td = rep_mx(g1), rep_mx(u1), rep_mx(d1)
            med_mx, _ = moe.moe_load_sweep_mx(moe.moe_mx_quantize(xs), tg, tu, td, SWEEP_MS, warmup=3,
                                              iters=args.sweep_iters)
            med_mx = [float(v) for v in med_mx]
            del tg, tu, td
            result["load_sweep_mx"] = {
                "M": SWEEP_MS, "us": [round(float(v), 2) for v in med_mx], "n_rot": n_rot_mx,
                "tflops": [round(6.0 * H * I * m / (u * 1e-6) / 1e12, 2) for m, u in zip(SWEEP_MS, med_mx)],
                "gbps": [round((mx_bytes + m * H * (1 + 1 / 32) + 2.0 * m * H) / (u * 1e-6) / 1e9, 1)
                         for m, u in zip(SWEEP_MS, med_mx)],
                "speedup_vs_bf16": [round(b / m, 2) for b, m in zip(med, med_mx)]}

    placement_inputs = None
    if not args.no_extras:
        result["reference_peaks"] = reference_peaks(torch, np, w, T, H, I, dt)
        result["sclk"] = read_sclk()
        result["placement"], placement_inputs = placement_section(moe, args.seed)

    if not args.no_cpu:
        result["cpu_baseline"] = cpu_baseline(li, args.cpu_seconds)
        if placement_inputs is not None:
            result["cpu_baseline"]["placement"] = placement_oracle_timing(*placement_inputs)

    print(json.dumps(result), flush=True)


def mx_section(moe, torch, np, shape, li, wg, wu, wd, cases, steps, key):
    """The MXFP8 expert FFN on the routed rows of each case (x_perm, offsets
    of the bf16 layer): weights quantised once, outside the timing; x_perm
    quantisation and the FFN timed with HIP events on the current stream."""
    H, I = shape.H, shape.I
    # dense code rows: unlike the bf16 rows, padding FP8 rows of 4 KiB
    # measured no faster
    tg, tu, td = (moe.moe_mx_quantize(t.contiguous()) for t in (wg, wu, wd))
    torch.cuda.synchronize()
    out = []
    for Tb, a, bb, bf16_us in cases:
        xp, offs = bb["x_perm"], bb["offsets"]
        counts = np.diff(offs.cpu().numpy())
        m = int(counts.sum())
        active = int((counts > 0).sum())
        n_rows = offs[-1:]  # routed rows only, as the layer would
        tx = moe.moe_mx_quantize(xp, row_count=n_rows)
        y, ws = moe.moe_grouped_swiglu_ffn_mx(tx, tg, tu, td, offs)
        for _ in range(3):
            moe.moe_mx_quantize(xp, out=tx, row_count=n_rows)
            moe.moe_grouped_swiglu_ffn_mx(tx, tg, tu, td, offs, ws=ws, y_perm=y)
        torch.cuda.synchronize()
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
        for e in ev:
            e[0].record()
            moe.moe_mx_quantize(xp, out=tx, row_count=n_rows)
            e[1].record()
            moe.moe_grouped_swiglu_ffn_mx(tx, tg, tu, td, offs, ws=ws, y_perm=y)
            e[2].record()
        torch.cuda.synchronize()
        q_us = float(np.median([e[0].elapsed_time(e[1]) for e in ev])) * 1e3
        f_us = float(np.median([e[1].elapsed_time(e[2]) for e in ev])) * 1e3
        flops = 6.0 * m * H * I
        # weights of active experts (codes + scales), x codes + scales, h out and in, y out (bf16)
        nbytes = active * 3 * H * I * (1 + 1 / 32) + m * H * (1 + 1 / 32) + 2 * m * I * (1 + 1 / 32) + 2 * m * H
        tf = flops / (f_us * 1e-6) / 1e12
        gb = nbytes / (f_us * 1e-6) / 1e9
        mfma = flops / (PEAK_FP8_TFLOPS * 1e12) >= nbytes / (PEAK_HBM_GBPS * 1e9)
        out.append({"T": Tb, "alpha": a, "M_loc": m, "active": active, "ffn_us": round(f_us, 2),
                    "x_quantize_us": round(q_us, 2), "bf16_ffn_us": round(bf16_us, 2),
                    "speedup_vs_bf16": round(bf16_us / f_us, 3), "tflops": round(tf, 1), "gbps": round(gb, 1),
                    "bound": "mfma" if mfma else "hbm",
                    "frac": round(tf / PEAK_FP8_TFLOPS if mfma else gb / PEAK_HBM_GBPS, 4),
                    "peak": PEAK_FP8_TFLOPS if mfma else PEAK_HBM_GBPS, "algorithmic_bytes": round(nbytes),
                    "traffic": traffic_from_profile(key(Tb, a))})
    return {"format": "MXFP8 (E4M3 elements, E8M0 scale per 32 along K), bf16 output", "cases": out}


def reference_peaks(torch, np, w, T, H, I, dt):
    """Achievable peaks on this GPU, for context next to the datasheet
    denominators: a 1 GiB device-to-device copy (torch), and the vendor dense
    GEMMs (torch.matmul, hipBLASLt) of the FFN's shapes at M = M_loc."""
    def timed(fn, reps=10):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps * 1e-3
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    t_copy = timed(lambda: dst.copy_(src))
    del src, dst
    out = {"copy_1GiB_GBps": round(2 * n / t_copy / 1e9, 1)}
    m = int(w["m_loc"])
    if dt == torch.bfloat16 and m > 0:
        a1 = torch.randn(m, H, device="cuda", dtype=dt)
        b1 = torch.randn(H, 2 * I, device="cuda", dtype=dt)
        a2 = torch.randn(m, I, device="cuda", dtype=dt)
        b2 = torch.randn(I, H, device="cuda", dtype=dt)
        t1 = timed(lambda: torch.matmul(a1, b1))
        t2 = timed(lambda: torch.matmul(a2, b2))
        out["vendor_dense_gemm_us"] = {"gate_up_shape": round(t1 * 1e6, 1), "down_shape": round(t2 * 1e6, 1),
                                       "sum": round((t1 + t2) * 1e6, 1),
                                       "tflops": round(6.0 * m * H * I / (t1 + t2) / 1e12, 1)}
        del a1, b1, a2, b2
    return out


def read_sclk():
    """Current shader clock as rocm-smi reports it (None if unavailable)."""
    import subprocess
    try:
        r = subprocess.run(["rocm-smi", "--showclocks"], capture_output=True, text=True, timeout=20)
    except Exception:
        return None
    for line in r.stdout.splitlines():
        if "sclk" in line:
            return line.split(":", 1)[-1].strip()
    return None


PLACE_LAYERS, PLACE_GPUS, PLACE_T = 58, 8, 4096
PLACE_SWEEP_MS = [1, 8, 64, 256, 1024, 4096]


def placement_section(moe, seed):
    """ViBE's placement control path on this GPU for a DSV3-shaped model:
    58 MoE layers x 256 experts over 8 GPUs (32 slots each), f_g fitted from a
    sweep of one DSV3-shaped expert on this GPU and scaled per GPU by up to
    7 % (seeded), synthetic activation matrices with the rank-bias skew
    (alpha = 1) before and after a routing drift (8 rank swaps per layer).
    Times are HIP-event medians of the GPU calls; predicted layer latencies
    come from moe_placement_cost."""
    import numpy as np
    import torch
    from synth import CONFIGS, make_activation_matrix, make_experts, make_router

    shape = CONFIGS["dsv3_shard"]
    Lyr, G, E, k = PLACE_LAYERS, PLACE_GPUS, shape.E, shape.k
    cap = E // G
    up = lambda a, dt=torch.bfloat16: torch.from_numpy(np.ascontiguousarray(a)).cuda().to(dt).contiguous()
    g1, u1, d1 = make_experts(shape, [0], seed=seed)
    e_bytes = 3 * shape.H * shape.I * 2
    n_rot = max(1, -(-2 * MALL_BYTES // e_bytes))
    rep = lambda a: moe.pad_weight_rows(up(a).repeat(n_rot, 1, 1))
    xs = up(make_router(shape, max(PLACE_SWEEP_MS), 0.0, seed=seed)[0])
    med, _ = moe.moe_load_sweep(xs, rep(g1), rep(u1), rep(d1), PLACE_SWEEP_MS, warmup=3, iters=10)
    kn, kt = moe.moe_fit_latency_model(PLACE_SWEEP_MS, med)
    scale = 1.0 + 0.07 * np.random.default_rng(seed + 7).random(G)
    KN, KT = np.tile(kn, (G, 1)), np.outer(scale, kt)
    W1 = make_activation_matrix(Lyr, E, PLACE_T, k, 1.0, seed)
    W2 = make_activation_matrix(Lyr, E, PLACE_T, k, 1.0, seed, rank_swaps=8)
    d = lambda a, dt=torch.float64: torch.from_numpy(np.ascontiguousarray(a)).cuda().to(dt).contiguous()
    dW1, dW2, dKN, dKT = d(W1), d(W2), d(KN), d(KT)
    eKN, eKT = d(np.tile([1.0, 2.0], (G, 1))), d(np.tile([1.0, 2.0], (G, 1)))   # EPLB: f(n) = n

    def timed(fn, reps=20):
        fn()
        torch.cuda.synchronize()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for a, b in ev:
            a.record()
            fn()
            b.record()
        torch.cuda.synchronize()
        return float(np.median([a.elapsed_time(b) for a, b in ev]) * 1e3)

    vibe, _, _ = moe.moe_place_greedy(dW1, dKN, dKT, cap=cap)
    eplb, _, _ = moe.moe_place_greedy(dW1, eKN, eKT, cap=cap)
    contig = d(np.tile(np.arange(E) // cap, (Lyr, 1)), torch.int32)
    t_greedy = timed(lambda: moe.moe_place_greedy(dW1, dKN, dKT, cap=cap, assign=vibe))
    upd = vibe.clone()
    swaps = moe.moe_place_incremental(dW2, dKN, dKT, upd, eps=0.03)
    copies = iter([vibe.clone() for _ in range(21)])   # each timed call starts from the same placement
    t_incr = timed(lambda: moe.moe_place_incremental(dW2, dKN, dKT, next(copies), eps=0.03))
    t_drift = timed(lambda: moe.moe_drift_distance(dW2, dW1, delta=0.05))
    ring = torch.zeros((100, Lyr, E), dtype=torch.int32, device="cuda")
    sums = torch.zeros((Lyr, E), dtype=torch.float64, device="cuda")
    cnt = d(W1, torch.int32)
    t_push = timed(lambda: moe.moe_window_push(cnt, ring, sums, 0))
    dist, trig = moe.moe_drift_distance(dW2, dW1, delta=0.05)

    def total(W, A):
        _, lat, latg = moe.moe_placement_cost(W, A, dKN, dKT)
        return (round(float(lat.max(dim=1).values.sum().item()), 1),
                round(float(latg.max(dim=1).values.sum().item()), 1))

    pred = {"contiguous": total(dW1, contig), "eplb": total(dW1, eplb), "vibe": total(dW1, vibe),
            "after_drift_kept": total(dW2, vibe), "after_drift_incremental": total(dW2, upd),
            "after_drift_fresh_greedy": total(dW2, moe.moe_place_greedy(dW2, dKN, dKT, cap=cap)[0])}
    sw = swaps.cpu().numpy()
    out = {
        "workload": f"{Lyr} MoE layers x {E} experts on {G} GPUs ({cap} slots each), DSV3-shaped expert "
                    f"f_g from this GPU's sweep x (1 + 0.07 u_g), T={PLACE_T} tokens top-{k} per layer, alpha=1",
        "f_knots": {"n": [int(v) for v in kn], "us": [round(float(v), 2) for v in kt]},
        "gpu_speed_scale": [round(float(v), 4) for v in scale],
        "greedy_us": round(t_greedy, 2), "incremental_us": round(t_incr, 2),
        "drift_distance_us": round(t_drift, 2), "window_push_us": round(t_push, 2),
        "drift_max_distance": round(float(dist.max().item()), 4), "drift_trigger": int(trig.item()),
        "swaps_per_layer": {"mean": round(float(sw.mean()), 2), "max": int(sw.max())},
        "moved_by_fresh_greedy_per_layer": round(float(
            (moe.moe_place_greedy(dW2, dKN, dKT, cap=cap)[0] != vibe).sum(dim=1).float().mean().item()), 1),
        "predicted_sum_of_layer_latency_us": {k2: {"max_f_of_load": v[0], "max_sum_f_per_expert": v[1]}
                                              for k2, v in pred.items()},
    }
    return out, (W1, W2, KN, KT, cap)


def placement_oracle_timing(W1, W2, KN, KT, cap, layers=8):
    """The placement oracle on the first `layers` layers of the same inputs."""
    from oracle import placement_oracle as PO
    t = time.perf_counter()
    starts = [PO.greedy_placement(W1[l], KN, KT, cap=cap)[0] for l in range(layers)]
    t_g = time.perf_counter() - t
    t = time.perf_counter()
    for l in range(layers):
        PO.incremental_update(starts[l], W2[l], KN, KT, eps=0.03)
    t_i = time.perf_counter() - t
    return {"greedy_ms_per_layer": round(t_g / layers * 1e3, 3),
            "incremental_ms_per_layer": round(t_i / layers * 1e3, 3), "cores": 1,
            "sample": f"first {layers} of {W1.shape[0]} layers (pure Python, one thread)"}


def cpu_baseline(li, target_s):
    """The oracle, as it is, on the first n tokens of the same batch."""
    import numpy as np
    from oracle import moe_oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([int(i.get("num_threads", 1)) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = len(os.sched_getaffinity(0))
    shape = li.shape
    bf16 = shape.dtype == "bf16"

    def run(n):
        t = time.perf_counter()
        r = O.moe_layer(li.x[:n], li.w_router, li.bias, shape.k, li.expert_map, li.w_gate, li.w_up, li.w_down,
                        bf16=bf16)
        return time.perf_counter() - t, r

    n = min(li.T, 64)
    dt, r = run(n)
    while dt < target_s / 4 and n < li.T:
        n = min(li.T, int(n * max(2.0, min(8.0, target_s / max(dt, 1e-3)))))
        dt, r = run(n)
    # median of three runs of the chosen sample when they fit the time target
    times = [dt]
    if 2 * dt <= target_s:
        times += [run(n)[0] for _ in range(2)]
    dt = float(np.median(times))
    w = layer_work(shape, n, r["counts"], li.local)
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            model = next((ln.split(":", 1)[1].strip() for ln in fh if ln.startswith("model name")), model)
    except OSError:
        pass
    return {"value": round(w["layer_flops"] / dt / 1e12, 5), "unit": "TFLOP/s", "cores": threads,
            "kind": "oracle", "seconds": round(dt, 2), "runs": len(times), "cpu_model": model,
            "affinity_cpus": len(os.sched_getaffinity(0)),
            "sample": f"first {n} of {li.T} tokens of the same workload, whole layer (numpy fp32 BLAS), "
                      f"median of {len(times)} run(s)"}


if __name__ == "__main__":
    main()
