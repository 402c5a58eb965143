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
    for f in ("ffn_kernels.hip", "common.hpp"):
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
    wg, wu, wd = up(li.w_gate), up(li.w_up), up(li.w_down)
    t_gen = time.time() - t_gen
    emap = li.expert_map
    E_local = len(li.local)

    def make_bufs(Tb, xb):
        b = {}
        moe.moe_layer(xb, wr, bias, k, emap, wg, wu, wd, bufs=b)
        return b

    def run_timed(xb, bb, Tb, steps, warmup):
        """Warmup, then `steps` timed layer passes with per-stage HIP events."""
        names = ["gate_topk", "histogram_scan", "permute", "grouped_swiglu_ffn", "combine"]
        for _ in range(warmup):
            moe.moe_layer(xb, wr, bb["bias"], k, emap, wg, wu, wd, bufs=bb)
        torch.cuda.synchronize()
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)] for _ in range(steps)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for s in range(steps):
            ev = evs[s]
            ev[0].record()
            ids, wts, _ = moe.moe_gate_topk(xb, wr, bb["bias"], k, ids=bb["ids"], weights=bb["weights"])
            ev[1].record()
            counts, offsets, hws = moe.moe_expert_histogram_scan(ids, E, emap, ws=bb["hist_ws"],
                                                                 counts=bb["counts"], offsets=bb["offsets"])
            ev[2].record()
            xp, ps, dest = moe.moe_permute(xb, ids, emap, hws, x_perm=bb["x_perm"], perm_src=bb["perm_src"],
                                           dest=bb["dest"])
            ev[3].record()
            yp, _ = moe.moe_grouped_swiglu_ffn(xp, wg, wu, wd, offsets, ws=bb["ffn_ws"], y_perm=bb["y_perm"])
            ev[4].record()
            moe.moe_unpermute_combine(yp, wts, dest, Tb, out=bb["out"])
            ev[5].record()
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        stage = {n: float(np.mean([evs[s][i].elapsed_time(evs[s][i + 1]) for s in range(steps)])) * 1e3
                 for i, n in enumerate(names)}
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
        "kernel": "moe_grouped_swiglu_ffn (gate/up and down GEMMs + split-K reductions)",
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
                   "seed": args.seed, "M_loc": w["m_loc"], "active_local_experts": w["active"]},
        "us_per_layer": round(us, 2),
        "layer_gbps": round(w["layer_bytes"] / (us * 1e-6) / 1e9, 1),
        "stages_us": {n: round(v, 2) for n, v in stage.items()},
        "roofline": roofline,
        "gen_s": round(t_gen, 1),
    }

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
        rep = lambda a: up(a).repeat(n_rot, 1, 1).contiguous()
        xs = up(make_router(shape, max(SWEEP_MS), 0.0, seed=args.seed)[0])
        med, _ = moe.moe_load_sweep(xs, rep(g1), rep(u1), rep(d1), SWEEP_MS, warmup=3, iters=args.sweep_iters)
        med = [float(v) for v in med]
        result["load_sweep"] = {"M": SWEEP_MS, "us": [round(float(v), 2) for v in med], "n_rot": n_rot,
                                "tflops": [round(6.0 * H * I * m / (u * 1e-6) / 1e12, 2) for m, u in
                                           zip(SWEEP_MS, med)],
                                "gbps": [round((e_bytes + 2.0 * m * H * 2) / (u * 1e-6) / 1e9, 1) for m, u in
                                         zip(SWEEP_MS, med)]}

    if not args.no_cpu:
        result["cpu_baseline"] = cpu_baseline(li, args.cpu_seconds)

    print(json.dumps(result), flush=True)


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
    w = layer_work(shape, n, r["counts"], li.local)
    return {"value": round(w["layer_flops"] / dt / 1e12, 5), "unit": "TFLOP/s", "cores": threads,
            "kind": "oracle", "seconds": round(dt, 2),
            "sample": f"first {n} of {li.T} tokens of the same workload, whole layer (numpy fp32 BLAS)"}


if __name__ == "__main__":
    main()
