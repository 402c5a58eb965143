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
    sweeps = {}
    if not args.no_extras:
        # every (T, alpha) point of every workload, the headline workload's
        # weights reused, each other workload's generated and uploaded once
        table = []
        for name, sh in CONFIGS.items():
            if name == args.config:
                rows = skew_rows(moe, torch, np, sh, li.local, li.expert_map, wg, wu, wd, args)
            else:
                rows = workload_skew_rows(moe, torch, np, name, args)
            table.extend(rows)
        result["skew_table"] = table
        # latency vs load on one expert of every workload, cold and at steady
        # state (Section 4.2.1), weight copies rotated past the 256 MB cache
        for name, sh in CONFIGS.items():
            sweeps[name] = sweep_section(moe, torch, np, sh, args.seed, args.sweep_iters)
        result["load_sweep"] = sweeps
        if dt == torch.bfloat16:
            result["load_sweep_mx"] = mx_sweep_section(moe, torch, np, shape, li, args, sweeps.get(args.config))

    placement_inputs = None
    if not args.no_extras:
        result["reference_peaks"] = reference_peaks(torch, np, w, T, H, I, dt)
        result["sclk"] = read_sclk()
        result["placement"], placement_inputs = placement_section(moe, args.seed, sweeps.get("dsv3_shard"))

    if not args.no_cpu:
        result["cpu_baseline"] = cpu_baseline(li, args.cpu_seconds)
        result["cpu_baseline"]["single_thread"] = cpu_single_thread(li)
        if placement_inputs is not None:
            result["cpu_baseline"]["placement"] = placement_oracle_timing(*placement_inputs)

    print(json.dumps(result), flush=True)


def _up(torch, np, a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda().to(dtype).contiguous()


def time_layer(moe, torch, np, x, wr, bias, k, emap, wg, wu, wd, bb, steps, warmup, fuse):
    """`steps` timed layer passes (after `warmup`), HIP events around each
    stage on the current stream; returns (mean layer ms, per-stage mean us)."""
    names = ["gate_topk", "histogram_scan", "permute", "grouped_swiglu_ffn", "combine"]
    T, E = x.shape[0], wr.shape[0]
    for _ in range(warmup):
        moe.moe_layer(x, wr, bias, k, emap, wg, wu, wd, bufs=bb, fuse_gather=fuse)
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)] for _ in range(steps)]
    for s_ in range(steps):
        ev = evs[s_]
        ev[0].record()
        ids, wts, _ = moe.moe_gate_topk(x, wr, bias, k, ids=bb["ids"], weights=bb["weights"], ws=bb["gate_ws"])
        ev[1].record()
        counts, offsets, hws = moe.moe_expert_histogram_scan(ids, E, emap, ws=bb["hist_ws"], counts=bb["counts"],
                                                             offsets=bb["offsets"])
        ev[2].record()
        xp, ps, dest = moe.moe_permute(x, ids, emap, hws, x_perm=bb.get("x_perm"), perm_src=bb["perm_src"],
                                       dest=bb["dest"], gather=not fuse)
        ev[3].record()
        if fuse:
            yp, _ = moe.moe_grouped_swiglu_ffn_gather(x, ps, k, wg, wu, wd, offsets, ws=bb["ffn_ws"],
                                                      y_perm=bb["y_perm"])
        else:
            yp, _ = moe.moe_grouped_swiglu_ffn(xp, wg, wu, wd, offsets, ws=bb["ffn_ws"], y_perm=bb["y_perm"])
        ev[4].record()
        moe.moe_unpermute_combine(yp, wts, dest, T, out=bb["out"])
        ev[5].record()
    torch.cuda.synchronize()
    per = {n: [evs[s_][i].elapsed_time(evs[s_][i + 1]) * 1e3 for s_ in range(steps)] for i, n in enumerate(names)}
    stage = {n: float(np.mean(v)) for n, v in per.items()}
    return sum(stage.values()) * 1e-3, stage


def skew_rows(moe, torch, np, sh, local, emap, wg, wu, wd, args):
    """One row per (T, alpha) of a workload: layer time and the FFN against
    both roofline denominators (weights already on the GPU)."""
    from synth import make_router
    bf16 = sh.dtype == "bf16"
    dt = torch.bfloat16 if bf16 else torch.float32
    peak_f = PEAK_BF16_TFLOPS if bf16 else PEAK_FP32_TFLOPS
    rows = []
    for Tb in sh.Ts:
        for a in sh.alphas:
            xs, w_r, bs, _ = make_router(sh, Tb, a, seed=args.seed)
            xb, wrb, bb_bias = _up(torch, np, xs, dt), _up(torch, np, w_r, dt), _up(torch, np, bs, torch.float32)
            bb = {}
            moe.moe_layer(xb, wrb, bb_bias, sh.k, emap, wg, wu, wd, bufs=bb, fuse_gather=bf16)
            # each point first runs its own layer for ~0.2 s, so it is timed at
            # its own operating point (clock), not at the one the previous,
            # possibly much heavier, point left behind
            torch.cuda.synchronize()
            t_w = time.perf_counter()
            n_w = 0
            while time.perf_counter() - t_w < 0.2:
                for _ in range(4):
                    moe.moe_layer(xb, wrb, bb_bias, sh.k, emap, wg, wu, wd, bufs=bb, fuse_gather=bf16)
                n_w += 4
                torch.cuda.synchronize()
            ms_b, st_b = time_layer(moe, torch, np, xb, wrb, bb_bias, sh.k, emap, wg, wu, wd, bb,
                                    max(5, args.steps // 2), 3, bf16)
            wb = layer_work(sh, Tb, bb["counts"].cpu().numpy(), local)
            fu = st_b["grouped_swiglu_ffn"]
            cnt = bb["counts"].cpu().numpy()[np.asarray(local)]
            rows.append({"workload": sh.name, "T": Tb, "alpha": a, "us_per_layer": round(ms_b * 1e3, 2),
                         "layer_tflops": round(wb["layer_flops"] / (ms_b * 1e-3) / 1e12, 2),
                         "stages_us": {n: round(v, 2) for n, v in st_b.items()},
                         "ffn_us": round(fu, 2), "M_loc": wb["m_loc"], "active": wb["active"],
                         "max_rows_per_expert": int(cnt.max()) if cnt.size else 0,
                         "ffn_tflops": round(wb["ffn_flops"] / (fu * 1e-6) / 1e12, 2),
                         "ffn_gbps": round(wb["ffn_bytes"] / (fu * 1e-6) / 1e9, 1),
                         "ffn_frac_mfma": round(wb["ffn_flops"] / (fu * 1e-6) / 1e12 / peak_f, 4),
                         "ffn_frac_hbm": round(wb["ffn_bytes"] / (fu * 1e-6) / 1e9 / PEAK_HBM_GBPS, 4),
                         "ffn_binding_frac": round(max(wb["ffn_flops"] / (peak_f * 1e12),
                                                       wb["ffn_bytes"] / (PEAK_HBM_GBPS * 1e9)) / (fu * 1e-6), 4)})
            del bb, xb
    return rows


def workload_skew_rows(moe, torch, np, name, args):
    """skew_rows for a workload whose weights are generated here (and freed)."""
    from synth import CONFIGS, make_layer
    sh = CONFIGS[name]
    li = make_layer(sh, 1, 0.0, seed=args.seed)
    dt = torch.bfloat16 if sh.dtype == "bf16" else torch.float32
    ws = [_up(torch, np, a, dt) for a in (li.w_gate, li.w_up, li.w_down)]
    if dt == torch.bfloat16:
        ws = [moe.pad_weight_rows(t) for t in ws]
    del li.w_gate, li.w_up, li.w_down
    rows = skew_rows(moe, torch, np, sh, li.local, li.expert_map, *ws, args)
    del ws
    torch.cuda.empty_cache()
    return rows


def sclk_now():
    """Current shader clock (MHz) from the driver's DPM table in sysfs, or None."""
    import glob
    import re
    for path in sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk")):
        try:
            with open(path) as fh:
                txt = fh.read()
        except OSError:
            continue
        for ln in txt.splitlines():
            if ln.rstrip().endswith("*"):
                m = re.search(r"(\d+)\s*mhz", ln, re.I)
                if m:
                    return int(m.group(1))
    return None


class ClockSampler:
    """Reads sclk every `period` s in a thread while the block runs; the
    summary leaves out deep-sleep readings (< 400 MHz, idle gaps between
    launches)."""

    def __init__(self, period=0.002):
        import threading
        self.period, self.samples, self._stop = period, [], threading.Event()
        self._t = threading.Thread(target=self._run, daemon=True)

    def _run(self):
        while not self._stop.is_set():
            v = sclk_now()
            if v is not None:
                self.samples.append(v)
            self._stop.wait(self.period)

    def __enter__(self):
        self._t.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        self._t.join()

    def median(self):
        import statistics
        busy = [v for v in self.samples if v >= 400]
        return int(statistics.median(busy)) if busy else None


def sweep_section(moe, torch, np, sh, seed, iters):
    """Latency vs token load of one expert of workload `sh` (Section 4.2.1).

    cold:   each point alone (3 warm-up runs, then `iters` timed runs), the
            GPU otherwise idle;
    steady: first the GPU is held under the expert's largest load until the
            shader clock settles (three consecutive 50 ms windows within 2 %,
            at least 2 s, at most 20 s), then every point is preceded by
            about 30 ms of that load, so each is timed at the operating point
            of sustained MoE work.
    Every point records the median shader clock sampled while it ran."""
    from synth import make_experts, make_router
    from synth.moe_inputs import local_subset
    H, I = sh.H, sh.I
    bf16 = sh.dtype == "bf16"
    dt = torch.bfloat16 if bf16 else torch.float32
    es = 2 if bf16 else 4
    e_bytes = 3 * H * I * es
    n_rot = max(1, -(-2 * MALL_BYTES // e_bytes))
    g1, u1, d1 = make_experts(sh, [int(local_subset(sh, seed)[0])], seed=seed)
    if bf16:
        rep = lambda a: moe.pad_weight_rows(_up(torch, np, a, dt).repeat(n_rot, 1, 1))
    else:
        rep = lambda a: _up(torch, np, a, dt).repeat(n_rot, 1, 1).contiguous()
    wg, wu, wd = rep(g1), rep(u1), rep(d1)
    Mmax = max(SWEEP_MS)
    xs = _up(torch, np, make_router(sh, Mmax, 0.0, seed=seed)[0], dt)
    y = torch.empty((Mmax, H), dtype=dt, device="cuda")
    ws = None

    def point(M, warmup, n):
        nonlocal ws
        with ClockSampler() as cs:
            med, _ = moe.moe_load_sweep(xs, wg, wu, wd, [M], warmup=warmup, iters=n, y_scratch=y, ws=ws)
        return float(med[0]), cs.median()

    # workspace sized for the largest load, shared by every call
    ffn_bytes = moe.ffn_ws_bytes(1, H, I, Mmax, dt)
    ws = torch.zeros(ffn_bytes + 256, dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    time.sleep(0.5)
    cold = [point(M, 3, iters) for M in SWEEP_MS]
    # heat: repeat the largest load in ~50 ms windows until the clock settles
    t_big = max(cold[-1][0], 1.0) * 1e-6
    n_burst = max(1, int(0.05 / t_big))
    hist, t0 = [], time.perf_counter()
    while True:
        _, c = point(Mmax, 0, n_burst)
        hist.append(c or 0)
        el = time.perf_counter() - t0
        last = hist[-3:]
        if el > 20.0 or (el > 2.0 and len(last) == 3 and min(last) > 0 and max(last) <= 1.02 * min(last)):
            break
    n_keep = max(1, int(0.03 / t_big))
    steady = []
    for M in SWEEP_MS:
        point(Mmax, 0, n_keep)
        steady.append(point(M, 0, iters))
    del wg, wu, wd, xs, y, ws
    torch.cuda.empty_cache()
    fl = lambda pts: [round(6.0 * H * I * m / (u * 1e-6) / 1e12, 2) for m, (u, _) in zip(SWEEP_MS, pts)]
    gb = lambda pts: [round((e_bytes + 2.0 * m * H * es) / (u * 1e-6) / 1e9, 1) for m, (u, _) in zip(SWEEP_MS, pts)]
    return {"workload": sh.name, "H": H, "I": I, "M": SWEEP_MS, "n_rot": n_rot, "iters": iters,
            "cold": {"us": [round(u, 2) for u, _ in cold], "sclk_mhz": [c for _, c in cold],
                     "tflops": fl(cold), "gbps": gb(cold)},
            "steady": {"us": [round(u, 2) for u, _ in steady], "sclk_mhz": [c for _, c in steady],
                       "tflops": fl(steady), "gbps": gb(steady),
                       "warmup_s": round(time.perf_counter() - t0, 1), "warmup_sclk_mhz": hist[-3:]}}


def mx_sweep_section(moe, torch, np, shape, li, args, bf16_sweep):
    """The MXFP8 FFN on the same expert as the workload's bf16 sweep (cold)."""
    from synth import make_experts, make_router
    H, I = shape.H, shape.I
    mx_bytes = 3 * H * I * (1 + 1 / 32)
    n_rot = max(1, -(-2 * MALL_BYTES // int(mx_bytes)))
    g1, u1, d1 = make_experts(shape, [int(li.local[0])], seed=args.seed)
    rep = lambda a: moe.moe_mx_quantize(_up(torch, np, a, torch.bfloat16).repeat(n_rot, 1, 1).contiguous())
    tg, tu, td = rep(g1), rep(u1), rep(d1)
    xs = _up(torch, np, make_router(shape, max(SWEEP_MS), 0.0, seed=args.seed)[0], torch.bfloat16)
    med, _ = moe.moe_load_sweep_mx(moe.moe_mx_quantize(xs), tg, tu, td, SWEEP_MS, warmup=3, iters=args.sweep_iters)
    med = [float(v) for v in med]
    del tg, tu, td
    torch.cuda.empty_cache()
    out = {"workload": shape.name, "M": SWEEP_MS, "us": [round(v, 2) for v in med], "n_rot": n_rot,
           "tflops": [round(6.0 * H * I * m / (u * 1e-6) / 1e12, 2) for m, u in zip(SWEEP_MS, med)],
           "gbps": [round((mx_bytes + m * H * (1 + 1 / 32) + 2.0 * m * H) / (u * 1e-6) / 1e9, 1)
                    for m, u in zip(SWEEP_MS, med)]}
    if bf16_sweep is not None:
        out["speedup_vs_bf16_cold"] = [round(b / m, 2) for b, m in zip(bf16_sweep["cold"]["us"], med)]
    return out


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
    """Current shader clock as the driver reports it (None if unavailable)."""
    v = sclk_now()
    if v is not None:
        return f"{v} MHz"
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


def placement_section(moe, seed, dsv3_sweep=None):
    """ViBE's placement control path on this GPU for a DSV3-shaped model:
    58 MoE layers x 256 experts over 8 GPUs (32 slots each), f_g fitted from a
    sweep of one DSV3-shaped expert on this GPU and scaled per GPU by up to
    7 % (seeded), synthetic activation matrices with the rank-bias skew
    (alpha = 1) before and after a routing drift (8 rank swaps per layer).
    Times are HIP-event medians of the GPU calls; predicted layer latencies
    come from moe_placement_cost. With `dsv3_sweep` (sweep_section's result
    for the DSV3-shaped workload) f is fitted from its steady-state curve."""
    import numpy as np
    import torch
    from synth import CONFIGS, make_activation_matrix, make_experts, make_router

    shape = CONFIGS["dsv3_shard"]
    Lyr, G, E, k = PLACE_LAYERS, PLACE_GPUS, shape.E, shape.k
    cap = E // G
    up = lambda a, dt=torch.bfloat16: torch.from_numpy(np.ascontiguousarray(a)).cuda().to(dt).contiguous()
    if dsv3_sweep is not None:
        f_src = "steady-state sweep of the DSV3-shaped expert (load_sweep)"
        kn, kt = moe.moe_fit_latency_model(dsv3_sweep["M"], dsv3_sweep["steady"]["us"])
    else:
        f_src = "cold sweep of the DSV3-shaped expert"
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
        "f_knots": {"n": [int(v) for v in kn], "us": [round(float(v), 2) for v in kt], "source": f_src},
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


def cpu_model_name():
    """The host CPU as lscpu names it (model, family/model/stepping, sockets)."""
    import subprocess
    info = {}
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for ln in out.splitlines():
            if ":" in ln:
                k, v = ln.split(":", 1)
                info[k.strip()] = v.strip()
    except Exception:
        pass
    name = info.get("Model name") or info.get("BIOS Model name") or "unknown"
    extra = ", ".join(f"{k} {info[k]}" for k in ("CPU family", "Model", "Stepping", "Socket(s)", "CPU max MHz")
                      if k in info)
    return f"{name} ({extra})" if extra else name


def cpu_single_thread(li):
    """The oracle with one BLAS thread on the decode-sized and tiny workloads
    (whole layer, every token)."""
    import numpy as np
    from threadpoolctl import threadpool_limits
    from oracle import moe_oracle as O
    from synth import CONFIGS, make_layer
    out = []
    for name, T, a in (("tiny", 64, 1.0), ("mixtral", 32, 0.0), ("qwen3", 128, 0.0)):
        sh = CONFIGS[name]
        if li.shape.name == name:   # the headline workload's weights, this batch's router inputs
            from synth import make_router
            lj = li
            x, w_r, bias, _ = make_router(sh, T, a, seed=li.seed)
        else:
            lj = make_layer(sh, T, a, seed=li.seed)
            x, w_r, bias = lj.x, lj.w_router, lj.bias
        with threadpool_limits(1):
            t = time.perf_counter()
            r = O.moe_layer(x, w_r, bias, sh.k, lj.expert_map, lj.w_gate, lj.w_up, lj.w_down,
                            bf16=sh.dtype == "bf16")
            dt = time.perf_counter() - t
        w = layer_work(sh, T, r["counts"], lj.local)
        out.append({"workload": name, "T": T, "alpha": a, "seconds": round(dt, 3),
                    "tflops": round(w["layer_flops"] / dt / 1e12, 6), "us_per_layer": round(dt * 1e6, 1),
                    "cores": 1})
        del lj
    return out


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
    model = cpu_model_name()
    return {"value": round(w["layer_flops"] / dt / 1e12, 5), "unit": "TFLOP/s", "cores": threads,
            "kind": "oracle", "seconds": round(dt, 2), "runs": len(times), "cpu_model": model,
            "affinity_cpus": len(os.sched_getaffinity(0)),
            "sample": f"first {n} of {li.T} tokens of the same workload, whole layer (numpy fp32 BLAS), "
                      f"median of {len(times)} run(s)"}


if __name__ == "__main__":
    main()
