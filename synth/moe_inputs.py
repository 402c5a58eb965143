"""Seeded synthetic inputs for the MoE expert-shard layer.

Recipe (the workloads the paper profiles are trained DeepSeek-V3 / Qwen-3
layers driven by ShareGPT and Sonnet, Section 5.1 and Table 2; neither the
checkpoints nor the datasets are available, so seeded synthetic inputs of the
same shapes stand in for them, and a rank bias stands in for their routing
skew, cf. the per-GPU token shares of Section 3):

* ``x [T, H]``: N(0, 1) draws put on the 1/64 grid and clipped to +-255/64.
* ``w_router [E, H]`` (row e is expert e's routing vector): N(0, 1/H) draws put
  on the 2^-q grid, q = ceil(log2(16 sqrt(H))), clipped to +-255 * 2^-q.
  With both grids every product x*w is a multiple of 2^-(6+q); as long as
  sum_h |x_th| |w_eh| < 2^(24-6-q) every partial sum, in any order, is an
  exactly representable fp32 value, so router logits do not depend on the
  summation order. ``make_router`` checks that bound (Cauchy-Schwarz form).
* ``bias [E]``: b_e = fp32(-alpha * ln(rank_e)), rank a seeded permutation of
  1..E; rank 1 is the hottest expert, alpha = 0 means no skew.
* expert weights, stored out-features by in-features (the nn.Linear layout):
  ``w_gate[e], w_up[e]`` are [I, H] with N(0, 1/H) entries and ``w_down[e]`` is
  [H, I] with N(0, 1/I) entries. bf16 configs round them (RNE) to bf16 values.
* the local expert subset of a shard: a seeded subset, sorted ascending; local
  slot = position in that order. ``expert_map[e]`` is the slot or -1.

Every role draws from its own PCG64 stream spawned from ``SeedSequence(seed)``;
expert e draws from the e-th child of the expert stream, so a shard generates
only its own experts and gets the same values as the full layer would.
Arrays are float32 numpy arrays holding bf16-representable values for bf16
configs, so converting them to a bf16 tensor is exact.
"""
from __future__ import annotations

import concurrent.futures as _cf
import dataclasses
import math
import os

import numpy as np

# Stream roles spawned from SeedSequence(seed). Fixed order: never reorder.
_ROLE_X, _ROLE_ROUTER, _ROLE_RANK, _ROLE_SUBSET, _ROLE_EXPERTS = range(5)
_N_ROLES = 5
# x rows are drawn in fixed blocks, each from its own stream, so that threads
# can fill them in parallel without the values depending on the thread count.
_X_BLOCK_ROWS = 1024


@dataclasses.dataclass(frozen=True)
class LayerShape:
    name: str
    H: int            # hidden size
    I: int            # expert intermediate size
    E: int            # global experts
    k: int            # experts per token
    E_local: int      # experts computed on this GPU
    dtype: str        # "f32" or "bf16"
    Ts: tuple         # token counts the workload is run at
    alphas: tuple     # skew levels


CONFIGS = {
    # Tiny fp32 layer: every step checkable by brute force.
    "tiny": LayerShape("tiny", H=128, I=256, E=8, k=2, E_local=8, dtype="f32",
                       Ts=(64,), alphas=(1.0,)),
    # Mixtral-8x7B-shaped layer, all 8 experts on one GPU.
    "mixtral": LayerShape("mixtral", H=4096, I=14336, E=8, k=2, E_local=8,
                          dtype="bf16", Ts=(32, 4096), alphas=(0.0, 1.0)),
    # Qwen3-30B-A3B-shaped layer, all 128 experts local: many small-M experts.
    "qwen3": LayerShape("qwen3", H=2048, I=768, E=128, k=8, E_local=128,
                        dtype="bf16", Ts=(128, 8192), alphas=(0.0, 1.0, 1.5)),
    # DeepSeek-V3-shaped shard: 32 of 256 experts computed on this GPU.
    "dsv3_shard": LayerShape("dsv3_shard", H=7168, I=2048, E=256, k=8, E_local=32,
                             dtype="bf16", Ts=(16384,), alphas=(0.0, 1.0, 1.5)),
    # Llama-4-Maverick-shaped shard: 16 of 128 experts, top-1.
    "maverick_shard": LayerShape("maverick_shard", H=5120, I=8192, E=128, k=1,
                                 E_local=16, dtype="bf16", Ts=(32768,),
                                 alphas=(0.0, 1.0, 1.5)),
}


def round_to_bf16_values(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 value (ties to even), as float32.

    Input shaping only: the generated weights must be exactly representable in
    bf16 so that both sides see identical operands.
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + (np.uint32(0x7FFF) + lsb)) & np.uint32(0xFFFF0000)
    return r.view(np.float32)


def router_grid_q(H: int) -> int:
    """Exponent q of the router-weight grid 2^-q for hidden size H."""
    return int(math.ceil(math.log2(16.0 * math.sqrt(H))))


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _roles(seed: int):
    return np.random.SeedSequence(seed).spawn(_N_ROLES)


def _make_x(ss: np.random.SeedSequence, T: int, H: int) -> np.ndarray:
    n_blocks = (T + _X_BLOCK_ROWS - 1) // _X_BLOCK_ROWS
    kids = ss.spawn(max(n_blocks, 1))
    x = np.empty((T, H), np.float32)

    def fill(b):
        r0 = b * _X_BLOCK_ROWS
        r1 = min(T, r0 + _X_BLOCK_ROWS)
        g = np.random.Generator(np.random.PCG64(kids[b]))
        blk = x[r0:r1]
        g.standard_normal(out=blk, dtype=np.float32)
        np.rint(blk * np.float32(64.0), out=blk)
        np.clip(blk, -255.0, 255.0, out=blk)
        blk *= np.float32(1.0 / 64.0)

    if n_blocks > 1:
        with _cf.ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(fill, range(n_blocks)))
    elif T > 0:
        fill(0)
    return x


def make_router(shape: LayerShape, T: int, alpha: float, seed: int,
                check_bound: bool = True):
    """x [T,H], w_router [E,H], bias [E], rank [E] for one layer-batch."""
    H, E = shape.H, shape.E
    roles = _roles(seed)
    x = _make_x(roles[_ROLE_X], T, H)
    q = router_grid_q(H)
    g = np.random.Generator(np.random.PCG64(roles[_ROLE_ROUTER]))
    w = g.standard_normal((E, H), dtype=np.float32) * np.float32(1.0 / math.sqrt(H))
    w = np.clip(np.rint(w * np.float32(2.0 ** q)), -255.0, 255.0).astype(np.float32)
    w *= np.float32(2.0 ** -q)
    g = np.random.Generator(np.random.PCG64(roles[_ROLE_RANK]))
    rank = g.permutation(E).astype(np.int64) + 1
    bias = (-float(alpha) * np.log(rank.astype(np.float64))).astype(np.float32)
    if check_bound and T > 0:
        # Cauchy-Schwarz bound on sum_h |x_th| |w_eh|: must stay below
        # 2^(24-6-q) so every partial sum is exact in fp32.
        xn = float(np.sqrt((x.astype(np.float64) ** 2).sum(axis=1)).max())
        wn = float(np.sqrt((w.astype(np.float64) ** 2).sum(axis=1)).max())
        limit = 2.0 ** (24 - 6 - q)
        if not xn * wn < limit:
            raise ValueError(f"router grid bound violated: {xn * wn} >= {limit}")
    return x, w, bias, rank


def local_subset(shape: LayerShape, seed: int) -> np.ndarray:
    """Sorted global ids of the experts computed on this GPU."""
    if shape.E_local == shape.E:
        return np.arange(shape.E, dtype=np.int64)
    roles = _roles(seed)
    g = np.random.Generator(np.random.PCG64(roles[_ROLE_SUBSET]))
    sub = g.choice(shape.E, size=shape.E_local, replace=False)
    return np.sort(sub).astype(np.int64)


def expert_map_for(shape: LayerShape, local: np.ndarray) -> np.ndarray:
    m = np.full(shape.E, -1, np.int32)
    m[np.asarray(local, dtype=np.int64)] = np.arange(len(local), dtype=np.int32)
    return m


def make_experts(shape: LayerShape, experts, seed: int):
    """w_gate [n,I,H], w_up [n,I,H], w_down [n,H,I] for the given global ids."""
    H, I = shape.H, shape.I
    experts = [int(e) for e in experts]
    n = len(experts)
    roles = _roles(seed)
    kids = roles[_ROLE_EXPERTS].spawn(shape.E)
    wg = np.empty((n, I, H), np.float32)
    wu = np.empty((n, I, H), np.float32)
    wd = np.empty((n, H, I), np.float32)
    sg = np.float32(1.0 / math.sqrt(H))
    sd = np.float32(1.0 / math.sqrt(I))
    bf16 = shape.dtype == "bf16"

    def fill(slot):
        g = np.random.Generator(np.random.PCG64(kids[experts[slot]]))
        for dst, s in ((wg[slot], sg), (wu[slot], sg), (wd[slot], sd)):
            g.standard_normal(out=dst, dtype=np.float32)
            dst *= s
            if bf16:
                dst[...] = round_to_bf16_values(dst)

    if n > 1:
        with _cf.ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(fill, range(n)))
    elif n == 1:
        fill(0)
    return wg, wu, wd


@dataclasses.dataclass
class LayerInputs:
    shape: LayerShape
    T: int
    alpha: float
    seed: int
    x: np.ndarray          # [T, H] float32 (grid values)
    w_router: np.ndarray   # [E, H] float32 (grid values)
    bias: np.ndarray       # [E] float32
    rank: np.ndarray       # [E] int64, 1 = hottest
    local: np.ndarray      # [E_local] sorted global ids
    expert_map: np.ndarray  # [E] int32: local slot or -1
    w_gate: np.ndarray | None = None   # [E_local, I, H]
    w_up: np.ndarray | None = None     # [E_local, I, H]
    w_down: np.ndarray | None = None   # [E_local, H, I]


def make_layer(shape, T: int, alpha: float, seed: int = 0,
               with_experts: bool = True) -> LayerInputs:
    """All inputs of one layer-batch for a named config or a LayerShape."""
    if isinstance(shape, str):
        shape = CONFIGS[shape]
    x, w, bias, rank = make_router(shape, T, alpha, seed)
    local = local_subset(shape, seed)
    emap = expert_map_for(shape, local)
    li = LayerInputs(shape, T, float(alpha), seed, x, w, bias, rank, local, emap)
    if with_experts:
        li.w_gate, li.w_up, li.w_down = make_experts(shape, local, seed)
    return li


def make_activation_matrix(L: int, E: int, T: int, k: int, alpha: float, seed: int,
                           rank_swaps: int = 0, drift_seed: int = 1):
    """Per-layer expert loads W [L, E] (float64 counts) of T tokens routed top-k.

    Layer l has its own seeded rank permutation; token t picks the k experts
    with the largest -alpha * ln(rank_e) + g_te, g i.i.d. standard Gumbel (a
    synthetic router with the rank-bias skew). ``rank_swaps`` > 0 exchanges
    the ranks of that many random expert pairs per layer first (a routing
    drift: other experts become hot), drawn from ``drift_seed``.
    """
    root = np.random.SeedSequence(seed)
    kids = root.spawn(2 * L)
    dkids = np.random.SeedSequence(drift_seed).spawn(L)
    W = np.zeros((L, E), np.float64)
    for l in range(L):
        g = np.random.Generator(np.random.PCG64(kids[2 * l]))
        rank = g.permutation(E).astype(np.int64) + 1
        if rank_swaps:
            d = np.random.Generator(np.random.PCG64(dkids[l]))
            for _ in range(rank_swaps):
                i, j = d.choice(E, 2, replace=False)
                rank[i], rank[j] = rank[j], rank[i]
        prior = -float(alpha) * np.log(rank.astype(np.float64))
        t = np.random.Generator(np.random.PCG64(kids[2 * l + 1]))
        score = prior[None, :] + t.gumbel(size=(T, E))
        top = np.argpartition(-score, k - 1, axis=1)[:, :k]
        W[l] = np.bincount(top.ravel(), minlength=E)
    return W
