"""CPU tests of the seeded input generator and of the router-grid exactness."""
import dataclasses

import numpy as np
import pytest

from synth import CONFIGS, make_router, make_experts, make_layer, router_grid_q
from synth.moe_inputs import local_subset, expert_map_for
from oracle import moe_oracle as O


@pytest.mark.parametrize("name", sorted(CONFIGS))
def test_router_logits_order_independent(name):
    """On the grids every fp32 summation order gives the same logits.

    The oracle's fp32 BLAS result must equal the fp64 result bit for bit, and
    so must a reversed-order fp32 accumulation: this is what lets the GPU's
    top-k match the oracle's exactly.
    """
    shape = CONFIGS[name]
    x, w, b, rank = make_router(shape, 96, alpha=1.0, seed=0)
    acc32 = np.matmul(x, w.T).astype(np.float32)
    acc64 = np.matmul(x.astype(np.float64), w.T.astype(np.float64))
    assert np.array_equal(acc32.astype(np.float64), acc64)
    rev = np.zeros_like(acc32)
    for h in range(shape.H - 1, -1, -1):  # reversed order, fp32 each step
        rev = (rev + (x[:, h:h + 1] * w[:, h][None, :]).astype(np.float32)).astype(np.float32)
    assert np.array_equal(rev, acc32)
    z = O.router_logits(x, w, b)
    assert np.array_equal(z, (acc64.astype(np.float32) + b).astype(np.float32))


def test_router_grids():
    shape = CONFIGS["dsv3_shard"]
    x, w, b, rank = make_router(shape, 64, alpha=1.5, seed=1)
    assert np.all(np.abs(x) <= 255 / 64) and np.array_equal(x * 64, np.rint(x * 64))
    q = router_grid_q(shape.H)
    assert q == 11
    assert np.array_equal(w * 2.0 ** q, np.rint(w * 2.0 ** q))
    assert sorted(rank.tolist()) == list(range(1, shape.E + 1))
    np.testing.assert_array_equal(b, (-1.5 * np.log(rank.astype(np.float64))).astype(np.float32))
    assert [router_grid_q(CONFIGS[n].H) for n in ("tiny", "qwen3", "mixtral", "maverick_shard")] \
        == [8, 10, 10, 11]


def test_deterministic_and_seeded():
    shape = CONFIGS["qwen3"]
    a = make_router(shape, 40, 1.0, seed=3)
    b = make_router(shape, 40, 1.0, seed=3)
    c = make_router(shape, 40, 1.0, seed=4)
    for u, v in zip(a, b):
        assert np.array_equal(u, v)
    assert not np.array_equal(a[0], c[0])
    # x rows do not depend on T (prefix property of the per-block streams)
    big = make_router(shape, 2100, 1.0, seed=3)[0]
    assert np.array_equal(big[:40], a[0])


def test_shard_weights_match_full_layer():
    """A shard's expert weights equal the full layer's for the same experts."""
    small = dataclasses.replace(CONFIGS["dsv3_shard"], H=16, I=8, E=12, E_local=4)
    full = make_experts(dataclasses.replace(small, E_local=12), range(12), seed=5)
    local = local_subset(small, 5)
    assert len(local) == 4 and np.all(np.diff(local) > 0)
    part = make_experts(small, local, seed=5)
    for f, p in zip(full, part):
        assert np.array_equal(f[local], p)
    emap = expert_map_for(small, local)
    assert np.array_equal(np.where(emap >= 0)[0], local)
    assert np.array_equal(emap[local], np.arange(4))


def test_bf16_weights_representable():
    import torch
    small = dataclasses.replace(CONFIGS["qwen3"], H=64, I=32, E=4, E_local=4)
    for a in make_experts(small, range(4), seed=0):
        t = torch.from_numpy(a).to(torch.bfloat16).float().numpy()
        assert np.array_equal(t, a)


def test_tiny_layer_inputs():
    li = make_layer("tiny", 64, 1.0, seed=0)
    assert li.x.shape == (64, 128) and li.w_gate.shape == (8, 256, 128)
    assert li.w_down.shape == (8, 128, 256)
    assert np.array_equal(li.expert_map, np.arange(8))
