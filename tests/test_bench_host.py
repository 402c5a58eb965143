"""Host-side checks of bench.py: the one-GPU contract, the algorithmic work
it divides by, and when it reports counter-based traffic. No GPU needed."""
import json
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from synth import CONFIGS  # noqa: E402


@pytest.mark.parametrize("argv,env", [(["--gpus", "2"], {}), (["--gpus", "8"], {}), ([], {"WORLD_SIZE": "2"})])
def test_more_than_one_gpu_exits(argv, env):
    """Several GPUs are refused before anything is imported or measured."""
    e = dict(os.environ, **env)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *argv], capture_output=True, text=True,
                       env=e, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_layer_work_closed_form():
    """Flops and bytes of a small layer worked out by hand: H = 4, I = 6,
    3 experts, top-2, bf16, T = 5, 3 + 0 + 7 routed rows."""
    shape = CONFIGS["qwen3"].__class__(name="hand", H=4, I=6, E=3, k=2, E_local=3, dtype="bf16", Ts=(5,),
                                       alphas=(0.0,))
    w = bench.layer_work(shape, 5, [3, 0, 7], [0, 1, 2])
    assert w["m_loc"] == 10 and w["active"] == 2
    assert w["ffn_flops"] == 6 * 4 * 6 * 10                 # 2 flops per MAC, three H x I matrices
    assert w["layer_flops"] == 6 * 4 * 6 * 10 + 2 * 5 * 4 * 3  # plus the router's logits
    assert w["ffn_bytes"] == 3 * 4 * 6 * 2 * 2 + 2 * 10 * 4 * 2  # active experts' weights, x_perm in, y_perm out
    # weights, x in and out, router weights, ids and weights of k slots per token
    assert w["layer_bytes"] == 3 * 4 * 6 * 2 * 2 + 2 * 5 * 4 * 2 + 4 * 3 * 2 + 16 * 5 * 2


def test_layer_work_sharded_fp32():
    """Only local experts count; fp32 elements are 4 bytes."""
    shape = CONFIGS["tiny"]
    w = bench.layer_work(shape, 64, [5, 9, 0, 2, 7, 0, 1, 3], [1, 2, 3])
    assert w["m_loc"] == 11 and w["active"] == 2
    assert w["ffn_bytes"] == 3 * shape.H * shape.I * 4 * 2 + 2 * 11 * shape.H * 4


def _fake_root(tmp_path, sha_matches):
    """A copy of the kernel sources and a profile record for one workload."""
    src = os.path.join(ROOT, "paper_2606_00735_amd", "csrc")
    dst = tmp_path / "paper_2606_00735_amd" / "csrc"
    dst.mkdir(parents=True)
    for f in ("ffn_kernels.hip", "common.hpp", "mx.hpp"):
        shutil.copy(os.path.join(src, f), dst / f)
    (tmp_path / "profiles").mkdir()
    sha = bench.source_sha() if sha_matches else "0" * 16
    rec = {"w-T8-a0-s0": {"source_sha": sha, "bytes_per_call": 12345.0}}
    (tmp_path / "profiles" / "ffn_traffic.json").write_text(json.dumps(rec))
    return str(tmp_path)


def test_traffic_only_from_counters_on_the_current_source(tmp_path, monkeypatch):
    root = _fake_root(tmp_path, sha_matches=True)
    monkeypatch.setattr(bench, "ROOT", root)
    assert bench.traffic_from_profile("w-T8-a0-s0") == 12345.0
    assert bench.traffic_from_profile("other-T8-a0-s0") is None
    # any change to a kernel source makes the record stale
    with open(os.path.join(root, "paper_2606_00735_amd", "csrc", "mx.hpp"), "a") as fh:
        fh.write("\n")
    assert bench.traffic_from_profile("w-T8-a0-s0") is None


def test_traffic_none_for_other_source_or_missing_file(tmp_path, monkeypatch):
    root = _fake_root(tmp_path, sha_matches=False)
    monkeypatch.setattr(bench, "ROOT", root)
    assert bench.traffic_from_profile("w-T8-a0-s0") is None
    os.remove(os.path.join(root, "profiles", "ffn_traffic.json"))
    assert bench.traffic_from_profile("w-T8-a0-s0") is None
