"""Build libmoe.so (HIP for gfx950) in-tree with hipcc.

    python -m paper_2606_00735_amd.build

Every HIP source is compiled for gfx950 only, without packed-fp32 VALU ops.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libmoe.so")

SOURCES = ["route_kernels.hip", "ffn_kernels.hip", "mx_kernels.hip", "placement_kernels.hip", "moe_abi.cpp"]
HEADERS = ["common.hpp", "launch.hpp", "mx.hpp"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: a ROCm toolchain is required to build libmoe")


FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-function"]


def command(out: str = LIB, extra=()) -> list:
    """One hipcc command that compiles and links every source."""
    srcs = [os.path.join(CSRC, s) for s in SOURCES]
    return [hipcc(), *FLAGS, "-shared", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
            "-x", "hip", *srcs, *extra, "-o", out]


def compile_commands(objdir: str) -> list:
    """(object path, hipcc command) per source, for a parallel build."""
    out = []
    for s in SOURCES:
        obj = os.path.join(objdir, s + ".o")
        out.append((obj, [hipcc(), *FLAGS, "-I", os.path.join(ROOT, "include"), "-I", CSRC,
                          "-x", "hip", "-c", os.path.join(CSRC, s), "-o", obj]))
    return out


STAMP = LIB + ".srchash"


def source_hash() -> str:
    """sha256 over every source and header that goes into libmoe.so."""
    import hashlib
    h = hashlib.sha256()
    for f in SOURCES + HEADERS:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    with open(os.path.join(ROOT, "include", "moe.h"), "rb") as fh:
        h.update(fh.read())
    return h.hexdigest()


def is_fresh() -> bool:
    """True when libmoe.so was built from the sources as they are now."""
    try:
        with open(STAMP) as fh:
            return os.path.exists(LIB) and fh.read().strip() == source_hash()
    except OSError:
        return False


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in r.stderr.splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed ({r.returncode}):\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)


def build(verbose: bool = False) -> str:
    """Compile libmoe.so next to this file (one hipcc per source, in
    parallel, then a link step); returns its path."""
    import concurrent.futures as cf
    import tempfile
    tmp = LIB + ".tmp"
    with tempfile.TemporaryDirectory(prefix="libmoe_build_") as objdir:
        jobs = compile_commands(objdir)
        with cf.ThreadPoolExecutor(len(jobs)) as ex:
            list(ex.map(lambda j: _run(j[1], verbose), jobs))
        _run([hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *[o for o, _ in jobs], "-o", tmp], verbose)
    os.replace(tmp, LIB)
    with open(STAMP, "w") as fh:
        fh.write(source_hash())
    return LIB


if __name__ == "__main__":
    if len(sys.argv) > 1 and sys.argv[1] == "--check":
        sys.exit(0 if is_fresh() else 1)
    print(build(verbose=True))
