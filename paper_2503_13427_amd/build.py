"""Compile libmlstm.so (HIP kernels + C ABI) for gfx950 with hipcc, in-tree.

Every translation unit is compiled to an object in parallel, then linked.
Flags: -O3, gfx950 only, and packed-fp32 instruction selection disabled
(-Xclang -target-feature -Xclang -packed-fp32-ops) for every HIP source.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJDIR = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libmlstm.so")
# the same sources with the device bounds checks compiled in (-DMLSTM_DEBUG; mlstm_debug_flags)
DEBUG_OBJDIR = os.path.join(PKG, "_build_debug")
DEBUG_LIB = os.path.join(PKG, "libmlstm_debug.so")
ARCH = "gfx950"

SOURCES = ["mlstm_abi.cpp", "mlstm_step.hip", "mlstm_chunkwise_f32.hip", "mlstm_chunkwise_mfma.hip",
           "mlstm_output_norm.hip", "mlstm_gate_preact.hip",
           "mlstm_parallel_bwd.hip", "mlstm_chunkwise_bwd.hip"]
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-I", INCLUDE, "-I", CSRC,
          "-Wall", "-Wno-unused-result"]
NO_PACKED_FP32 = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _hipcc() -> str:
    for p in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if p and os.path.exists(p):
            return p
    return "hipcc"


def _compile(src: str, debug: bool = False) -> str:
    obj = os.path.join(DEBUG_OBJDIR if debug else OBJDIR, os.path.splitext(src)[0] + ".o")
    extra = ["-DMLSTM_DEBUG"] if debug else []
    cmd = [_hipcc()] + COMMON + NO_PACKED_FP32 + extra + ["-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    # hipcc's host pass does not know the packed-fp32 feature and says so; that is harmless
    return obj


BUILD_INFO = os.path.join(PKG, "build_info.json")


def _write_build_info() -> None:
    """Records the git commit the library was built from (and whether the tree had uncommitted
    changes) next to it, so that a copy of the tree without its .git still says what it runs."""
    import json

    info = {"git_commit": None, "git_dirty": None}
    try:
        r = subprocess.run(["git", "-C", ROOT, "rev-parse", "HEAD"], capture_output=True, text=True, timeout=10)
        if r.returncode == 0:
            info["git_commit"] = r.stdout.strip()
            d = subprocess.run(["git", "-C", ROOT, "status", "--porcelain", "--untracked-files=no"],
                               capture_output=True, text=True, timeout=10)
            info["git_dirty"] = bool(d.stdout.strip()) if d.returncode == 0 else None
    except (OSError, subprocess.SubprocessError):
        pass
    with open(BUILD_INFO, "w") as f:
        json.dump(info, f)


def build(verbose: bool = False, debug: bool = False) -> str:
    """Builds libmlstm.so, or with ``debug`` libmlstm_debug.so (device bounds checks compiled in)."""
    os.makedirs(DEBUG_OBJDIR if debug else OBJDIR, exist_ok=True)
    with cf.ThreadPoolExecutor(min(8, len(SOURCES))) as ex:
        objs = list(ex.map(lambda src: _compile(src, debug), SOURCES))
    target = DEBUG_LIB if debug else LIB
    tmp = target + ".tmp%d" % os.getpid()
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, target)
    if not debug:
        _write_build_info()
    if verbose:
        print(target)
    return target


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
