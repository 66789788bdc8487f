"""Host-sanitized build of libmlstm: AddressSanitizer and UndefinedBehaviorSanitizer on the host code
(argument validation, workspace arithmetic, launch set-up), for CPU-side checking only.

The device code is compiled exactly as in ``build.py``: every sanitizer flag is preceded by
``-Xarch_host``, so only the host pass is instrumented.  The objects are linked with the host clang
against the shared ASan runtime; a process that loads ``libmlstm_san.so`` must preload that runtime
(``runtime_path()``) and select the library with ``MLSTM_LIBRARY`` (see ``binding.py``).  Nothing on
the GPU path uses this sanitized library.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess
import sys

from . import build as B

OBJDIR = os.path.join(B.PKG, "_build_san")
LIB = os.path.join(B.PKG, "libmlstm_san.so")
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer",
            "-Xarch_host", "-g"]
LINK_SAN = ["-fsanitize=address", "-fsanitize=undefined", "-shared-libasan"]


def runtime_path() -> str:
    """The clang ASan runtime to preload (``LD_PRELOAD``)."""
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not hits:
        raise FileNotFoundError("clang ASan runtime not found under /opt/rocm/llvm")
    return hits[-1]


def _compile(src: str) -> str:
    obj = os.path.join(OBJDIR, os.path.splitext(src)[0] + ".o")
    cmd = [B._hipcc()] + B.COMMON + B.NO_PACKED_FP32 + HOST_SAN + ["-x", "hip", "-c", os.path.join(B.CSRC, src),
                                                                  "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    return obj


def build() -> str:
    os.makedirs(OBJDIR, exist_ok=True)
    with cf.ThreadPoolExecutor(min(8, len(B.SOURCES))) as ex:
        objs = list(ex.map(_compile, B.SOURCES))
    clangxx = os.path.join("/opt/rocm/llvm/bin", "clang++")
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [clangxx, "-shared", "-fPIC"] + LINK_SAN + ["-o", tmp] + objs + ["-L/opt/rocm/lib", "-lamdhip64",
                                                                        "-Wl,-rpath,/opt/rocm/lib"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
    sys.exit(0)
