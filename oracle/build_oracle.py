"""Build ``liboracle_mlstm.so`` from ``mlstm_oracle.c`` with gcc.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).  IEEE fp64: no
fast-math flags, so the C oracle evaluates exactly what it states.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "mlstm_oracle.c")
LIB = os.path.join(HERE, "liboracle_mlstm.so")
# host-sanitized variant (AddressSanitizer + UndefinedBehaviorSanitizer, gcc runtime): a process that
# loads it preloads libasan and sets MLSTM_ORACLE_LIBRARY to its path
LIB_SAN = os.path.join(HERE, "liboracle_mlstm_san.so")
SANITIZE = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer", "-g"]


def build(force: bool = True, sanitize: bool = False) -> str:
    lib = LIB_SAN if sanitize else LIB
    if not force and os.path.exists(lib) and os.path.getmtime(lib) >= os.path.getmtime(SRC):
        return lib
    tmp = lib + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99", "-Wall", "-Wextra",
           "-fno-fast-math", "-ffp-contract=off"] + (SANITIZE if sanitize else []) + [SRC, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(force="--lazy" not in sys.argv, sanitize="--sanitize" in sys.argv))
