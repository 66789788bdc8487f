"""Host-code sanitizers (CPU only): the library's argument validation and launch set-up built with
AddressSanitizer + UndefinedBehaviorSanitizer (``paper_2503_13427_amd/build_sanitize.py``, host pass
only) runs the C-ABI validation suite, and the C oracle built with the same sanitizers (gcc) runs the
oracle pins.  Each suite runs in a child process that preloads its sanitizer runtime (clang's for the
hipcc-built library, gcc's for the oracle: the two cannot share a process) and stops at the first
report (``halt_on_error``); leak checking is off (the interpreter itself does not free everything)."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(args, env_extra, timeout=600):
    env = dict(os.environ)
    env.update(env_extra)
    env.update(ASAN_OPTIONS="detect_leaks=0:alloc_dealloc_mismatch=0:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-s", "-p", "no:cacheprovider"] + args, cwd=ROOT,
                       env=env, capture_output=True, text=True, timeout=timeout)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    return out


@pytest.mark.skipif(shutil.which("/opt/rocm/bin/hipcc") is None and shutil.which("hipcc") is None,
                    reason="hipcc is not available")
def test_abi_validation_under_asan_ubsan():
    from paper_2503_13427_amd import build_sanitize
    lib = build_sanitize.build()
    out = _run(["tests/test_abi_cpu.py"], {"LD_PRELOAD": build_sanitize.runtime_path(), "MLSTM_LIBRARY": lib})
    assert " passed" in out


def test_oracle_under_asan_ubsan():
    from oracle import build_oracle
    lib = build_oracle.build(force=True, sanitize=True)
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    out = _run(["tests/test_oracle_pins.py", "-m", "not gpu"], {"LD_PRELOAD": asan, "MLSTM_ORACLE_LIBRARY": lib})
    assert " passed" in out
