"""The oracle's pins under AddressSanitizer and UndefinedBehaviorSanitizer.

A child process builds oracle.c with -fsanitize=address,undefined (every
finding aborts the process), preloads the ASan runtime and runs the oracle's
pin tests against that build: no out-of-bounds access, use of freed memory,
signed overflow, misaligned access or other undefined behaviour in any path
the pins exercise (1-D and nd shares, every signature and product, the fp32
loop, the attention products, bf16 rounding, argument checks). The planted-
mistake tests are left out (they compile mutated copies of their own).
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _runtime(name):
    r = subprocess.run(["gcc", "-print-file-name=" + name], capture_output=True, text=True)
    path = r.stdout.strip()
    return path if r.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


def test_oracle_pins_under_asan_and_ubsan():
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("gcc's ASan runtime is not installed")
    env = dict(os.environ, ORACLE_SANITIZE="1", LD_PRELOAD=asan,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", OMP_NUM_THREADS="2")
    cmd = [sys.executable, "-m", "pytest", "-x", "-q", "-s", "-p", "no:cacheprovider",
           "-k", "not planted",
           "tests/test_oracle_pins.py", "tests/test_oracle_nd_pins.py",
           "tests/test_oracle_attn_pins.py", "tests/test_oracle_search_pins.py"]
    r = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert " passed" in out, out[-2000:]
