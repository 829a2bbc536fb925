"""The host side of the library and the CPU oracle under AddressSanitizer.

Both are built with ASan (the library's host code by hipcc with the
sanitizer on the host side only, the oracle by clang), and the oracle's pins
and the library's host checks (test_oracle_pins.py, test_abi.py) run against
those builds in a child process with clang's ASan runtime preloaded.  Any
out-of-bounds access, use after free or double free in the host argument
checks, the workspace sizing or the oracle ends the child with an ASan
report.  No GPU is used: the host checks return before any launch."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2608_05483_amd import build as B  # noqa: E402


def _asan_runtime():
    try:
        out = subprocess.run([oracle.ASAN_CC, "-print-file-name=libclang_rt.asan-x86_64.so"],
                             capture_output=True, text=True, check=True).stdout.strip()
    except (OSError, subprocess.CalledProcessError):
        return None
    return out if os.path.isabs(out) and os.path.exists(out) else None


def test_oracle_and_host_checks_under_asan():
    rt = _asan_runtime()
    if rt is None:
        pytest.skip("clang's AddressSanitizer runtime is not installed")
    lib = B.build_asan()
    olib = oracle.build_asan()
    env = dict(os.environ, LD_PRELOAD=rt, PLORA_LIB=lib, PLORA_ORACLE_LIB=olib,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0")
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                          "-m", "not gpu", os.path.join(ROOT, "tests", "test_oracle_pins.py"),
                          os.path.join(ROOT, "tests", "test_abi.py")],
                         cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = res.stdout + res.stderr
    assert "AddressSanitizer" not in out, out[-4000:]
    assert res.returncode == 0, out[-4000:]
    assert " passed" in res.stdout
