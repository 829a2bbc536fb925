"""Build the gfx950 shared library ``libplora.so`` in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SRC = os.path.join(PKG, "csrc", "plora.hip")
ATTN_SRC = os.path.join(PKG, "csrc", "attention.hip")
PROBE_SRC = os.path.join(PKG, "csrc", "read_ceiling.hip")
HEADER = os.path.join(ROOT, "include", "plora.h")
LIB = os.path.join(PKG, "libplora.so")
PROBE_LIB = os.path.join(PKG, "libplora_probe.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Packed fp32 VALU ops are switched off: hipcc would otherwise form
# v_pk_{add,mul,fma}_f32 from plain float code.
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
         "-Wall", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _hipcc(srcs, out: str, verbose: bool) -> str:
    tmp = out + ".tmp%d" % os.getpid()
    srcs = [srcs] if isinstance(srcs, str) else list(srcs)
    cmd = [HIPCC, *FLAGS, "-I", os.path.join(ROOT, "include"), *srcs, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in res.stderr.splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + err)
    if verbose and err.strip():
        print(err, file=sys.stderr)
    os.replace(tmp, out)
    return out


def build(verbose: bool = False) -> str:
    """Compile every HIP source of the package (always recompiles): the
    product library and the read-ceiling probe the benchmark reports."""
    _hipcc([SRC, ATTN_SRC], LIB, verbose)
    _hipcc(PROBE_SRC, PROBE_LIB, verbose)
    return LIB


def is_built() -> bool:
    return os.path.exists(LIB)


if __name__ == "__main__":
    print(build(verbose=True))
