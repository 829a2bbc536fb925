"""Build the gfx950 shared library ``libplora.so`` in-tree with hipcc.

Each kernel has a source file of its own (``csrc/k_*.hip``), so the device
compiles, which take most of the time, run in parallel; the objects are then
linked into one library with the host side (``csrc/plora.hip``) and the
split-KV attention kernels (``csrc/attention.hip``)."""
from __future__ import annotations

import glob
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
SRCS = sorted(glob.glob(os.path.join(CSRC, "k_*.hip"))) + [
    os.path.join(CSRC, "plora.hip"), os.path.join(CSRC, "attention.hip")]
PROBE_SRC = os.path.join(CSRC, "read_ceiling.hip")
HEADER = os.path.join(ROOT, "include", "plora.h")
LIB = os.path.join(PKG, "libplora.so")
PROBE_LIB = os.path.join(PKG, "libplora_probe.so")
OBJ_DIR = os.path.join(PKG, "_build")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Packed fp32 VALU ops are switched off: hipcc would otherwise form
# v_pk_{add,mul,fma}_f32 from plain float code.
ARCH = ["--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang",
        "-packed-fp32-ops"]
CFLAGS = [*ARCH, "-O3", "-std=c++17", "-fPIC", "-Wall", "-I",
          os.path.join(ROOT, "include"), "-I", CSRC]
NOISE = "is not a recognized feature for this target"


def _run(cmd, verbose: bool) -> None:
    res = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in res.stderr.splitlines() if NOISE not in l)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + " ".join(cmd) + "\n" + err)
    if verbose and err.strip():
        print(err, file=sys.stderr)


def _object(src: str, verbose: bool) -> str:
    os.makedirs(OBJ_DIR, exist_ok=True)
    obj = os.path.join(OBJ_DIR, os.path.basename(src) + ".o")
    tmp = obj + ".tmp%d" % os.getpid()
    _run([HIPCC, *CFLAGS, "-c", src, "-o", tmp], verbose)
    os.replace(tmp, obj)
    return obj


def _link(objs, out: str, verbose: bool) -> str:
    tmp = out + ".tmp%d" % os.getpid()
    _run([HIPCC, *ARCH, "-shared", "-fPIC", *objs, "-o", tmp], verbose)
    os.replace(tmp, out)
    return out


def jobs() -> int:
    return max(1, min(16, len(os.sched_getaffinity(0))))


def build(verbose: bool = False) -> str:
    """Compile every HIP source of the package (always recompiles): the
    product library and the read-ceiling probe the benchmark reports."""
    with ThreadPoolExecutor(max_workers=jobs()) as ex:
        futs = [ex.submit(_object, s, verbose) for s in SRCS + [PROBE_SRC]]
        objs = [f.result() for f in futs]
    _link(objs[:-1], LIB, verbose)
    _link(objs[-1:], PROBE_LIB, verbose)
    return LIB


def is_built() -> bool:
    return os.path.exists(LIB)


# The same library with its host code instrumented by AddressSanitizer (the
# device code is compiled as for the product), for the CPU sanitizer test;
# loaded only with clang's ASan runtime preloaded (its __asan_* symbols are
# left for that runtime to provide).
ASAN_DIR = os.path.join(OBJ_DIR, "asan")
ASAN_LIB = os.path.join(ASAN_DIR, "libplora.so")
ASAN_HOST = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer"]


def _asan_object(src: str, verbose: bool) -> str:
    os.makedirs(ASAN_DIR, exist_ok=True)
    obj = os.path.join(ASAN_DIR, os.path.basename(src) + ".o")
    tmp = obj + ".tmp%d" % os.getpid()
    _run([HIPCC, *CFLAGS, *ASAN_HOST, "-c", src, "-o", tmp], verbose)
    os.replace(tmp, obj)
    return obj


def build_asan(verbose: bool = False) -> str:
    """The host side (plora.hip: argument checks, workspace layout, plans)
    compiled with the sanitizer, linked with the product build's objects of
    the kernel files (whose host code is their launchers), built if absent."""
    host = os.path.join(CSRC, "plora.hip")
    others = [s for s in SRCS if s != host]
    objs = [os.path.join(OBJ_DIR, os.path.basename(s) + ".o") for s in others]
    missing = [s for s, o in zip(others, objs) if not os.path.exists(o)]
    with ThreadPoolExecutor(max_workers=jobs()) as ex:
        futs = [ex.submit(_asan_object, host, verbose)] + \
               [ex.submit(_object, s, verbose) for s in missing]
        asan_host = futs[0].result()
        for f in futs[1:]:
            f.result()
    return _link([asan_host] + objs, ASAN_LIB, verbose)


if __name__ == "__main__":
    print(build(verbose=True))
