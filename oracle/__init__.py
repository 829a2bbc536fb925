"""CPU oracle for the batched heterogeneous-adapter LoRA apply.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product
library (``paper_2608_05483_amd``) never imports it, and the two share no
code: this package wraps ``plora_oracle.c``, a plain fp32 C implementation
of the paper's definition (section II-A, y = x(W + AB); section V-A, the four
strategies that all compute the same y), loaded through ctypes.

Every function takes numpy arrays holding bf16 bit patterns (uint16), int32
ids and ranks, int64 element offsets and fp32 scales, and returns numpy
arrays.  See ``plora_oracle.c`` for the exact arithmetic and the readings of
the paper it takes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "plora_oracle.c")
_LIB = os.path.join(_HERE, "libplora_oracle.so")
# AddressSanitizer build (clang, its ASan runtime preloaded by the caller;
# single-threaded: the results do not depend on the thread count)
ASAN_LIB = os.path.join(_HERE, "_build", "asan", "libplora_oracle.so")
ASAN_CC = "/opt/rocm/llvm/bin/clang"

# -O2 with no FMA contraction and no fast-math: each product and each sum is
# rounded exactly once, in the order the source states.
CFLAGS = ["-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-fPIC",
          "-shared", "-std=c11", "-Wall", "-Wextra"]


def build(force: bool = True) -> str:
    """Compile the oracle with gcc into ``oracle/libplora_oracle.so``."""
    if not force and os.path.exists(_LIB) and \
            os.path.getmtime(_LIB) >= os.path.getmtime(_SRC):
        return _LIB
    tmp = _LIB + ".tmp%d" % os.getpid()
    subprocess.check_call(["gcc", *CFLAGS, _SRC, "-o", tmp, "-lm"])
    os.replace(tmp, _LIB)
    return _LIB


def build_asan() -> str:
    """Compile the oracle with AddressSanitizer into oracle/_build/asan."""
    os.makedirs(os.path.dirname(ASAN_LIB), exist_ok=True)
    tmp = ASAN_LIB + ".tmp%d" % os.getpid()
    flags = [f for f in CFLAGS if f not in ("-fopenmp", "-O2")]
    subprocess.check_call([ASAN_CC, "-O1", "-g", "-fsanitize=address",
                           "-fno-omit-frame-pointer", *flags, _SRC, "-o", tmp, "-lm"])
    os.replace(tmp, ASAN_LIB)
    return ASAN_LIB


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        # PLORA_ORACLE_LIB names another build to load (the sanitizer test's)
        path = os.environ.get("PLORA_ORACLE_LIB") or build(force=False)
        L = ctypes.CDLL(path)
        P = ctypes.c_void_p
        i32, i64 = ctypes.c_int32, ctypes.c_int64
        L.oracle_segment.argtypes = [P, i32, i32, P, P, P, P, P]
        L.oracle_segment.restype = ctypes.c_int
        L.oracle_shrink.argtypes = [P, i64, i32, P, i32, i32, P, P, P, P, i64, i32]
        L.oracle_shrink.restype = None
        L.oracle_expand.argtypes = [P, i64, i32, P, i32, i32, P, P, P, P, P, i64,
                                    P, P, i32]
        L.oracle_expand.restype = None
        L.oracle_apply.argtypes = [P, i64, i32, P, i32, i32, i32, P, P, P, P, P,
                                   P, P, i64, P, P, i32]
        L.oracle_apply.restype = ctypes.c_int
        L.oracle_apply_grouped.argtypes = [P, i64, i32, P, P, P, i32, i32, i32,
                                           i32, P, P, P, P, P, P, P, i64, P, P,
                                           P, i32]
        L.oracle_apply_grouped.restype = ctypes.c_int
        L.oracle_bf16_decode.argtypes = [P, P, i64]
        L.oracle_bf16_encode.argtypes = [P, P, i64]
        L.oracle_max_threads.argtypes = []
        L.oracle_max_threads.restype = ctypes.c_int
        _lib = L
    return _lib


def _p(a: np.ndarray | None):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(np.asarray(a, dtype=dtype))


def max_threads() -> int:
    return int(lib().oracle_max_threads())


def bf16_to_f32(bits) -> np.ndarray:
    """Exact bf16 -> fp32 decode (the bits become the high half)."""
    b = _c(bits, np.uint16)
    out = np.empty(b.shape, np.float32)
    lib().oracle_bf16_decode(_p(b), _p(out), b.size)
    return out


def f32_to_bf16(values) -> np.ndarray:
    """fp32 -> bf16 bits, round to nearest, ties to even."""
    v = _c(values, np.float32)
    out = np.empty(v.shape, np.uint16)
    lib().oracle_bf16_encode(_p(v), _p(out), v.size)
    return out


@dataclass
class Segments:
    perm: np.ndarray     # int32[T]
    seg_ptr: np.ndarray  # int32[cap + 1]
    seg_id: np.ndarray   # int32[cap]
    meta: np.ndarray     # int32[4] = n_seg, n_valid, n_none, n_invalid

    @property
    def n_seg(self) -> int:
        return int(self.meta[0])


def segment(idx, n_adapters: int) -> Segments:
    """Counting-sort segmentation (per-adapter batches, section VI-B)."""
    idx = _c(idx, np.int32)
    T = idx.size
    cap = min(T, n_adapters)
    perm = np.empty(T, np.int32)
    seg_ptr = np.empty(cap + 1, np.int32)
    seg_id = np.empty(max(cap, 0), np.int32)
    meta = np.empty(4, np.int32)
    hist = np.empty(n_adapters + 1, np.int32)
    rc = lib().oracle_segment(_p(idx), T, n_adapters, _p(perm), _p(seg_ptr),
                              _p(seg_id), _p(meta), _p(hist))
    if rc != 0:
        raise RuntimeError("oracle_segment failed")
    return Segments(perm, seg_ptr, seg_id, meta)


def shrink(x, idx, A, a_off, ranks, h_in: int, ldv: int | None = None,
           n_threads: int = 1, fill=np.nan) -> np.ndarray:
    """v[t, c] = sum_k x[t, k] A_i[k, c] in fp32 (strategy E4's m = xA)."""
    x = _c(x, np.uint16)
    idx = _c(idx, np.int32)
    ranks = _c(ranks, np.int32)
    T = idx.size
    N = ranks.size
    if ldv is None:
        ldv = int(ranks.max()) if N else 0
        ldv = max(ldv, 1)
    v = np.full((T, ldv), fill, np.float32)
    lib().oracle_shrink(_p(x), x.shape[1] if x.ndim == 2 else h_in, T, _p(idx),
                        N, h_in, _p(_c(A, np.uint16)), _p(_c(a_off, np.int64)),
                        _p(ranks), _p(v), ldv, n_threads)
    return v


def expand(v, idx, B, b_off, ranks, scales, y_in, h_out: int,
           n_threads: int = 1):
    """Returns (yref fp32, y bf16 bits): y_in + s_i v B_i per valid token."""
    v = _c(v, np.float32)
    idx = _c(idx, np.int32)
    ranks = _c(ranks, np.int32)
    y_in = _c(y_in, np.uint16)
    T = idx.size
    yref = np.empty((T, h_out), np.float32)
    yout = np.empty((T, h_out), np.uint16)
    lib().oracle_expand(_p(v), v.shape[1], T, _p(idx), ranks.size, h_out,
                        _p(_c(B, np.uint16)), _p(_c(b_off, np.int64)), _p(ranks),
                        _p(_c(scales, np.float32)), _p(y_in), y_in.shape[1],
                        _p(yref), _p(yout), n_threads)
    return yref, yout


def apply(x, idx, A, a_off, B, b_off, ranks, scales, y_base, h_in: int,
          h_out: int, n_threads: int = 1):
    """Per-token apply; returns (yref fp32, y bf16 bits)."""
    x = _c(x, np.uint16)
    idx = _c(idx, np.int32)
    ranks = _c(ranks, np.int32)
    y_base = _c(y_base, np.uint16)
    T = idx.size
    yref = np.empty((T, h_out), np.float32)
    yout = np.empty((T, h_out), np.uint16)
    rc = lib().oracle_apply(_p(x), x.shape[1] if T else h_in, T, _p(idx),
                            ranks.size, h_in, h_out, _p(_c(A, np.uint16)),
                            _p(_c(a_off, np.int64)), _p(_c(B, np.uint16)),
                            _p(_c(b_off, np.int64)), _p(ranks),
                            _p(_c(scales, np.float32)), _p(y_base),
                            y_base.shape[1] if T else h_out, _p(yref), _p(yout),
                            n_threads)
    if rc != 0:
        raise RuntimeError("oracle_apply: rank above the oracle's limit")
    return yref, yout


def apply_grouped(x, idx, A, a_off, B, b_off, ranks, scales, y_base,
                  h_in: int, h_out: int, segs: Segments | None = None):
    """Grouped apply over oracle segments; returns (yref fp32, y bf16)."""
    x = _c(x, np.uint16)
    idx = _c(idx, np.int32)
    ranks = _c(ranks, np.int32)
    y_base = _c(y_base, np.uint16)
    T = idx.size
    if segs is None:
        segs = segment(idx, ranks.size)
    n_seg = segs.n_seg
    longest = int(np.max(np.diff(segs.seg_ptr[:n_seg + 1]))) if n_seg else 1
    max_rank = max(int(ranks.max()) if ranks.size else 1, 1)
    scratch = np.empty(longest * max_rank, np.float32)
    yref = np.empty((T, h_out), np.float32)
    yout = np.empty((T, h_out), np.uint16)
    rc = lib().oracle_apply_grouped(
        _p(x), x.shape[1] if T else h_in, T, _p(segs.perm), _p(segs.seg_ptr),
        _p(segs.seg_id), n_seg, ranks.size, h_in, h_out, _p(_c(A, np.uint16)),
        _p(_c(a_off, np.int64)), _p(_c(B, np.uint16)), _p(_c(b_off, np.int64)),
        _p(ranks), _p(_c(scales, np.float32)), _p(y_base),
        y_base.shape[1] if T else h_out, _p(yref), _p(yout), _p(scratch),
        max_rank)
    if rc != 0:
        raise RuntimeError("oracle_apply_grouped failed")
    return yref, yout


def apply_multi(x, idx, stacks, y_bases, h_in: int, n_threads: int = 1):
    """The apply for several projections of one layer that read the same x
    and token ids (section VII-A attaches adapters to the attention
    projections and the FFN; section II-A gives each its own A and B): each
    projection is the single-projection definition on its own stack.

    stacks: per projection a tuple (A, a_off, B, b_off, ranks, scales, h_out);
    y_bases: per projection its y_base.  Returns a list of (yref, y bf16)."""
    return [apply(x, idx, A, a_off, B, b_off, ranks, scales, yb, h_in, h_out,
                  n_threads=n_threads)
            for (A, a_off, B, b_off, ranks, scales, h_out), yb in zip(stacks, y_bases)]
