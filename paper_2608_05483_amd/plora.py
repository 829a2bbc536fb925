"""Thin Python binding of ``libplora.so`` (include/plora.h).

Argument marshalling only: every function forwards raw device pointers,
sizes and the caller's HIP stream to the C ABI of the same name and raises
``PloraError`` on a non-OK status.  torch is used for device memory and
streams; the helper classes at the bottom allocate the buffers a call needs
as torch tensors and fill the ABI structs from them.

Importing this module loads the HIP library and fails loudly if it has not
been built (``python -m paper_2608_05483_amd.build``); there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

from . import build as _build

PLORA_OK = 0
PLORA_ERR_INVALID_ARG = 1
PLORA_ERR_UNSUPPORTED = 2
PLORA_ERR_WORKSPACE_TOO_SMALL = 3
PLORA_ERR_HIP = 4
PLORA_MAX_RANK = 128
PLORA_MAX_TOKENS = 16384
PLORA_TILE_TOKENS = 32
PLORA_SMALL_BATCH_TILE_TOKENS = 2
PLORA_DECODE_TILE_TOKENS = 1


def tile_tokens(T: int) -> int:
    """Tokens per tile of a batch of T tokens (include/plora.h)."""
    if T <= 64:
        return PLORA_DECODE_TILE_TOKENS
    return PLORA_SMALL_BATCH_TILE_TOKENS if T <= 256 else PLORA_TILE_TOKENS
PLORA_META_WORDS = 8
PLORA_MAX_PROJECTIONS = 8

EXPORTED = ("plora_tile_capacity", "plora_workspace_bytes", "plora_workspace_init",
            "plora_segment", "plora_shrink", "plora_expand", "plora_apply",
            "plora_segment_apply", "plora_segment_apply_launches",
            "plora_apply_multi", "plora_workspace_bytes_multi",
            "plora_check_adapters", "plora_status_string",
            "plora_debug_last_hip_error", "plora_debug_set_exchange_polls",
            "plora_pool_device_pointer", "plora_workspace_counters",
            "plora_segment_apply_noalloc", "plora_segment_workspace_bytes",
            # include/plora_attention.h
            "plora_attn_partitions", "plora_attn_workspace_bytes", "plora_attn_partial",
            "plora_attn_merge", "plora_attn_decode")


class PloraError(RuntimeError):
    def __init__(self, fn: str, status: int):
        msg = f"{fn}: {status_string(status)}"
        if status == PLORA_ERR_HIP:
            msg += f" (hipError_t {int(lib.plora_debug_last_hip_error())})"
        super().__init__(msg)
        self.status = status


class plora_adapters(ctypes.Structure):
    _fields_ = [("n_adapters", ctypes.c_int32), ("h_in", ctypes.c_int32),
                ("h_out", ctypes.c_int32), ("max_rank", ctypes.c_int32),
                ("A", ctypes.c_void_p), ("B", ctypes.c_void_p),
                ("a_len", ctypes.c_int64), ("b_len", ctypes.c_int64),
                ("a_off", ctypes.c_void_p), ("b_off", ctypes.c_void_p),
                ("ranks", ctypes.c_void_p), ("scales", ctypes.c_void_p),
                ("A_pool", ctypes.c_void_p), ("B_pool", ctypes.c_void_p),
                ("a_pool_len", ctypes.c_int64), ("b_pool_len", ctypes.c_int64)]


class plora_segments(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int32), ("cap", ctypes.c_int32),
                ("tile_cap", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("perm", ctypes.c_void_p), ("seg_ptr", ctypes.c_void_p),
                ("seg_id", ctypes.c_void_p), ("meta", ctypes.c_void_p),
                ("tiles", ctypes.c_void_p)]


# PLORA_LIB names another build of the library to load instead (the
# sanitizer test loads the AddressSanitizer build this way).
LIB_PATH = os.environ.get("PLORA_LIB") or _build.LIB


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is not built; run `python -m paper_2608_05483_amd.build`")
    # torch ships its own libamdhip64 whose dependants name it without the
    # ".7" suffix; if this library (linked against the system runtime) were
    # loaded first, the process would end up with two HIP runtimes and torch's
    # streams and allocations would be foreign to our launches.  Loading torch
    # first makes the dynamic linker bind libplora.so to torch's runtime.
    import torch  # noqa: F401
    L = ctypes.CDLL(LIB_PATH)
    P, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    AD, SG = ctypes.POINTER(plora_adapters), ctypes.POINTER(plora_segments)
    L.plora_tile_capacity.argtypes = [i32, i32]
    L.plora_tile_capacity.restype = i32
    L.plora_workspace_bytes.argtypes = [i32, AD]
    L.plora_workspace_bytes.restype = sz
    L.plora_workspace_init.argtypes = [P, sz, P]
    L.plora_segment.argtypes = [P, SG, i32, P, sz, P]
    L.plora_segment_workspace_bytes.argtypes = [i32, i32]
    L.plora_segment_workspace_bytes.restype = sz
    L.plora_shrink.argtypes = [P, i64, AD, SG, P, i64, P, sz, P]
    L.plora_expand.argtypes = [P, i64, AD, SG, P, i64, P, sz, P]
    L.plora_apply.argtypes = [P, i64, AD, SG, P, i64, P, sz, P]
    L.plora_segment_apply.argtypes = [P, P, i64, AD, SG, P, i64, P, sz, P]
    L.plora_segment_apply_noalloc.argtypes = [P, P, i64, AD, SG, P, i64, P]
    L.plora_segment_apply_noalloc.restype = ctypes.c_int
    L.plora_segment_apply_launches.argtypes = [i32, AD]
    L.plora_segment_apply_launches.restype = i32
    L.plora_apply_multi.argtypes = [P, i64, AD, i32, SG, ctypes.POINTER(P),
                                    ctypes.POINTER(i64), P, sz, P]
    L.plora_workspace_bytes_multi.argtypes = [i32, AD, i32]
    L.plora_workspace_bytes_multi.restype = sz
    L.plora_check_adapters.argtypes = [AD, ctypes.POINTER(i32), P]
    L.plora_status_string.argtypes = [ctypes.c_int]
    L.plora_status_string.restype = ctypes.c_char_p
    L.plora_debug_last_hip_error.argtypes = []
    L.plora_debug_last_hip_error.restype = i32
    L.plora_pool_device_pointer.argtypes = [P, ctypes.POINTER(P)]
    L.plora_pool_device_pointer.restype = ctypes.c_int
    L.plora_workspace_counters.argtypes = [P, sz, ctypes.POINTER(i64), P]
    L.plora_workspace_counters.restype = ctypes.c_int
    L.plora_debug_set_exchange_polls.argtypes = [i32]
    L.plora_debug_set_exchange_polls.restype = None
    L.plora_attn_partitions.argtypes = [i64]
    L.plora_attn_partitions.restype = i32
    L.plora_attn_workspace_bytes.argtypes = [i32, i32, i64]
    L.plora_attn_workspace_bytes.restype = sz
    F = ctypes.c_float
    L.plora_attn_partial.argtypes = [P, P, P, P, i32, i32, i64, F, P, P, P, P]
    L.plora_attn_merge.argtypes = [P, P, P, P, i32, i32, i64, P, P]
    L.plora_attn_decode.argtypes = [P, P, P, P, i32, i32, i64, F, P, P, sz, P]
    for fn in ("plora_attn_partial", "plora_attn_merge", "plora_attn_decode"):
        getattr(L, fn).restype = ctypes.c_int
    for fn in ("plora_workspace_init", "plora_segment", "plora_shrink",
               "plora_expand", "plora_apply", "plora_segment_apply", "plora_apply_multi",
               "plora_check_adapters"):
        getattr(L, fn).restype = ctypes.c_int
    return L


lib = _load()


def _ok(fn: str, status: int) -> None:
    if status != PLORA_OK:
        raise PloraError(fn, status)


def status_string(status: int) -> str:
    return lib.plora_status_string(status).decode()


# ---- the C ABI, one Python function per entry point -------------------------

def plora_tile_capacity(T: int, n_adapters: int) -> int:
    return int(lib.plora_tile_capacity(T, n_adapters))


def plora_workspace_bytes(T: int, ad: plora_adapters) -> int:
    return int(lib.plora_workspace_bytes(T, ctypes.byref(ad)))


def plora_workspace_init(ws: int, ws_bytes: int, stream: int) -> None:
    _ok("plora_workspace_init", lib.plora_workspace_init(ws, ws_bytes, stream))


def plora_segment_workspace_bytes(T: int, n_adapters: int) -> int:
    return int(lib.plora_segment_workspace_bytes(T, n_adapters))


def plora_segment(idx: int, seg: plora_segments, n_adapters: int, ws: int | None,
                  ws_bytes: int, stream: int) -> None:
    _ok("plora_segment", lib.plora_segment(idx, ctypes.byref(seg), n_adapters, ws,
                                           ws_bytes, stream))


def plora_shrink(x: int, ldx: int, ad: plora_adapters, seg: plora_segments, v: int,
                 ldv: int, ws: int, ws_bytes: int, stream: int) -> None:
    _ok("plora_shrink", lib.plora_shrink(x, ldx, ctypes.byref(ad), ctypes.byref(seg),
                                         v, ldv, ws, ws_bytes, stream))


def plora_expand(v: int, ldv: int, ad: plora_adapters, seg: plora_segments, y: int,
                 ldy: int, ws: int | None, ws_bytes: int, stream: int) -> None:
    _ok("plora_expand", lib.plora_expand(v, ldv, ctypes.byref(ad), ctypes.byref(seg),
                                         y, ldy, ws, ws_bytes, stream))


def plora_apply(x: int, ldx: int, ad: plora_adapters, seg: plora_segments, y: int,
                ldy: int, ws: int, ws_bytes: int, stream: int) -> None:
    _ok("plora_apply", lib.plora_apply(x, ldx, ctypes.byref(ad), ctypes.byref(seg),
                                       y, ldy, ws, ws_bytes, stream))


def plora_segment_apply(idx: int, x: int, ldx: int, ad: plora_adapters, seg: plora_segments,
                        y: int, ldy: int, ws: int, ws_bytes: int, stream: int) -> None:
    _ok("plora_segment_apply",
        lib.plora_segment_apply(idx, x, ldx, ctypes.byref(ad), ctypes.byref(seg), y, ldy, ws,
                                ws_bytes, stream))


def plora_segment_apply_noalloc(idx: int, x: int, ldx: int, ad: plora_adapters,
                                seg: plora_segments, y: int, ldy: int, stream: int) -> None:
    _ok("plora_segment_apply_noalloc",
        lib.plora_segment_apply_noalloc(idx, x, ldx, ctypes.byref(ad), ctypes.byref(seg), y,
                                        ldy, stream))


def plora_segment_apply_launches(T: int, ad: plora_adapters) -> int:
    return int(lib.plora_segment_apply_launches(T, ctypes.byref(ad)))


def _stack_array(ads):
    arr = (plora_adapters * len(ads))()
    for i, a in enumerate(ads):
        arr[i] = a
    return arr


def plora_workspace_bytes_multi(T: int, ads) -> int:
    """ads: a sequence of plora_adapters structs."""
    return int(lib.plora_workspace_bytes_multi(T, _stack_array(ads), len(ads)))


def plora_apply_multi(x: int, ldx: int, ads, seg: plora_segments, ys, ldys, ws: int,
                      ws_bytes: int, stream: int) -> None:
    """ads: plora_adapters structs; ys, ldys: device pointers and leading
    dimensions, one per projection."""
    n = len(ads)
    yarr = (ctypes.c_void_p * n)(*ys)
    larr = (ctypes.c_int64 * n)(*ldys)
    _ok("plora_apply_multi", lib.plora_apply_multi(x, ldx, _stack_array(ads), n,
                                                   ctypes.byref(seg), yarr, larr, ws,
                                                   ws_bytes, stream))


def plora_pool_device_pointer(host: int) -> int:
    d = ctypes.c_void_p()
    _ok("plora_pool_device_pointer", lib.plora_pool_device_pointer(host, ctypes.byref(d)))
    return int(d.value)


def plora_workspace_counters(ws: int, ws_bytes: int, stream: int) -> tuple:
    """(work items that computed v alone, tokens skipped for an unusable
    adapter entry), counted since the workspace was zeroed.  Synchronous."""
    out = (ctypes.c_int64 * 2)()
    _ok("plora_workspace_counters", lib.plora_workspace_counters(ws, ws_bytes, out, stream))
    return int(out[0]), int(out[1])


def plora_debug_set_exchange_polls(polls: int) -> None:
    lib.plora_debug_set_exchange_polls(polls)


def plora_check_adapters(ad: plora_adapters, stream: int) -> int:
    """-1 if every adapter entry is usable, else the first bad index."""
    bad = ctypes.c_int32(-1)
    st = lib.plora_check_adapters(ctypes.byref(ad), ctypes.byref(bad), stream)
    if st == PLORA_ERR_INVALID_ARG and bad.value >= 0:
        return bad.value
    _ok("plora_check_adapters", st)
    return -1


# ---- torch-backed buffers ----------------------------------------------------

def _stream(stream=None) -> int:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


class Adapters:
    """Device-resident adapter stack and its ABI struct."""

    def __init__(self, A, B, a_off, b_off, ranks, scales, h_in: int, h_out: int,
                 max_rank: int, A_pool=None, B_pool=None):
        """A_pool / B_pool: optional pinned host tensors that negative offsets
        name (element -1 - o)."""
        self.A, self.B = A, B
        self.A_pool, self.B_pool = A_pool, B_pool
        self.a_off, self.b_off, self.ranks, self.scales = a_off, b_off, ranks, scales
        self.h_in, self.h_out, self.max_rank = h_in, h_out, max_rank
        self.n_adapters = int(ranks.numel())
        ptr = lambda t: t.data_ptr() if t is not None else None
        # pools: the device address of the pinned host memory (refused if the
        # memory is not pinned and mapped)
        pool = lambda t: plora_pool_device_pointer(t.data_ptr()) if t is not None else None
        self.struct = plora_adapters(
            self.n_adapters, h_in, h_out, max_rank, ptr(A), ptr(B),
            A.numel() if A is not None else 0, B.numel() if B is not None else 0,
            a_off.data_ptr(), b_off.data_ptr(), ranks.data_ptr(), scales.data_ptr(),
            pool(A_pool), pool(B_pool), A_pool.numel() if A_pool is not None else 0,
            B_pool.numel() if B_pool is not None else 0)

    @classmethod
    def from_arrays(cls, A, B, a_off, b_off, ranks, scales, h_in, h_out,
                    max_rank=None, device="cuda"):
        import numpy as np
        import torch
        t = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(device=device,
                                                                       dtype=dt)
        ranks_np = np.asarray(ranks, np.int32)
        if max_rank is None:
            mr = int(ranks_np.max()) if ranks_np.size else 8
            max_rank = max(8, (mr + 7) // 8 * 8)
        return cls(t(np.asarray(A, np.uint16).view(np.int16), torch.int16),
                   t(np.asarray(B, np.uint16).view(np.int16), torch.int16),
                   t(np.asarray(a_off, np.int64), torch.int64),
                   t(np.asarray(b_off, np.int64), torch.int64),
                   t(ranks_np, torch.int32), t(np.asarray(scales, np.float32),
                                               torch.float32),
                   h_in, h_out, max_rank)

    @classmethod
    def from_workload(cls, w, device="cuda"):
        return cls.from_arrays(w.A, w.B, w.a_off, w.b_off, w.ranks, w.scales,
                               w.h_in, w.h_out, device=device)


class Segments:
    """Device buffers of one token batch's grouping and its ABI struct."""

    def __init__(self, T: int, n_adapters: int, device="cuda"):
        import torch
        self.T, self.n_adapters = T, n_adapters
        self.cap = min(T, n_adapters)
        self.tile_cap = plora_tile_capacity(T, n_adapters)
        i32 = dict(dtype=torch.int32, device=device)
        self.perm = torch.empty(max(T, 1), **i32)
        self.seg_ptr = torch.empty(self.cap + 1, **i32)
        self.seg_id = torch.empty(max(self.cap, 1), **i32)
        self.meta = torch.zeros(PLORA_META_WORDS, **i32)
        self.tiles = torch.empty(max(self.tile_cap, 1) * 4, **i32)
        self.struct = plora_segments(T, self.cap, self.tile_cap, 0,
                                     self.perm.data_ptr(), self.seg_ptr.data_ptr(),
                                     self.seg_id.data_ptr(), self.meta.data_ptr(),
                                     self.tiles.data_ptr())


class Workspace:
    """Zero-initialised workspace of plora_workspace_bytes(T, stack) bytes, or
    plora_workspace_bytes_multi(T, stacks) for a list of stacks."""

    def __init__(self, T: int, ad, device="cuda", stream=None):
        import torch
        if isinstance(ad, (list, tuple)):
            self.nbytes = plora_workspace_bytes_multi(T, [a.struct for a in ad])
        else:
            self.nbytes = plora_workspace_bytes(T, ad.struct)
        self.buf = None
        if self.nbytes:
            self.buf = torch.empty(self.nbytes, dtype=torch.uint8, device=device)
            plora_workspace_init(self.buf.data_ptr(), self.nbytes, _stream(stream))

    @property
    def ptr(self) -> int | None:
        return self.buf.data_ptr() if self.buf is not None else None

    def counters(self, stream=None) -> tuple:
        """(exchange give-ups, skipped tokens) since the workspace was zeroed."""
        return plora_workspace_counters(self.ptr, self.nbytes, _stream(stream))


def segment(idx, segs: Segments, stream=None, ws=None) -> None:
    """ws: an optional uint8 tensor (or Workspace) of at least
    plora_segment_workspace_bytes bytes, for the many-work-group form."""
    if isinstance(ws, Workspace):
        ptr, n = ws.ptr, ws.nbytes
    elif ws is not None:
        ptr, n = ws.data_ptr(), ws.numel() * ws.element_size()
    else:
        ptr, n = None, 0
    plora_segment(idx.data_ptr(), segs.struct, segs.n_adapters, ptr, n, _stream(stream))


def shrink(x, ad: Adapters, segs: Segments, v, ws: Workspace, stream=None) -> None:
    plora_shrink(x.data_ptr(), x.stride(0), ad.struct, segs.struct, v.data_ptr(),
                 v.stride(0), ws.ptr, ws.nbytes, _stream(stream))


def expand(v, ad: Adapters, segs: Segments, y, stream=None, ws: Workspace | None = None) -> None:
    """ws is optional: given, the call counts skipped tokens into it."""
    plora_expand(v.data_ptr(), v.stride(0), ad.struct, segs.struct, y.data_ptr(),
                 y.stride(0), ws.ptr if ws is not None else None,
                 ws.nbytes if ws is not None else 0, _stream(stream))


def apply(x, ad: Adapters, segs: Segments, y, ws: Workspace, stream=None) -> None:
    plora_apply(x.data_ptr(), x.stride(0), ad.struct, segs.struct, y.data_ptr(),
                y.stride(0), ws.ptr, ws.nbytes, _stream(stream))


def segment_apply(idx, x, ad: Adapters, segs: Segments, y, ws: Workspace, stream=None) -> None:
    """segment() then apply() on the same batch, as one call."""
    plora_segment_apply(idx.data_ptr(), x.data_ptr(), x.stride(0), ad.struct, segs.struct,
                        y.data_ptr(), y.stride(0), ws.ptr, ws.nbytes, _stream(stream))


def segment_apply_noalloc(idx, x, ad: Adapters, segs: Segments, y, stream=None) -> None:
    """segment_apply() without a workspace: the library's static one (at
    most 256 tokens; calls on one GPU must not overlap)."""
    plora_segment_apply_noalloc(idx.data_ptr(), x.data_ptr(), x.stride(0), ad.struct,
                                segs.struct, y.data_ptr(), y.stride(0), _stream(stream))


# ---- split-KV decode attention (include/plora_attention.h) --------------------

ATTN_HEAD_DIM = 128
ATTN_CHUNK = 256


def attn_partitions(max_len: int) -> int:
    return int(lib.plora_attn_partitions(max_len))


def attn_workspace_bytes(batch: int, heads: int, max_len: int) -> int:
    return int(lib.plora_attn_workspace_bytes(batch, heads, max_len))


def attn_partial(q, k, v, lens, scale: float, m, l, o, stream=None) -> None:
    """q [B, H, 128], k / v [B, H, Lmax, 128] (bf16 bits as int16 tensors),
    lens int32 [B]; m, l float32 [B, H, P], o float32 [B, H, P, 128]."""
    Bn, H, Lmax = k.shape[0], k.shape[1], k.shape[2]
    _ok("plora_attn_partial", lib.plora_attn_partial(
        q.data_ptr(), k.data_ptr(), v.data_ptr(), lens.data_ptr(), Bn, H, Lmax, scale,
        m.data_ptr(), l.data_ptr(), o.data_ptr(), _stream(stream)))


def attn_merge(m, l, o, lens, out, max_len: int, stream=None) -> None:
    Bn, H = m.shape[0], m.shape[1]
    _ok("plora_attn_merge", lib.plora_attn_merge(
        m.data_ptr(), l.data_ptr(), o.data_ptr(), lens.data_ptr(), Bn, H, max_len,
        out.data_ptr(), _stream(stream)))


def attn_decode(q, k, v, lens, scale: float, out, ws, stream=None) -> None:
    """ws: a uint8 tensor of at least attn_workspace_bytes bytes."""
    Bn, H, Lmax = k.shape[0], k.shape[1], k.shape[2]
    _ok("plora_attn_decode", lib.plora_attn_decode(
        q.data_ptr(), k.data_ptr(), v.data_ptr(), lens.data_ptr(), Bn, H, Lmax, scale,
        out.data_ptr(), ws.data_ptr() if ws is not None else None,
        ws.numel() if ws is not None else 0, _stream(stream)))


def apply_multi(x, ads, segs: Segments, ys, ws: Workspace, stream=None) -> None:
    """ads: Adapters, one per projection; ys: their output tensors."""
    plora_apply_multi(x.data_ptr(), x.stride(0), [a.struct for a in ads], segs.struct,
                      [y.data_ptr() for y in ys], [y.stride(0) for y in ys], ws.ptr,
                      ws.nbytes, _stream(stream))
