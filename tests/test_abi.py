"""The C ABI library without a GPU: it loads, exports every entry point the
header declares, and its host-side argument checks return the documented
status codes before anything is launched."""
import ctypes
import os
import re

import pytest

from paper_2608_05483_amd import build as B
from paper_2608_05483_amd import plora as P

INCLUDE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")
HEADERS = [os.path.join(INCLUDE, h) for h in ("plora.h", "plora_attention.h")]

FAKE = 0x10000  # an aligned non-null address; never dereferenced by these checks


def declared_functions():
    text = "".join(open(h).read() for h in HEADERS)
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(plora_[a-z_]+)\s*\(", text)))


def test_header_declares_the_expected_calls():
    names = declared_functions()
    for fn in ("plora_segment", "plora_shrink", "plora_expand", "plora_apply",
               "plora_apply_multi", "plora_workspace_bytes", "plora_workspace_bytes_multi",
               "plora_status_string"):
        assert fn in names
    assert set(names) == set(P.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(P.LIB_PATH)
    for fn in declared_functions():
        assert hasattr(lib, fn), fn


def test_status_strings():
    assert P.status_string(P.PLORA_OK) == "PLORA_OK"
    assert P.status_string(P.PLORA_ERR_HIP) == "PLORA_ERR_HIP"
    assert P.status_string(99) == "PLORA_ERR_UNKNOWN"


def test_tile_capacity():
    assert P.plora_tile_capacity(0, 10) == 0
    assert P.plora_tile_capacity(64, 1000) == 64
    assert P.plora_tile_capacity(8192, 32) == 32 + 8192 // 32
    assert P.plora_tile_capacity(5, 1) == 5            # tiles of 1 token up to 64
    assert P.plora_tile_capacity(64, 1) == 64
    assert P.plora_tile_capacity(65, 1) == 1 + 65 // 2  # tiles of 2 tokens up to 256
    assert P.plora_tile_capacity(256, 1) == 1 + 128
    assert P.plora_tile_capacity(300, 1) == 1 + 300 // 32
    assert [P.tile_tokens(T) for T in (1, 64, 65, 256, 257)] == [1, 1, 2, 2, 32]
    # the bound holds for the worst batch: every segment of length Kk+1
    for T, N in [(40, 3), (100, 3), (256, 7), (1000, 7), (16384, 1000)]:
        cap = min(T, N)
        K = P.tile_tokens(T)
        assert P.plora_tile_capacity(T, N) >= min(T, cap + T // K)


def _ad(**kw):
    a = dict(n_adapters=4, h_in=256, h_out=256, max_rank=8, A=FAKE, B=FAKE,
             a_len=4 * 256 * 8, b_len=4 * 256 * 8, a_off=FAKE, b_off=FAKE,
             ranks=FAKE, scales=FAKE)
    a.update(kw)
    return P.plora_adapters(**a)


def _seg(T=8, N=4, **kw):
    s = dict(T=T, cap=min(T, N), tile_cap=P.plora_tile_capacity(T, N), reserved=0,
             perm=FAKE, seg_ptr=FAKE, seg_id=FAKE, meta=FAKE, tiles=FAKE)
    s.update(kw)
    return P.plora_segments(**s)


def _apply_status(ad=None, seg=None, x=FAKE, ldx=256, y=FAKE, ldy=256, ws=FAKE,
                  ws_bytes=None):
    ad = ad or _ad()
    seg = seg or _seg()
    if ws_bytes is None:
        ws_bytes = P.plora_workspace_bytes(seg.T, ad)
    return P.lib.plora_apply(x, ldx, ctypes.byref(ad), ctypes.byref(seg), y, ldy, ws,
                             ws_bytes, None)


def _expected_ws(T, N, h_in, max_rank):
    """The documented layout: 336 64-bit epochs and two counters, 4096
    readiness words (64-bit), then one exchange region of
    8 x PLORA_SMALL_BATCH_TILE_TOKENS x 128 64-bit words per tile slot for min(336, max(8, cap8)) slots
    (cap8 = the tile capacity rounded up to 8), then the partial sums of v
    over min(8, h_in / 512) slices of h_in (fp32), each section 256-byte
    aligned."""
    up = lambda v: (v + 255) // 256 * 256
    k = min(8, max(1, h_in // 512))
    slots = min(336, max(8, (P.plora_tile_capacity(T, N) + 7) // 8 * 8))
    head = up(up(336 * 8 + 2 * 8) + 4096 * 8)
    return up(up(head + slots * 8 * P.PLORA_SMALL_BATCH_TILE_TOKENS * 128 * 8) + k * T * max_rank * 4)


def test_workspace_size_and_checks():
    for h_in, k in [(256, 1), (1024, 2), (4096, 8), (32768, 8)]:
        ad = _ad(h_in=h_in, max_rank=16)
        assert P.plora_workspace_bytes(100, ad) == _expected_ws(100, 4, h_in, 16)
        assert P.plora_workspace_bytes(100, ad) >= k * 100 * 16 * 4
    # the exchange regions stop growing at 336 tile slots
    big = _ad(n_adapters=1000, h_in=4096, max_rank=16)
    for T in (8, 64, 300, 1024, 16384):
        assert P.plora_workspace_bytes(T, big) == _expected_ws(T, 1000, 4096, 16)
    assert (P.plora_workspace_bytes(16384, big) - 8 * 16384 * 16 * 4
            < 337 * 8 * P.PLORA_SMALL_BATCH_TILE_TOKENS * 128 * 8 + 4096 * 8 + 4096)
    ad = _ad()
    assert P.plora_workspace_bytes(0, ad) == 0
    assert P.lib.plora_workspace_init(None, 0, None) == P.PLORA_OK
    need = P.plora_workspace_bytes(8, ad)
    assert need > 0
    assert _apply_status(ws_bytes=need - 16) == P.PLORA_ERR_WORKSPACE_TOO_SMALL
    assert _apply_status(ws=None) == P.PLORA_ERR_INVALID_ARG
    assert _apply_status(ws=FAKE + 8) == P.PLORA_ERR_UNSUPPORTED
    # plora_expand takes no workspace: its checks pass with none (T = 0 so
    # nothing is launched on the fake pointers)
    empty = _seg(T=0, N=4, perm=None, seg_ptr=None, seg_id=None, meta=None, tiles=None)
    assert P.lib.plora_expand(FAKE, 8, ctypes.byref(ad), ctypes.byref(empty), FAKE, 256,
                              None, 0, None) == P.PLORA_OK


def test_large_model_dimensions_pass_host_checks():
    # LDS use does not grow with h_in or h_out; an empty batch returns right
    # after the checks, so nothing is ever launched on the fake pointers
    empty = _seg(T=0, N=4, perm=None, seg_ptr=None, seg_id=None, meta=None, tiles=None)
    for h in (16384, 32768):
        st = _apply_status(ad=_ad(h_in=h, h_out=h, max_rank=128), seg=empty, ldx=h, ldy=h)
        assert st == P.PLORA_OK


@pytest.mark.parametrize("kw,status", [
    (dict(h_in=260), P.PLORA_ERR_UNSUPPORTED),
    (dict(h_out=12), P.PLORA_ERR_UNSUPPORTED),
    (dict(max_rank=12), P.PLORA_ERR_UNSUPPORTED),
    (dict(max_rank=136), P.PLORA_ERR_UNSUPPORTED),
    (dict(max_rank=0), P.PLORA_ERR_UNSUPPORTED),
    (dict(h_in=0), P.PLORA_ERR_INVALID_ARG),
    (dict(A=None), P.PLORA_ERR_INVALID_ARG),
    (dict(A=FAKE + 2), P.PLORA_ERR_UNSUPPORTED),
    (dict(n_adapters=-1), P.PLORA_ERR_INVALID_ARG),
])
def test_adapter_checks(kw, status):
    assert _apply_status(ad=_ad(**kw)) == status


@pytest.mark.parametrize("kw,status", [
    (dict(ldx=200), P.PLORA_ERR_INVALID_ARG),
    (dict(ldy=100), P.PLORA_ERR_INVALID_ARG),
    (dict(ldx=260), P.PLORA_ERR_UNSUPPORTED),
    (dict(x=None), P.PLORA_ERR_INVALID_ARG),
    (dict(y=FAKE + 8), P.PLORA_ERR_UNSUPPORTED),
])
def test_operand_checks(kw, status):
    assert _apply_status(**kw) == status


def test_segment_struct_checks():
    assert _apply_status(seg=_seg(cap=3)) == P.PLORA_ERR_INVALID_ARG
    assert _apply_status(seg=_seg(tile_cap=99)) == P.PLORA_ERR_INVALID_ARG
    assert _apply_status(seg=_seg(T=-1, cap=-1, tile_cap=0)) == P.PLORA_ERR_INVALID_ARG
    big = P.PLORA_MAX_TOKENS + 1
    assert _apply_status(seg=_seg(T=big, N=4)) == P.PLORA_ERR_UNSUPPORTED
    assert _apply_status(seg=_seg(perm=None)) == P.PLORA_ERR_INVALID_ARG


def test_empty_batch_is_a_no_op_everywhere():
    ad = _ad()
    seg = _seg(T=0, N=4, perm=None, seg_ptr=None, seg_id=None, meta=None, tiles=None)
    assert P.lib.plora_segment(None, ctypes.byref(seg), 4, None, 0, None) == P.PLORA_OK
    assert _apply_status(seg=seg, x=None, y=None) == P.PLORA_OK
    assert P.lib.plora_expand(None, 8, ctypes.byref(ad), ctypes.byref(seg), None, 256,
                              None, 0, None) == P.PLORA_OK
    ws = P.plora_workspace_bytes(0, ad)
    assert P.lib.plora_shrink(None, 256, ctypes.byref(ad), ctypes.byref(seg), None, 8,
                              FAKE, ws, None) == P.PLORA_OK


def test_segment_rejects_oversized_key_space():
    # 2^ceil(log2 T) * (N + 1) must fit 32 bits
    T = 16384
    N = 1 << 20
    seg = _seg(T=T, N=N)
    assert P.lib.plora_segment(FAKE, ctypes.byref(seg), N, None, 0, None) == \
        P.PLORA_ERR_UNSUPPORTED


def test_shrink_and_expand_leading_dimension_checks():
    ad, seg = _ad(), _seg()
    ws = P.plora_workspace_bytes(8, ad)
    st = P.lib.plora_shrink(FAKE, 256, ctypes.byref(ad), ctypes.byref(seg), FAKE, 4,
                            FAKE, ws, None)
    assert st == P.PLORA_ERR_INVALID_ARG  # ldv < max_rank
    st = P.lib.plora_shrink(FAKE, 256, ctypes.byref(ad), ctypes.byref(seg), FAKE, 10,
                            FAKE, ws, None)
    assert st == P.PLORA_ERR_UNSUPPORTED  # ldv not a multiple of 4
    st = P.lib.plora_expand(FAKE, 8, ctypes.byref(ad), ctypes.byref(seg), FAKE, 255,
                            None, 0, None)
    assert st == P.PLORA_ERR_INVALID_ARG


def test_one_hip_runtime_per_process():
    """The binding must bind libplora.so to torch's HIP runtime; a second
    libamdhip64 in the process makes torch's streams foreign to our launches.
    Checked in a fresh interpreter so import order is the binding's own."""
    import subprocess
    import sys
    code = ("from paper_2608_05483_amd import plora\n"
            "m = open('/proc/self/maps').read().splitlines()\n"
            "print(len({l.split()[-1] for l in m if 'libamdhip64' in l}))\n")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    out = subprocess.run([sys.executable, "-c", code], cwd=root, capture_output=True,
                         text=True, timeout=300)
    assert out.returncode == 0, out.stderr
    assert out.stdout.strip().splitlines()[-1] == "1"


def _multi_status(ads, n=None, x=FAKE, ldx=256, ys=None, ldys=None, ws=FAKE, ws_bytes=None,
                  seg=None):
    seg = seg or _seg()
    n = len(ads) if n is None else n
    arr = (P.plora_adapters * max(len(ads), 1))(*ads)
    ys = [FAKE] * len(ads) if ys is None else ys
    ldys = [a.h_out for a in ads] if ldys is None else ldys
    yarr = (ctypes.c_void_p * max(len(ys), 1))(*ys)
    larr = (ctypes.c_int64 * max(len(ldys), 1))(*ldys)
    if ws_bytes is None:
        ws_bytes = P.lib.plora_workspace_bytes_multi(seg.T, arr, max(n, 1))
    return P.lib.plora_apply_multi(x, ldx, arr, n, ctypes.byref(seg), yarr, larr, ws,
                                   ws_bytes, None)


def test_apply_multi_host_checks():
    """plora_apply_multi's host-side rules, on fake device pointers (every
    case returns before anything is launched)."""
    a, b = _ad(), _ad(h_out=128)
    # workspace: n cap8 tile slots, the largest partial-sum section
    arr = (P.plora_adapters * 2)(a, b)
    need = P.lib.plora_workspace_bytes_multi(8, arr, 2)
    up = lambda v: (v + 255) // 256 * 256
    slots = min(336, max(8, 2 * ((P.plora_tile_capacity(8, 4) + 7) // 8 * 8)))
    assert need == up(up(up(up(336 * 8 + 2 * 8) + 4096 * 8) + slots * 8 * P.PLORA_SMALL_BATCH_TILE_TOKENS * 128 * 8) + 8 * 8 * 4)
    assert need >= P.plora_workspace_bytes(8, a)
    assert P.lib.plora_workspace_bytes_multi(8, arr, 0) == 0
    assert P.lib.plora_workspace_bytes_multi(8, arr, P.PLORA_MAX_PROJECTIONS + 1) == 0
    assert _multi_status([a, b], ws_bytes=need - 16) == P.PLORA_ERR_WORKSPACE_TOO_SMALL
    assert _multi_status([a, b], ws=None) == P.PLORA_ERR_INVALID_ARG
    assert _multi_status([a, b], n=0) == P.PLORA_ERR_INVALID_ARG
    assert _multi_status([a] * 9) == P.PLORA_ERR_UNSUPPORTED
    # stacks must share n_adapters and h_in (one x, one batch)
    assert _multi_status([a, _ad(h_in=512)]) == P.PLORA_ERR_INVALID_ARG
    assert _multi_status([a, _ad(n_adapters=3)]) == P.PLORA_ERR_INVALID_ARG
    # per-projection output checks
    assert _multi_status([a, b], ys=[FAKE, None]) == P.PLORA_ERR_INVALID_ARG
    assert _multi_status([a, b], ldys=[256, 64]) == P.PLORA_ERR_INVALID_ARG
    assert _multi_status([a, b], ldys=[256, 132]) == P.PLORA_ERR_UNSUPPORTED
    assert _multi_status([a, b], ys=[FAKE, FAKE + 8]) == P.PLORA_ERR_UNSUPPORTED
    assert _multi_status([a, b], ldx=255) == P.PLORA_ERR_INVALID_ARG
    # a bad stack is reported as for plora_apply
    assert _multi_status([a, _ad(max_rank=12)]) == P.PLORA_ERR_UNSUPPORTED
    # an empty batch launches nothing
    empty = _seg(T=0, N=4, perm=None, seg_ptr=None, seg_id=None, meta=None, tiles=None)
    assert _multi_status([a, b], seg=empty, ws=None, ws_bytes=0) == P.PLORA_OK


def _segapply_status(ad=None, seg=None, idx=FAKE, x=FAKE, ldx=256, y=FAKE, ldy=256, ws=FAKE,
                     ws_bytes=None):
    ad = ad or _ad()
    seg = seg or _seg()
    if ws_bytes is None:
        ws_bytes = P.plora_workspace_bytes(seg.T, ad)
    return P.lib.plora_segment_apply(idx, x, ldx, ctypes.byref(ad), ctypes.byref(seg), y, ldy,
                                     ws, ws_bytes, None)


def test_segment_apply_host_checks():
    assert _segapply_status(idx=None) == P.PLORA_ERR_INVALID_ARG
    assert _segapply_status(x=None) == P.PLORA_ERR_INVALID_ARG
    assert _segapply_status(y=None) == P.PLORA_ERR_INVALID_ARG
    assert _segapply_status(ldx=200) == P.PLORA_ERR_INVALID_ARG
    assert _segapply_status(ldy=260) == P.PLORA_ERR_UNSUPPORTED
    assert _segapply_status(x=FAKE + 8) == P.PLORA_ERR_UNSUPPORTED
    assert _segapply_status(ad=_ad(h_out=12)) == P.PLORA_ERR_UNSUPPORTED
    assert _segapply_status(seg=_seg(cap=3)) == P.PLORA_ERR_INVALID_ARG
    assert _segapply_status(ws=None) == P.PLORA_ERR_INVALID_ARG
    assert _segapply_status(ws_bytes=256) == P.PLORA_ERR_WORKSPACE_TOO_SMALL
    empty = _seg(T=0, N=4, perm=None, seg_ptr=None, seg_id=None, meta=None, tiles=None)
    assert _segapply_status(seg=empty, idx=None, x=None, y=None) == P.PLORA_OK


def test_segment_workspace_bytes():
    """The many-work-group segmentation's table: (ceil(T / 1024) + 1) x
    (N + 2) int32, 256-byte rounded, above 1024 tokens over 2048 to 8191 ids
    (fewer ids take the one-launch counting sort, which needs none)."""
    f = P.plora_segment_workspace_bytes
    assert f(1024, 3000) == 0 and f(0, 5) == 0
    assert f(1025, 1000) == 0 and f(16384, 2047) == 0 and f(16384, 7) == 0
    assert f(1025, 2048) == (3 * 2050 * 4 + 255) // 256 * 256
    assert f(16384, 3000) == (17 * 3002 * 4 + 255) // 256 * 256
    assert f(5000, 8191) > 0 and f(5000, 8192) == 0
    # the apply's workspace covers it
    ad = _ad(n_adapters=3000, h_in=256, h_out=256, max_rank=8)
    assert P.plora_workspace_bytes(16384, ad) >= f(16384, 3000)


def test_segment_apply_noalloc_host_checks():
    """The allocation-free call refuses batches above its static workspace's
    256 tokens, and checks its arguments like plora_segment_apply, before
    anything touches the device."""
    L = P.lib

    def st(ad=None, seg=None, idx=FAKE, x=FAKE, ldx=256, y=FAKE, ldy=256):
        ad = ad or _ad()
        seg = seg or _seg()
        return L.plora_segment_apply_noalloc(idx, x, ldx, ctypes.byref(ad), ctypes.byref(seg),
                                             y, ldy, None)
    dec = _ad(n_adapters=1000, h_in=4096, h_out=4096, max_rank=128)
    assert st(ad=dec, seg=_seg(T=257, N=1000), ldx=4096, ldy=4096) == P.PLORA_ERR_UNSUPPORTED
    assert st(ad=dec, seg=_seg(T=16384, N=1000), ldx=4096, ldy=4096) == \
        P.PLORA_ERR_UNSUPPORTED
    assert st(idx=None) == P.PLORA_ERR_INVALID_ARG
    assert st(x=None) == P.PLORA_ERR_INVALID_ARG
    assert st(ldx=200) == P.PLORA_ERR_INVALID_ARG
    assert st(ldy=260) == P.PLORA_ERR_UNSUPPORTED
    assert st(y=FAKE + 8) == P.PLORA_ERR_UNSUPPORTED
    assert st(ad=_ad(max_rank=136)) == P.PLORA_ERR_UNSUPPORTED
    assert st(seg=_seg(cap=3)) == P.PLORA_ERR_INVALID_ARG
    empty = _seg(T=0, N=4, perm=None, seg_ptr=None, seg_id=None, meta=None, tiles=None)
    assert st(seg=empty, idx=None, x=None, y=None) == P.PLORA_OK


def test_adapter_blocks_must_stay_below_2gib():
    # adapter blocks are read through 32-bit byte offsets: max(h_in, h_out)
    # * max_rank * 2 bytes must stay below 2^31 (checked before the empty
    # batch returns)
    empty = _seg(T=0, N=4, perm=None, seg_ptr=None, seg_id=None, meta=None, tiles=None)
    h = 1 << 23
    big = _ad(h_in=h, h_out=256, max_rank=128)
    assert _apply_status(ad=big, seg=empty, ldx=h) == P.PLORA_ERR_UNSUPPORTED
    ok = _ad(h_in=1 << 22, h_out=256, max_rank=128)
    assert _apply_status(ad=ok, seg=empty, ldx=1 << 22) == P.PLORA_OK


def test_segment_apply_launch_count():
    dec = _ad(n_adapters=1000, h_in=4096, h_out=4096, max_rank=16)
    assert P.plora_segment_apply_launches(64, dec) == 1     # decode: one launch
    assert P.plora_segment_apply_launches(1, dec) == 1
    assert P.plora_segment_apply_launches(65, dec) == 1     # the whole work group segments
    assert P.plora_segment_apply_launches(256, dec) == 1
    assert P.plora_segment_apply_launches(257, dec) == 2    # segment, then the two-part launch
    assert P.plora_segment_apply_launches(4096, dec) == 2
    # above 4096 tile slots: segment, then shrink and expand launches
    wide = _ad(n_adapters=5000, h_in=4096, max_rank=16)
    assert P.plora_tile_capacity(5000, 5000) > 4096
    assert P.plora_segment_apply_launches(5000, wide) == 3
    assert P.plora_segment_apply_launches(8, _ad()) == 2    # h = 256: no split form
    assert P.plora_segment_apply_launches(0, dec) == 0
    assert P.plora_segment_apply_launches(8, _ad(h_in=12)) == 0


def test_attention_host_checks():
    L = P.lib
    assert P.attn_partitions(0) == 0 and P.attn_partitions(1) == 1
    assert P.attn_partitions(256) == 1 and P.attn_partitions(257) == 2
    assert P.attn_workspace_bytes(0, 32, 100) == 0
    # m and l: 2 x 3 x 2 floats each, 256-aligned; o: 12 x 128 floats
    assert P.attn_workspace_bytes(2, 3, 300) == 256 + 256 + 12 * 128 * 4
    args = dict(q=FAKE, k=FAKE, v=FAKE, lens=FAKE, B=2, H=4, Lm=300)

    def partial(**kw):
        a = {**args, **kw}
        return L.plora_attn_partial(a["q"], a["k"], a["v"], a["lens"], a["B"], a["H"], a["Lm"],
                                    0.1, FAKE, FAKE, FAKE, None)
    assert partial(q=None) == P.PLORA_ERR_INVALID_ARG
    assert partial(B=-1) == P.PLORA_ERR_INVALID_ARG
    assert partial(k=FAKE + 2) == P.PLORA_ERR_UNSUPPORTED
    assert partial(Lm=1 << 23) == P.PLORA_ERR_UNSUPPORTED   # 2^23 x 256 B per cache
    assert partial(B=0, q=None) == P.PLORA_OK
    ws = P.attn_workspace_bytes(2, 4, 300)
    dec = lambda ws_p, n: L.plora_attn_decode(FAKE, FAKE, FAKE, FAKE, 2, 4, 300, 0.1, FAKE,
                                              ws_p, n, None)
    assert dec(None, ws) == P.PLORA_ERR_INVALID_ARG
    assert dec(FAKE, ws - 1) == P.PLORA_ERR_WORKSPACE_TOO_SMALL
    assert L.plora_attn_merge(None, FAKE, FAKE, FAKE, 2, 4, 300, FAKE, None) == \
        P.PLORA_ERR_INVALID_ARG
