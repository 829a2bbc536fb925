"""Pins for the CPU oracle: each test ties it to something other than itself.

The paper prints no worked numeric example of the apply, so the pins are
(a) the plain definition evaluated exactly on small integer inputs with pure
Python integers, (b) closed forms for structured adapters, (c) float64 library
products (numpy matmul) inside a rigorous fp32 rounding-error bound, (d) brute
force sorting for the segmentation, (e) an independent exact-rational bf16
rounding, and (f) the invariants the method implies: one adapter equals
x A B, zero B leaves y_base, token order does not matter, grouped equals
ungrouped, the result is linear in the scale, and the four strategies of
section V-A (xA then B, or x times AB) agree.

Each pin is chosen so that a plausible slip in the oracle -- a transposed
operand, a wrong stride or offset, a dropped scale, a sign, an unstable sort,
a missed tie-break -- fails at least one of them.
"""
from __future__ import annotations

import itertools
import math
import random
from fractions import Fraction

import numpy as np
import pytest

import oracle
import refs
from paper_2608_05483_amd import workloads as W

U = 2.0 ** -24  # unit roundoff of fp32


def gamma(n: int) -> float:
    return n * U / (1 - n * U)


# ---------------------------------------------------------------------------
# independent bf16 helpers (pure Python, exact rationals)
# ---------------------------------------------------------------------------

def bf16_value(bits: int) -> Fraction | float:
    """Exact value of a bf16 bit pattern, from the IEEE binary format."""
    sign = -1 if bits & 0x8000 else 1
    e = (bits >> 7) & 0xFF
    m = bits & 0x7F
    if e == 0xFF:
        return float("nan") if m else sign * float("inf")
    if e == 0:
        return sign * Fraction(m, 1 << 7) * Fraction(2) ** (-126)
    return sign * (1 + Fraction(m, 1 << 7)) * Fraction(2) ** (e - 127)


def bf16_round(value: Fraction) -> int:
    """Round an exact rational to bf16 bits, nearest with ties to even,
    by searching the two neighbouring representable values."""
    if value == 0:
        return 0
    sign = 0x8000 if value < 0 else 0
    a = abs(value)
    max_finite = (2 - Fraction(1, 1 << 7)) * Fraction(2) ** 127
    # exponent of the binade holding a (normal range) or the subnormal step
    e = math.floor(math.log2(a)) if a >= Fraction(2) ** -126 else -126
    # guard the float log2 rounding
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    e = max(e, -126)
    step = Fraction(2) ** (e - 7)
    lo = (a // step) * step
    hi = lo + step
    if a - lo < hi - a:
        pick = lo
    elif a - lo > hi - a:
        pick = hi
    else:  # tie: even mantissa
        pick = lo if (lo / step) % 2 == 0 else hi
    if pick > max_finite:
        # halfway between max_finite and 2^128 rounds to inf as well
        return sign | 0x7F80
    if pick == 0:
        return sign
    pe = math.floor(math.log2(pick))
    while Fraction(2) ** pe > pick:
        pe -= 1
    while Fraction(2) ** (pe + 1) <= pick:
        pe += 1
    if pe < -126:  # subnormal
        m = int(pick / (Fraction(2) ** -133))
        return sign | m
    m = int((pick / Fraction(2) ** pe - 1) * 128)
    if m == 128:
        m = 0
        pe += 1
    return sign | ((pe + 127) << 7) | m


def f32_bits_to_fraction(u: int) -> Fraction | float:
    f = np.array([u], np.uint32).view(np.float32)[0]
    if not np.isfinite(f):
        return float(f)
    return Fraction(float(f))


# ---------------------------------------------------------------------------
# bf16 conversion pins
# ---------------------------------------------------------------------------

def test_bf16_decode_is_exact():
    bits = np.arange(0, 1 << 16, dtype=np.uint32).astype(np.uint16)
    got = oracle.bf16_to_f32(bits)
    want = (bits.astype(np.uint32) << 16).view(np.float32)
    same = (got.view(np.uint32) == want.view(np.uint32))
    assert same.all()
    # spot-check against the format definition
    for b in (0x3F80, 0xBF80, 0x4049, 0x0001, 0x7F7F, 0x0080):
        assert Fraction(float(got[b])) == bf16_value(b)


def test_bf16_encode_matches_exact_rational_rounding():
    rng = random.Random(7)
    cases = [0x3F808000, 0x3F818000, 0x3F80C000, 0x3F807FFF, 0x7F7FFFFF,
             0x7F7F8000, 0x7F7F7FFF, 0x00008000, 0x00018000, 0x00000001,
             0x807FFFFF, 0xBF808000, 0x00400000]
    for _ in range(4000):
        e = rng.randrange(1, 255)
        cases.append((rng.getrandbits(1) << 31) | (e << 23) | rng.getrandbits(23))
    for _ in range(500):  # exact ties
        e = rng.randrange(1, 254)
        cases.append((e << 23) | (rng.getrandbits(7) << 16) | 0x8000)
    u = np.array(cases, np.uint32)
    got = oracle.f32_to_bf16(u.view(np.float32))
    for ui, gi in zip(cases, got):
        want = bf16_round(f32_bits_to_fraction(ui))
        assert int(gi) == want, hex(ui)


def test_bf16_encode_specials():
    vals = np.array([np.inf, -np.inf, np.nan, 0.0, -0.0], np.float32)
    got = oracle.f32_to_bf16(vals)
    assert got[0] == 0x7F80 and got[1] == 0xFF80
    assert (got[2] & 0x7F80) == 0x7F80 and (got[2] & 0x7F) != 0
    assert got[3] == 0 and got[4] == 0x8000


# ---------------------------------------------------------------------------
# segmentation pins: brute-force sort and the invariants
# ---------------------------------------------------------------------------

def brute_segments(idx, N):
    valid = [t for t in range(len(idx)) if 0 <= idx[t] < N]
    order = sorted(valid, key=lambda t: (idx[t], t))
    T = len(idx)
    cap = min(T, N)
    perm = order + [-1] * (T - len(order))
    seg_ptr, seg_id = [], []
    for p, t in enumerate(order):
        if p == 0 or idx[order[p - 1]] != idx[t]:
            seg_ptr.append(p)
            seg_id.append(idx[t])
    n_seg = len(seg_id)
    seg_ptr = seg_ptr + [len(order)] * (cap + 1 - n_seg)
    seg_id = seg_id + [-1] * (cap - n_seg)
    meta = [n_seg, len(order), sum(1 for i in idx if i == -1),
            sum(1 for i in idx if i != -1 and not 0 <= i < N)]
    return perm, seg_ptr, seg_id, meta


def _seg_cases():
    rng = np.random.default_rng(3)
    out = [
        (np.zeros(0, np.int32), 5),
        (np.array([2], np.int32), 4),
        (np.array([-1, -1, -1], np.int32), 4),
        (np.array([7, -3, 4, 100], np.int32), 4),
        (np.full(17, 3, np.int32), 4),
        (np.array([0, 0, 0], np.int32), 1),
        (np.arange(9, dtype=np.int32)[::-1].copy(), 9),
        (np.array([5, 1, 5, 1, 5], np.int32), 1000),
    ]
    for T, N in [(8, 4), (64, 1000), (300, 7), (1000, 50), (257, 256)]:
        idx = rng.integers(-2, N + 2, size=T).astype(np.int32)
        out.append((idx, N))
        out.append((W.zipf_ids(rng, T, N, 1.0), N))
    return out


@pytest.mark.parametrize("case", range(len(_seg_cases())))
def test_segment_matches_brute_force_sort(case):
    idx, N = _seg_cases()[case]
    got = oracle.segment(idx, N)
    perm, seg_ptr, seg_id, meta = brute_segments(idx.tolist(), N)
    assert got.perm.tolist() == perm
    assert got.seg_ptr.tolist() == seg_ptr
    assert got.seg_id.tolist() == seg_id
    assert got.meta.tolist() == meta


@pytest.mark.parametrize("case", range(len(_seg_cases())))
def test_segment_invariants(case):
    idx, N = _seg_cases()[case]
    s = oracle.segment(idx, N)
    n_seg, n_valid = int(s.meta[0]), int(s.meta[1])
    valid = [t for t in range(idx.size) if 0 <= idx[t] < N]
    assert sorted(s.perm[:n_valid].tolist()) == valid          # a permutation
    assert (s.perm[n_valid:] == -1).all()
    sp = s.seg_ptr[:n_seg + 1]
    assert (np.diff(sp) > 0).all() and sp[0] == 0 if n_seg else True
    assert (np.diff(s.seg_id[:n_seg]) > 0).all()                # ascending ids
    for k in range(n_seg):
        toks = s.perm[sp[k]:sp[k + 1]]
        assert (idx[toks] == s.seg_id[k]).all()
        assert (np.diff(toks) > 0).all()                          # stable
    assert sum(np.diff(sp)) == n_valid


# ---------------------------------------------------------------------------
# apply pins
# ---------------------------------------------------------------------------

def _int_case(rng, T, N, h_in, h_out, ranks, scales, none_frac=0.2):
    ranks = np.asarray(ranks, np.int32)
    a_off = np.concatenate([[0], np.cumsum(ranks.astype(np.int64) * h_in)[:-1]])
    b_off = np.concatenate([[0], np.cumsum(ranks.astype(np.int64) * h_out)[:-1]])
    a_len = int(np.sum(ranks.astype(np.int64) * h_in))
    b_len = int(np.sum(ranks.astype(np.int64) * h_out))
    xi = rng.integers(-3, 4, size=(T, h_in))
    Ai = rng.integers(-2, 3, size=a_len)
    Bi = rng.integers(-2, 3, size=b_len)
    yi = rng.integers(-4, 5, size=(T, h_out))
    idx = rng.integers(0, N, size=T).astype(np.int32)
    drop = rng.random(T) < none_frac
    idx[drop] = rng.choice([-1, N, N + 3, -7], size=int(drop.sum()))
    enc = lambda a: W.to_bf16_bits(np.asarray(a, np.float32))
    return dict(xi=xi, Ai=Ai, Bi=Bi, yi=yi, idx=idx, ranks=ranks,
                a_off=a_off.astype(np.int64), b_off=b_off.astype(np.int64),
                scales=np.asarray(scales, np.float32), x=enc(xi), A=enc(Ai),
                B=enc(Bi), y=enc(yi), h_in=h_in, h_out=h_out, N=N)


def _exact_apply(c, t):
    """Pure-Python exact y[t] as rationals, from the definition."""
    i = int(c["idx"][t])
    h_in, h_out = c["h_in"], c["h_out"]
    ybase = [Fraction(int(v)) for v in c["yi"][t]]
    if not 0 <= i < c["N"] or c["ranks"][i] == 0:
        return ybase
    r = int(c["ranks"][i])
    ao, bo = int(c["a_off"][i]), int(c["b_off"][i])
    v = [sum(int(c["xi"][t][k]) * int(c["Ai"][ao + k * r + cc])
             for k in range(h_in)) for cc in range(r)]
    s = Fraction(float(c["scales"][i]))
    return [ybase[j] + s * sum(v[cc] * int(c["Bi"][bo + cc * h_out + j])
                               for cc in range(r)) for j in range(h_out)]


@pytest.mark.parametrize("seed,ranks", [(0, [8, 16, 0]), (1, [8, 16, 0]), (2, [8, 16, 0]),
                                        (3, [1, 3, 12, 0, 5]), (4, [2, 24, 7, 4, 13])])
def test_apply_exact_on_small_integers(seed, ranks):
    """Integer inputs keep every fp32 partial sum exact (< 2^24), so the
    oracle must reproduce the pure-Python exact result bit for bit, and its
    bf16 output must be the exact result rounded to nearest-even.  The ranks
    include ones that are not multiples of 8 (rows of A_i of odd length)."""
    rng = np.random.default_rng(seed)
    c = _int_case(rng, T=7, N=len(ranks), h_in=24, h_out=16, ranks=ranks,
                  scales=[1.0, 0.5, 2.0, 0.25, 4.0][:len(ranks)])
    yref, yout = oracle.apply(c["x"], c["idx"], c["A"], c["a_off"], c["B"],
                              c["b_off"], c["ranks"], c["scales"], c["y"],
                              c["h_in"], c["h_out"])
    for t in range(7):
        ex = _exact_apply(c, t)
        assert [Fraction(float(v)) for v in yref[t]] == ex, t
        assert yout[t].tolist() == [bf16_round(e) for e in ex], t


def test_apply_closed_form_selection_adapters():
    """A_i picks input features, B_i places them: with A_i[k, c] = [k ==
    pi_i(c)] and B_i[c, j] = [j == sigma_i(c)], y[t, sigma(c)] = s x[t, pi(c)]
    exactly (y_base = 0, s a power of two), all other columns zero."""
    rng = np.random.default_rng(11)
    N, h_in, h_out, r, T = 3, 40, 24, 8, 9
    ranks = np.full(N, r, np.int32)
    a_off = np.arange(N, dtype=np.int64) * h_in * r
    b_off = np.arange(N, dtype=np.int64) * r * h_out
    A = np.zeros(N * h_in * r, np.float32)
    B = np.zeros(N * r * h_out, np.float32)
    pis, sigmas = [], []
    for i in range(N):
        pi = rng.permutation(h_in)[:r]
        sg = rng.permutation(h_out)[:r]
        pis.append(pi)
        sigmas.append(sg)
        for c in range(r):
            A[a_off[i] + pi[c] * r + c] = 1.0
            B[b_off[i] + c * h_out + sg[c]] = 1.0
    scales = np.array([1.0, 2.0, 0.25], np.float32)
    xf = rng.standard_normal((T, h_in)).astype(np.float32)
    x = W.to_bf16_bits(xf)
    idx = rng.integers(0, N, T).astype(np.int32)
    y0 = np.zeros((T, h_out), np.uint16)
    yref, yout = oracle.apply(x, idx, W.to_bf16_bits(A), a_off,
                              W.to_bf16_bits(B), b_off, ranks, scales, y0,
                              h_in, h_out)
    xv = (x.astype(np.uint32) << 16).view(np.float32)
    for t in range(T):
        i = idx[t]
        want = np.zeros(h_out, np.float32)
        for c in range(r):
            want[sigmas[i][c]] = scales[i] * xv[t, pis[i][c]]
        assert (yref[t] == want).all()


_f64_reference = refs.f64_reference


@pytest.mark.parametrize("name,scale", [("tiny", "paper"), ("tiny", "parity"),
                                        ("decode", "parity"),
                                        ("ragged", "parity")])
def test_apply_within_fp32_bound_of_float64(name, scale):
    """Per-token float64 products (numpy matmul) pin the oracle within the
    standard recursive-summation bound gamma_n * sum|terms|."""
    w = W.make_workload(name, scale=scale, only_used=True)
    rng = np.random.default_rng(5)
    tokens = np.arange(w.T) if w.T <= 64 else np.sort(rng.choice(w.T, 48, False))
    sub = W.with_idx(w, w.idx)  # same arrays
    yref, _ = oracle.apply(sub.x[tokens], sub.idx[tokens], sub.A, sub.a_off,
                           sub.B, sub.b_off, sub.ranks, sub.scales,
                           sub.y_base[tokens], w.h_in, w.h_out)
    y64, bound = _f64_reference(w, tokens)
    err = np.abs(yref.astype(np.float64) - y64)
    assert (err <= bound).all(), float((err - bound).max())
    # the worst-case bound stays an order of magnitude below the LoRA delta,
    # so a wrong adapter, a transposed operand or a lost scale fails here;
    # single dropped terms are caught by the exact integer pin above
    delta = np.abs(y64 - _f64_reference(W.with_idx(w, np.full(w.T, -1, np.int32)),
                                        tokens)[0])
    assert np.median(bound[delta > 0]) < 0.1 * np.median(delta[delta > 0])


def test_single_adapter_equals_dense_product():
    """All tokens on one adapter: y = y_base + s (X A) B, and also
    y_base + s X (A B) -- strategies E1/E3 (y from A and B directly) and E4
    (m = xA shipped, then mB) compute the same function (section V-A)."""
    w = W.make_workload("decode", scale="parity", only_used=False,
                        idx=np.zeros(16, np.int32), n_adapters=2)
    yref, _ = oracle.apply(w.x, w.idx, w.A, w.a_off, w.B, w.b_off, w.ranks,
                           w.scales, w.y_base, w.h_in, w.h_out)
    dec = lambda b: (np.asarray(b, np.uint32) << 16).view(np.float32).astype(np.float64)
    r = int(w.ranks[0])
    A = dec(w.A[:w.h_in * r]).reshape(w.h_in, r)
    B = dec(w.B[:r * w.h_out]).reshape(r, w.h_out)
    X = dec(w.x)
    s = float(w.scales[0])
    e4 = dec(w.y_base) + s * np.matmul(np.matmul(X, A), B)
    e1 = dec(w.y_base) + s * np.matmul(X, np.matmul(A, B))
    S = np.abs(X) @ np.abs(A)
    bound = gamma(w.h_in + r + 2) * (abs(s) * ((S + np.abs(X @ A)) @ np.abs(B))
                                     + np.abs(e4)) * 1.01
    assert (np.abs(yref - e4) <= bound).all()
    assert (np.abs(yref - e1) <= bound + 1e-12).all()


def test_shrink_within_rigorous_bound():
    """v = x A_i with exact bf16 products: |v - v64| <= gamma_h sum|x A|."""
    w = W.make_workload("large", scale="parity", only_used=True)
    v = oracle.shrink(w.x, w.idx, w.A, w.a_off, w.ranks, w.h_in)
    dec = lambda b: (np.asarray(b, np.uint32) << 16).view(np.float32).astype(np.float64)
    for t in range(0, w.T, 17):
        i = int(w.idx[t])
        r = int(w.ranks[i])
        Ai = dec(w.A[w.a_off[i]:w.a_off[i] + w.h_in * r]).reshape(w.h_in, r)
        x = dec(w.x[t])
        v64 = x @ Ai
        S = np.abs(x) @ np.abs(Ai)
        assert (np.abs(v[t, :r] - v64) <= gamma(w.h_in) * S).all()


# ---------------------------------------------------------------------------
# invariants
# ---------------------------------------------------------------------------

def _apply(w, **kw):
    args = dict(x=w.x, idx=w.idx, A=w.A, a_off=w.a_off, B=w.B, b_off=w.b_off,
                ranks=w.ranks, scales=w.scales, y_base=w.y_base, h_in=w.h_in,
                h_out=w.h_out)
    args.update(kw)
    return oracle.apply(**args)


def _zero_sign(bits):
    b = np.asarray(bits).copy()
    b[b == 0x8000] = 0
    return b


def test_zero_B_gives_y_base_bitwise():
    w = W.make_workload("decode", only_used=True)
    _, yout = _apply(w, B=np.zeros_like(w.B))
    assert (_zero_sign(yout) == _zero_sign(w.y_base)).all()


def test_zero_scale_and_no_adapter_rows_keep_y_base():
    w = W.make_workload("ragged", only_used=True)
    _, yout = _apply(w, scales=np.zeros_like(w.scales))
    assert (_zero_sign(yout) == _zero_sign(w.y_base)).all()
    idx = w.idx.copy()
    idx[::3] = -1
    idx[1::7] = w.n_adapters + 5
    _, yout = _apply(w, idx=idx)
    skip = (idx < 0) | (idx >= w.n_adapters)
    assert (yout[skip] == w.y_base[skip]).all()
    ranks = w.ranks.copy()
    ranks[w.idx[0]] = 0
    _, yout = _apply(w, ranks=ranks)
    rows = w.idx == w.idx[0]
    assert (yout[rows] == w.y_base[rows]).all()


def test_token_permutation_invariance_bitwise():
    w = W.make_workload("decode", only_used=True)
    yref, yout = _apply(w)
    p = np.random.default_rng(2).permutation(w.T)
    yref_p, yout_p = _apply(w, x=w.x[p], idx=w.idx[p], y_base=w.y_base[p])
    assert (yref_p.view(np.uint32) == yref[p].view(np.uint32)).all()
    assert (yout_p == yout[p]).all()


@pytest.mark.parametrize("name", ["tiny", "decode", "ragged"])
def test_grouped_equals_ungrouped_bitwise(name):
    w = W.make_workload(name, only_used=True)
    yref, yout = _apply(w)
    g_ref, g_out = oracle.apply_grouped(w.x, w.idx, w.A, w.a_off, w.B, w.b_off,
                                        w.ranks, w.scales, w.y_base, w.h_in,
                                        w.h_out)
    assert (g_ref.view(np.uint32) == yref.view(np.uint32)).all()
    assert (g_out == yout).all()


def test_linear_in_scale_bitwise():
    """With y_base = 0, scaling s by a power of two scales every rounded
    result by the same power of two."""
    w = W.make_workload("decode", scale="parity", only_used=True)
    base_ref, base_out = _apply(w, scales=np.ones_like(w.scales))
    for s in (0.5, 2.0, 4.0, -1.0):
        ref, out = _apply(w, scales=np.full_like(w.scales, s))
        assert (ref.view(np.uint32) == (np.float32(s) * base_ref).view(np.uint32)).all()
        assert (oracle.bf16_to_f32(out).view(np.uint32) ==
                (np.float32(s) * oracle.bf16_to_f32(base_out)).view(np.uint32)).all()


def test_split_shrink_expand_equals_apply_bitwise():
    w = W.make_workload("ragged", only_used=True)
    yref, yout = _apply(w)
    v = oracle.shrink(w.x, w.idx, w.A, w.a_off, w.ranks, w.h_in)
    e_ref, e_out = oracle.expand(v, w.idx, w.B, w.b_off, w.ranks, w.scales,
                                 w.y_base, w.h_out)
    assert (e_ref.view(np.uint32) == yref.view(np.uint32)).all()
    assert (e_out == yout).all()


def test_thread_count_does_not_change_bits():
    w = W.make_workload("ragged", only_used=True)
    r1, o1 = _apply(w)
    r8, o8 = oracle.apply(w.x, w.idx, w.A, w.a_off, w.B, w.b_off, w.ranks,
                          w.scales, w.y_base, w.h_in, w.h_out, n_threads=8)
    assert (r1.view(np.uint32) == r8.view(np.uint32)).all() and (o1 == o8).all()


def test_nan_and_inf_propagate():
    w = W.make_workload("tiny", only_used=True)
    x = w.x.copy()
    x[0, 3] = 0x7FC0  # NaN
    x[1, 5] = 0x7F80  # +inf
    yref, _ = _apply(w, x=x)
    assert np.isnan(yref[0]).any() and not np.isfinite(yref[1]).all()
    assert np.isfinite(yref[2:]).all()


def _stack(w):
    return (w.A, w.a_off, w.B, w.b_off, w.ranks, w.scales, w.h_out)


@pytest.mark.parametrize("name", ["tiny", "decode"])
def test_apply_multi_each_projection_within_fp32_bound(name):
    """Several projections sharing x and the ids (different stacks, output
    widths): every projection's output lies within the fp32 bound of its own
    float64 product, so no projection reads another's stack or width."""
    ps = W.make_projections(name, scale="parity")
    if name == "decode":
        ps = [W.make_projections(name, scale="parity", h_outs=(4096, 1024, 512))[p]
              for p in range(3)]
    w0 = ps[0]
    tokens = refs.sample_tokens(w0.T, 24)
    outs = oracle.apply_multi(w0.x[tokens], w0.idx[tokens], [_stack(w) for w in ps],
                              [w.y_base[tokens] for w in ps], w0.h_in)
    assert len(outs) == len(ps)
    for w, (yref, _) in zip(ps, outs):
        assert yref.shape == (tokens.size, w.h_out)
        y64, bound = refs.f64_reference(w, tokens)
        assert (np.abs(yref.astype(np.float64) - y64) <= bound).all()
    # the stacks really differ, and so do the outputs
    assert not np.array_equal(outs[0][0][:, :ps[1].h_out], outs[1][0])
