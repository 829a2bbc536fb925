"""Pins of the split-KV decode attention oracle (section V-B): closed forms,
special cases that reduce to a library softmax, and the merge's equivalence
to the plain definition for any partition size and any arrival order."""
import numpy as np
import pytest
import scipy.special

import oracle
from oracle import attention as OA

D = 16


def bits(a):
    return oracle.f32_to_bf16(np.asarray(a, np.float32))


def rand_case(seed, Bn=3, H=2, Lmax=37, d=D, lens=None, sc=1.0):
    rng = np.random.default_rng(seed)
    q = bits(rng.normal(0, sc, (Bn, H, d)))
    K = bits(rng.normal(0, sc, (Bn, H, Lmax, d)))
    V = bits(rng.normal(0, 1, (Bn, H, Lmax, d)))
    lens = rng.integers(1, Lmax + 1, Bn) if lens is None else np.asarray(lens)
    return q, K, V, lens


def test_zero_query_averages_the_values():
    q, K, V, lens = rand_case(1)
    q[:] = 0
    o = OA.attention(q, K, V, lens, 0.25)
    Vf = oracle.bf16_to_f32(V).astype(np.float64)
    for b, n in enumerate(lens):
        assert np.allclose(o[b], Vf[b, :, :n].mean(axis=1), rtol=0, atol=1e-14)


def test_single_key_returns_its_value_exactly():
    q, K, V, _ = rand_case(2)
    o = OA.attention(q, K, V, [1, 1, 1], 0.5)
    assert np.array_equal(o, oracle.bf16_to_f32(V)[:, :, 0].astype(np.float64))


def test_matches_a_library_softmax():
    q, K, V, lens = rand_case(3)
    scale = 1 / np.sqrt(D)
    o = OA.attention(q, K, V, lens, scale)
    qf, Kf, Vf = (oracle.bf16_to_f32(a).astype(np.float64) for a in (q, K, V))
    for b, n in enumerate(lens):
        for h in range(q.shape[1]):
            p = scipy.special.softmax(scale * Kf[b, h, :n] @ qf[b, h])
            assert np.allclose(o[b, h], p @ Vf[b, h, :n], rtol=1e-13, atol=1e-14)


def test_a_dominant_key_takes_all_the_weight():
    q, K, V, _ = rand_case(4, Bn=1, H=1, Lmax=9)
    qf = np.zeros(D, np.float32)
    qf[0] = 8.0
    Kf = np.zeros((1, 1, 9, D), np.float32)
    Kf[0, 0, 5, 0] = 8.0                     # score 64 * scale against 0 elsewhere
    o = OA.attention(bits(qf[None, None]), bits(Kf), V, [9], 1.0)
    assert np.allclose(o[0, 0], oracle.bf16_to_f32(V)[0, 0, 5], rtol=0, atol=1e-25)


def test_scores_beyond_exp_range_stay_finite():
    # raw exp(s) would overflow; the anchor keeps every exponent <= 0
    q, K, V, lens = rand_case(5, sc=4.0)
    o = OA.attention(q, K, V, lens, 200.0)
    m, l, op = OA.partial(q, K, V, lens, 200.0, 5)
    assert np.isfinite(o).all() and np.isfinite(OA.merge(m, l, op)).all()
    assert np.allclose(OA.merge(m, l, op), o, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("chunk", [1, 3, 7, 16, 37, 64])
def test_merged_partials_equal_the_definition(chunk):
    q, K, V, lens = rand_case(6)
    scale = 1 / np.sqrt(D)
    m, l, o = OA.partial(q, K, V, lens, scale, chunk)
    assert np.allclose(OA.merge(m, l, o), OA.attention(q, K, V, lens, scale),
                       rtol=1e-12, atol=1e-13)


def test_any_arrival_order_gives_the_same_output():
    q, K, V, lens = rand_case(7, Lmax=64)
    m, l, o = OA.partial(q, K, V, lens, 0.3, 4)
    ref = OA.merge(m, l, o)
    rng = np.random.default_rng(0)
    for _ in range(10):
        order = rng.permutation(m.shape[2])
        assert np.allclose(OA.merge(m, l, o, order), ref, rtol=1e-13, atol=1e-14)


def test_empty_partitions_and_requests():
    q, K, V, _ = rand_case(8, Lmax=20)
    lens = np.array([0, 3, 20])
    m, l, o = OA.partial(q, K, V, lens, 0.5, 8)
    assert (m[0] == -np.inf).all() and (l[0] == 0).all() and (o[0] == 0).all()
    assert (m[1, :, 1:] == -np.inf).all()             # keys 8.. are past len 3
    out = OA.merge(m, l, o)
    assert (out[0] == 0).all()
    assert np.allclose(out, OA.attention(q, K, V, lens, 0.5), rtol=1e-12, atol=1e-13)
