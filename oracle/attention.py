"""CPU oracle for split-KV decode attention (section V-B).

TEST INFRASTRUCTURE ONLY.  Only ``tests/`` and ``bench.py``'s ``cpu_baseline``
leg may import this module; the product library never does, and the two share
no code.

Decode attention of one request b and head h over its KV cache of len_b keys:

    s_t = scale * <q, k_t>,  t < len_b;   o = sum_t softmax(s)_t v_t.

The paper spreads the KV cache over devices, has each compute the three steps
(scores, softmax, weighted sum of values) on its share with the partial
softmax of FlashAttention, keep an anchor, and lets the GPU rescale the
partial outputs into the exact global one, in whatever order they arrive
(section V-B).  Here a "partition" is a range of chunk keys:

    m_p = max_{t in p} s_t                         (the anchor)
    l_p = sum_{t in p} exp(s_t - m_p)
    o_p = sum_{t in p} exp(s_t - m_p) v_t          (not yet divided by l)

and the merge takes M = max_p m_p, w_p = exp(m_p - M), L = sum_p w_p l_p,
o = sum_p w_p o_p / L.  Everything is float64 from the bf16 bits.  Readings:
an empty partition has m = -inf, l = 0, o = 0 and contributes nothing; a
request with len_b = 0 gets o = 0 (a softmax over no keys is undefined).
"""
from __future__ import annotations

import numpy as np

from . import bf16_to_f32


def _f64(bits) -> np.ndarray:
    return bf16_to_f32(np.asarray(bits, np.uint16)).astype(np.float64)


def attention(q, K, V, lens, scale: float) -> np.ndarray:
    """The definition: q [B, H, d], K and V [B, H, Lmax, d] (bf16 bits), lens
    int [B]; returns o float64 [B, H, d]."""
    q, K, V = _f64(q), _f64(K), _f64(V)
    Bn, H, d = q.shape
    out = np.zeros((Bn, H, d), np.float64)
    for b in range(Bn):
        n = int(lens[b])
        if n <= 0:
            continue
        for h in range(H):
            s = scale * (K[b, h, :n] @ q[b, h])
            e = np.exp(s - s.max())
            out[b, h] = (e / e.sum()) @ V[b, h, :n]
    return out


def partial(q, K, V, lens, scale: float, chunk: int):
    """Each partition's anchor, sum and unnormalised output: m, l [B, H, P]
    and o [B, H, P, d] with P = ceil(Lmax / chunk)."""
    q, K, V = _f64(q), _f64(K), _f64(V)
    Bn, H, Lmax, d = K.shape
    P = max(1, -(-Lmax // chunk))
    m = np.full((Bn, H, P), -np.inf)
    l = np.zeros((Bn, H, P))
    o = np.zeros((Bn, H, P, d))
    for b in range(Bn):
        n = int(lens[b])
        for h in range(H):
            for p in range(P):
                lo, hi = p * chunk, min((p + 1) * chunk, n)
                if lo >= hi:
                    continue
                s = scale * (K[b, h, lo:hi] @ q[b, h])
                m[b, h, p] = s.max()
                e = np.exp(s - m[b, h, p])
                l[b, h, p] = e.sum()
                o[b, h, p] = e @ V[b, h, lo:hi]
    return m, l, o


def merge(m, l, o, order=None) -> np.ndarray:
    """Rescale the partials into the global output, taking the partitions in
    `order` (default ascending); rows whose partitions are all empty get 0."""
    Bn, H, P = m.shape
    order = range(P) if order is None else order
    out = np.zeros(o.shape[:2] + o.shape[3:])
    for b in range(Bn):
        for h in range(H):
            M = max(m[b, h, p] for p in order)
            if M == -np.inf:
                continue
            L = 0.0
            acc = np.zeros(o.shape[3])
            for p in order:
                if m[b, h, p] == -np.inf:
                    continue
                w = np.exp(m[b, h, p] - M)
                L += w * l[b, h, p]
                acc += w * o[b, h, p]
            out[b, h] = acc / L
    return out
