"""float64 references and rigorous rounding-error bounds shared by the tests.

For one token with adapter i (rank r), fp32 evaluation of
    y = y_base + s * (x A_i) B_i
with bf16 inputs (exact products x*A in fp32) and any summation order obeys
    |y_fp32 - y_exact| <= E = gamma_{h_in + r + 2} * (|s| ((S + |v|) @ |B_i|)
                                                      + |y_base| + |s d|)
where v = x A_i, S = |x| @ |A_i|, d = v B_i (the standard recursive-summation
bound gamma_n = n u / (1 - n u), u = 2^-24, applied to both contractions and
the final scale-and-add).  A bf16 store adds at most half a bf16 ulp.
"""
from __future__ import annotations

import numpy as np

U = 2.0 ** -24


def gamma(n: int) -> float:
    return n * U / (1 - n * U)


def dec(bits) -> np.ndarray:
    return (np.asarray(bits, np.uint32) << 16).view(np.float32).astype(np.float64)


def bf16_half_ulp(a: np.ndarray) -> np.ndarray:
    """Half the spacing of bf16 numbers at magnitude a (a >= 0)."""
    a = np.maximum(np.asarray(a, np.float64), 2.0 ** -126)
    e = np.floor(np.log2(a))
    return 0.5 * 2.0 ** (e - 7)


def f64_reference(w, tokens, idx=None, x=None, y_base=None, scales=None, ranks=None):
    """float64 y and the fp32 error bound E for the given token rows."""
    idx = w.idx if idx is None else idx
    x = w.x if x is None else x
    y_base = w.y_base if y_base is None else y_base
    scales = w.scales if scales is None else scales
    ranks = w.ranks if ranks is None else ranks
    ys, bounds = [], []
    for t in tokens:
        i = int(idx[t])
        yb = dec(y_base[t])
        if not 0 <= i < w.n_adapters or ranks[i] == 0:
            ys.append(yb)
            bounds.append(np.zeros_like(yb))
            continue
        r = int(ranks[i])
        Ai = dec(w.A[w.a_off[i]:w.a_off[i] + w.h_in * r]).reshape(w.h_in, r)
        Bi = dec(w.B[w.b_off[i]:w.b_off[i] + r * w.h_out]).reshape(r, w.h_out)
        xt = dec(x[t])
        s = float(scales[i])
        v = xt @ Ai
        S = np.abs(xt) @ np.abs(Ai)
        d = v @ Bi
        y = yb + s * d
        E = (gamma(w.h_in + r + 2) *
             (abs(s) * ((S + np.abs(v)) @ np.abs(Bi)) + np.abs(yb) + abs(s) * np.abs(d))
             ) * 1.01 + 1e-300
        ys.append(y)
        bounds.append(E)
    return np.array(ys), np.array(bounds)


def sample_tokens(T: int, k: int = 64, seed: int = 0) -> np.ndarray:
    if T <= k:
        return np.arange(T)
    return np.sort(np.random.default_rng(seed).choice(T, k, replace=False))
