"""Seeded synthetic workloads for the batched heterogeneous-adapter LoRA apply.

This module only draws inputs: token-to-adapter ids, activations, adapter
stacks, ranks, offsets and scales, as bf16 bit patterns (uint16) plus int and
fp32 arrays.  It holds none of the apply's arithmetic, so the CPU oracle and
the HIP path can both be fed from it without sharing any computation.

The paper's evaluation (section VII-A, Table VII) draws requests over
1000 adapters either uniformly or skewed (80% of requests to 50 adapters),
with ranks drawn from {8, 16, 32, 64, 128} and model dimensions 4096 to 16384
(section V-A).  Its traces (LMSYS Chatbot Arena) are not available; the five
configurations below stand in for them with the shapes, rank mix and skew of
that evaluation:

  tiny     T=8,   h=256,  r=8,  N=4,    idx uniform, s=1, y_base=0
  decode   T=64,  h=4096, r=16, N=1000, idx Zipf(1.0), s=2   (Llama-7B q-proj)
  large    T=256, h=4096, r=64, N=1000, idx uniform, s in {0.5, 1, 2}
  ragged   T=512, h=5120, r in {8,16,32,64}, N=1000, idx Zipf(0.8)  (13B)
  prefill  32 requests of 1..512 tokens, one adapter each, h_in=8192,
           h_out=1024, r=32  (mixed prefill + decode, GQA k/v shape)

Values are N(0, 0.02) for x, A and B (the "paper" scale) and N(0, 1) for
y_base except in ``tiny`` (y_base = 0).  The "parity" scale draws
x ~ N(0,1), A ~ N(0, 1/sqrt(h_in)), B ~ N(0, 1/sqrt(r)) and y_base = 0, so
that the LoRA delta is O(1) and an elementwise tolerance of 1e-2(1+|ref|)
actually tests it.

Zipf(a) over N adapters: P(id = k-1) proportional to k^-a for k = 1..N,
sampled by inverse CDF (numpy's own zipf is unbounded and needs a > 1).

Every array is a pure function of (config, seed, scale); each adapter's A and
B come from their own generator keyed by (seed, adapter id), so drawing only
the adapters a batch uses gives the same bits as drawing the whole stack.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace

import numpy as np

CONFIG_NAMES = ("tiny", "decode", "large", "ragged", "prefill")

# seeds: data seed 1000 + config number, as in the measurement plan
_CONFIG_SEED = {name: 1000 + i for i, name in enumerate(CONFIG_NAMES)}

_TAG_IDX, _TAG_X, _TAG_YB, _TAG_A, _TAG_B, _TAG_RANK, _TAG_SCALE, _TAG_REQ = \
    range(8)


@dataclass
class Workload:
    name: str
    T: int
    n_adapters: int
    h_in: int
    h_out: int
    max_rank: int
    idx: np.ndarray      # int32[T]
    x: np.ndarray        # uint16[T, h_in]   bf16 bits
    y_base: np.ndarray   # uint16[T, h_out]  bf16 bits
    ranks: np.ndarray    # int32[N]
    a_off: np.ndarray    # int64[N] element offsets into A
    b_off: np.ndarray    # int64[N] element offsets into B
    A: np.ndarray        # uint16[a_len]  A_i is h_in x r_i row-major
    B: np.ndarray        # uint16[b_len]  B_i is r_i x h_out row-major
    scales: np.ndarray   # float32[N]
    scale_kind: str = "paper"
    seed: int = 0
    meta: dict = field(default_factory=dict)

    @property
    def a_len(self) -> int:
        return int(self.A.size)

    @property
    def b_len(self) -> int:
        return int(self.B.size)


# ---- bf16 bit patterns of random draws -------------------------------------

def to_bf16_bits(values: np.ndarray) -> np.ndarray:
    """Round fp32 draws to bf16 bit patterns (nearest, ties to even).

    Used only to turn random draws into bf16 inputs; draws are finite."""
    u = np.ascontiguousarray(values, dtype=np.float32).view(np.uint32)
    rounded = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def _rng(seed: int, *tags: int) -> np.random.Generator:
    return np.random.default_rng([seed, *tags])


def _normal_bits(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    return to_bf16_bits(rng.standard_normal(shape, dtype=np.float32) *
                        np.float32(std))


# ---- token-to-adapter id draws ---------------------------------------------

def zipf_ids(rng: np.random.Generator, n: int, N: int, alpha: float) -> np.ndarray:
    """Finite Zipf over ids 0..N-1: P(k-1) ~ k^-alpha, by inverse CDF."""
    w = np.arange(1, N + 1, dtype=np.float64) ** (-alpha)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    u = rng.random(n)
    return np.minimum(np.searchsorted(cdf, u, side="right"), N - 1).astype(np.int32)


def uniform_ids(rng: np.random.Generator, n: int, N: int) -> np.ndarray:
    return rng.integers(0, N, size=n, dtype=np.int64).astype(np.int32)


def prefill_requests(rng: np.random.Generator, n_req: int, max_len: int, N: int):
    """Request lengths U{1..max_len}, one adapter per request, U[0, N)."""
    lens = rng.integers(1, max_len + 1, size=n_req)
    ads = rng.integers(0, N, size=n_req)
    return lens.astype(np.int64), ads.astype(np.int32)


# ---- configurations ---------------------------------------------------------

@dataclass(frozen=True)
class ConfigShape:
    T: int | None
    N: int
    h_in: int
    h_out: int
    rank: int | tuple
    dist: str            # "uniform", "zipf", "requests"
    alpha: float = 0.0
    scale: float | tuple = 1.0
    y_base: str = "normal"
    n_req: int = 0
    max_len: int = 0


CONFIGS = {
    "tiny": ConfigShape(8, 4, 256, 256, 8, "uniform", scale=1.0, y_base="zero"),
    "decode": ConfigShape(64, 1000, 4096, 4096, 16, "zipf", alpha=1.0, scale=2.0),
    "large": ConfigShape(256, 1000, 4096, 4096, 64, "uniform",
                         scale=(0.5, 1.0, 2.0)),
    "ragged": ConfigShape(512, 1000, 5120, 5120, (8, 16, 32, 64), "zipf",
                          alpha=0.8, scale=1.0),
    "prefill": ConfigShape(None, 1000, 8192, 1024, 32, "requests", scale=1.0,
                           n_req=32, max_len=512),
}


def draw_idx(name: str, seed: int, draw: int = 0) -> np.ndarray:
    """Token-to-adapter ids for one batch of config ``name``.

    ``draw`` selects an independent batch (the benchmark takes a fresh one
    per step); draw 0 is the batch the config's workload carries."""
    c = CONFIGS[name]
    rng = _rng(seed, _TAG_IDX, draw)
    if c.dist == "uniform":
        return uniform_ids(rng, c.T, c.N)
    if c.dist == "zipf":
        return zipf_ids(rng, c.T, c.N, c.alpha)
    lens, ads = prefill_requests(rng, c.n_req, c.max_len, c.N)
    return np.repeat(ads, lens).astype(np.int32)


def _ranks(name: str, seed: int) -> np.ndarray:
    c = CONFIGS[name]
    if isinstance(c.rank, tuple):
        rng = _rng(seed, _TAG_RANK)
        return np.asarray(c.rank, np.int32)[rng.integers(0, len(c.rank), c.N)]
    return np.full(c.N, c.rank, np.int32)


def _scales(name: str, seed: int) -> np.ndarray:
    c = CONFIGS[name]
    if isinstance(c.scale, tuple):
        rng = _rng(seed, _TAG_SCALE)
        return np.asarray(c.scale, np.float32)[rng.integers(0, len(c.scale), c.N)]
    return np.full(c.N, c.scale, np.float32)


def _stds(kind: str, h_in: int, r: int):
    if kind == "paper":
        return 0.02, 0.02, 0.02
    if kind == "parity":
        return 1.0, 1.0 / np.sqrt(h_in), 1.0 / np.sqrt(max(r, 1))
    raise ValueError(kind)


def fill_adapters(A: np.ndarray, B: np.ndarray, ranks, a_off, b_off, h_in: int,
                  h_out: int, seed: int, kind: str, ids) -> None:
    """Draw A_i and B_i in place for every adapter id in ``ids``."""
    for i in ids:
        i = int(i)
        r = int(ranks[i])
        if r == 0:
            continue
        _, sa, sb = _stds(kind, h_in, r)
        A[a_off[i]:a_off[i] + h_in * r] = _normal_bits(
            _rng(seed, _TAG_A, i), h_in * r, sa)
        B[b_off[i]:b_off[i] + r * h_out] = _normal_bits(
            _rng(seed, _TAG_B, i), r * h_out, sb)


def make_workload(name: str, seed: int | None = None, scale: str = "paper",
                  only_used: bool = False, idx: np.ndarray | None = None,
                  n_adapters: int | None = None, h_out: int | None = None,
                  stack_seed: int | None = None, ranks=None) -> Workload:
    """Build config ``name``.

    only_used: draw A/B only for adapters that ``idx`` references (the other
    adapters are zero); their bits match a full draw.
    idx / n_adapters: override the id draw or the adapter count (shapes stay).
    h_out / stack_seed: another projection of the same layer: its own output
    width and adapter stack (A/B drawn from stack_seed), with x, the ids, the
    ranks and the scales of ``seed``.
    ranks: override the config's ranks: one int for every adapter, or an
    int array of N entries (any values 0..128; blocks stay back to back).
    """
    c = CONFIGS[name]
    if h_out is not None:
        c = replace(c, h_out=h_out)
    if seed is None:
        seed = _CONFIG_SEED[name]
    N = c.N if n_adapters is None else n_adapters
    if idx is None:
        idx = draw_idx(name, seed)
    idx = np.ascontiguousarray(idx, np.int32)
    T = idx.size
    if ranks is not None:
        ranks = np.array(np.broadcast_to(np.asarray(ranks, np.int32), (N,)))
    elif N <= c.N:
        ranks = _ranks(name, seed)[:N]
    else:
        ranks = np.resize(_ranks(name, seed), N)
    scales = _scales(name, seed)[:N] if N <= c.N else np.resize(_scales(name, seed), N)
    ranks = np.ascontiguousarray(ranks, np.int32)
    scales = np.ascontiguousarray(scales, np.float32)
    a_sizes = ranks.astype(np.int64) * c.h_in
    b_sizes = ranks.astype(np.int64) * c.h_out
    a_off = np.concatenate([[0], np.cumsum(a_sizes)[:-1]]).astype(np.int64)
    b_off = np.concatenate([[0], np.cumsum(b_sizes)[:-1]]).astype(np.int64)
    A = np.zeros(int(a_sizes.sum()), np.uint16)
    B = np.zeros(int(b_sizes.sum()), np.uint16)
    ids = np.unique(idx[(idx >= 0) & (idx < N)]) if only_used else range(N)
    fill_adapters(A, B, ranks, a_off, b_off, c.h_in, c.h_out,
                  seed if stack_seed is None else stack_seed, scale, ids)
    sx, _, _ = _stds(scale, c.h_in, int(ranks.max()) if N else 1)
    x = _normal_bits(_rng(seed, _TAG_X), (T, c.h_in), sx)
    if scale == "parity" or c.y_base == "zero":
        y_base = np.zeros((T, c.h_out), np.uint16)
    else:
        ys = seed if stack_seed is None else stack_seed
        y_base = _normal_bits(_rng(ys, _TAG_YB), (T, c.h_out), 1.0)
    return Workload(name=name, T=T, n_adapters=N, h_in=c.h_in, h_out=c.h_out,
                    max_rank=int(ranks.max()) if N else 0, idx=idx, x=x,
                    y_base=y_base, ranks=ranks, a_off=a_off, b_off=b_off, A=A,
                    B=B, scales=scales, scale_kind=scale, seed=seed)


# The LoRA-injected projections of one layer that read the same x, per
# config: Llama-2-7B's attention projections q, k, v (4096 -> 4096 each,
# section VII-A's 7B model) for the decode shape; for the prefill shape, the
# GQA k and v projections (8192 -> 1024) and the q projection (8192 -> 8192).
PROJECTIONS = {
    "tiny": (256, 256, 128),
    "decode": (4096, 4096, 4096),
    "large": (4096, 4096, 4096),
    "ragged": (5120, 5120, 5120),
    "prefill": (8192, 1024, 1024),
}


def make_projections(name: str, n_proj: int | None = None, seed: int | None = None,
                     scale: str = "paper", idx: np.ndarray | None = None,
                     h_outs=None) -> list:
    """Workloads of the projections of one layer sharing x and the ids: the
    first is ``make_workload(name, ...)`` itself; projection p > 0 has its
    own adapter stack (drawn from seed + 7919 p) and output width."""
    if seed is None:
        seed = _CONFIG_SEED[name]
    hs = list(PROJECTIONS[name] if h_outs is None else h_outs)
    if n_proj is not None:
        hs = hs[:n_proj]
    out = [make_workload(name, seed, scale, idx=idx, h_out=hs[0])]
    for p in range(1, len(hs)):
        out.append(make_workload(name, seed, scale, idx=out[0].idx, h_out=hs[p],
                                 stack_seed=seed + 7919 * p))
    return out


def with_idx(w: Workload, idx: np.ndarray) -> Workload:
    """Same adapters and activations' draw, different token ids (T may change:
    x and y_base are redrawn for the new T)."""
    idx = np.ascontiguousarray(idx, np.int32)
    if idx.size == w.T:
        return replace(w, idx=idx)
    sx, _, _ = _stds(w.scale_kind, w.h_in, max(w.max_rank, 1))
    x = _normal_bits(_rng(w.seed, _TAG_X, idx.size), (idx.size, w.h_in), sx)
    if w.scale_kind == "parity" or not w.y_base.any():
        yb = np.zeros((idx.size, w.h_out), np.uint16)
    else:
        yb = _normal_bits(_rng(w.seed, _TAG_YB, idx.size), (idx.size, w.h_out), 1.0)
    return replace(w, idx=idx, T=idx.size, x=x, y_base=yb)


def adapter_bytes(ranks: np.ndarray, idx: np.ndarray, h_in: int, h_out: int,
                  n_adapters: int) -> int:
    """Bytes of A and B that one call must read: 2 r_i (h_in + h_out) per
    distinct valid adapter in the batch (the cost model's memory term,
    section VI-B, with bf16 values and h_in, h_out in place of D)."""
    idx = np.asarray(idx)
    ids = np.unique(idx[(idx >= 0) & (idx < n_adapters)])
    return int(2 * np.sum(ranks[ids].astype(np.int64)) * (h_in + h_out))
