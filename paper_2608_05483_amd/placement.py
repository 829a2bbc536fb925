"""Where each adapter lives: HBM or a pinned host pool (strategies E1 and E2).

The paper keeps every adapter in pooled memory and uses GPU memory as a
software-managed cache for it (section V-A).  On one MI355X the pool is pinned
host memory the kernels read directly (plora_adapters' A_pool / B_pool), so two
of its four strategies exist here:

  E1  A_i and B_i cached in HBM; the apply reads them there;
  E2  neither cached; the apply reads them from the pool over the host link.

(E3 and E4 need compute beside the pooled memory.)  This module holds the
decision, host logic only:

* ``cost_e1`` / ``cost_e2`` / ``lora_time``: the E1 and E2 rows of the
  per-strategy cost terms (Table IV, section VI-B), with the host link's bandwidth
  ``W_link`` and round trip ``L_link`` in place of the CXL link's, and the
  square model dimension D generalised to h_in and h_out (4 B D R flops
  become 2 B R (h_in + h_out), 2 D S R bytes become S R (h_in + h_out));
* ``Temperature``: the hot / cold metric of section VI-A (each request raises
  its adapter's temperature by a fixed increment, every step relaxes all
  temperatures toward the average by 0.1 of the gap);
* ``choose``: the strategy selection of Algorithm 1 (section VI-A) over
  {E1, E2}, per serving adapter, under an HBM budget: take the faster
  strategy by the cost model if it fits; otherwise evict cold adapters; if
  they are not enough, re-rank "E1 evicting hot adapters", "E1 evicting other
  serving adapters" (which then run as E2) and E2 by the cost model.  The
  paper's fourth candidate, evicting KV cache, has no counterpart here.
  Afterwards the hottest non-serving adapters (up to 50) are pre-cached in
  what budget is left;
* ``HbmCache``: the device side of a decision: an HBM slab of fixed capacity
  holding the cached adapters' blocks, the offsets that name slab or pool for
  each adapter, and the copies that bring an adapter in.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

E1, E2 = "E1", "E2"


@dataclass(frozen=True)
class Hardware:
    """The cost model's hardware parameters.  C_gpu: matrix throughput
    (flop/s); W_gpu: HBM bandwidth (B/s); W_link, L_link: the bandwidth (B/s)
    and round-trip latency (s) of the GPU's reads from pinned host memory;
    S: bytes per value."""
    C_gpu: float = 2.5e15
    W_gpu: float = 8.0e12
    W_link: float = 5.0e10
    L_link: float = 2.0e-6
    S: int = 2


def adapter_bytes(rank: int, h_in: int, h_out: int, S: int = 2) -> int:
    """Bytes of A_i and B_i together: S r (h_in + h_out)."""
    return int(S) * int(rank) * (int(h_in) + int(h_out))


def _terms(B, ranks, sel, h_in, h_out, S):
    B = np.asarray(B, np.int64)
    ranks = np.asarray(ranks, np.int64)
    sel = np.asarray(sel, bool)
    flops = 2.0 * (h_in + h_out) * float(np.sum(B[sel] * ranks[sel]))
    used = sel & (B > 0)
    nbytes = float(S) * (h_in + h_out) * float(np.sum(ranks[used]))
    return flops, nbytes, bool(used.any())


def cost_e1(B, ranks, sel, h_in: int, h_out: int, hw: Hardware) -> float:
    """T_GPU_E1 for the adapters selected by sel: max(compute, HBM reads of
    the adapters serving at least one request), zero without work."""
    flops, nbytes, any_used = _terms(B, ranks, sel, h_in, h_out, hw.S)
    if not any_used:
        return 0.0
    return max(flops / hw.C_gpu, nbytes / hw.W_gpu)


def cost_e2(B, ranks, sel, h_in: int, h_out: int, hw: Hardware) -> float:
    """T_GPU_E2: max(compute, two link latencies plus the pool reads over
    the link), zero without work."""
    flops, nbytes, any_used = _terms(B, ranks, sel, h_in, h_out, hw.S)
    if not any_used:
        return 0.0
    return max(flops / hw.C_gpu, 2.0 * hw.L_link + nbytes / hw.W_link)


def lora_time(B, ranks, strategy, h_in: int, h_out: int, hw: Hardware) -> float:
    """T_LoRA_GPU = T_GPU_E1 + T_GPU_E2 for a per-adapter strategy array
    (values E1 / E2; adapters without requests cost nothing)."""
    strategy = np.asarray(strategy)
    return (cost_e1(B, ranks, strategy == E1, h_in, h_out, hw) +
            cost_e2(B, ranks, strategy == E2, h_in, h_out, hw))


class Temperature:
    """Per-adapter temperature: request() raises one adapter's by
    `increment`; step() moves every temperature toward the current average by
    `relax` of the gap."""

    def __init__(self, n: int, increment: float = 1.0, relax: float = 0.1):
        self.t = np.zeros(int(n), np.float64)
        self.increment = float(increment)
        self.relax = float(relax)

    def request(self, adapters) -> None:
        np.add.at(self.t, np.asarray(adapters, np.int64), self.increment)

    def step(self) -> None:
        self.t += self.relax * (self.t.mean() - self.t)

    def order(self, candidates) -> np.ndarray:
        """candidates hottest first (ties: lower id first)."""
        c = np.asarray(candidates, np.int64)
        return c[np.lexsort((c, -self.t[c]))]


@dataclass
class Decision:
    strategy: np.ndarray                # E1 / E2 for every adapter (non-serving: where it lives)
    resident: np.ndarray                # bool: cached in HBM after this step
    loads: list = field(default_factory=list)     # adapters to bring into HBM
    evictions: list = field(default_factory=list)  # adapters dropped from HBM
    cost: float = 0.0                   # lora_time of the serving adapters


def choose(B, ranks, h_in: int, h_out: int, hw: Hardware, budget: int, resident,
           temp: Temperature, n_hot: int = 50) -> Decision:
    """One step of the selection for batch counts B (requests per adapter):
    serving adapters in descending order of B (ties: lower id), each placed as
    described in the module docstring, then pre-caching.  `resident` (bool
    array) is what HBM holds before the step; the result never holds more
    than `budget` bytes."""
    B = np.asarray(B, np.int64)
    ranks = np.asarray(ranks, np.int64)
    n = B.size
    res = np.array(resident, bool, copy=True)
    size = np.array([adapter_bytes(r, h_in, h_out, hw.S) for r in ranks], np.int64)
    used = int(size[res].sum())
    strategy = np.where(res, E1, E2).astype(object)
    serving = np.nonzero(B > 0)[0]
    serving = serving[np.lexsort((serving, -B[serving]))]
    non_serving = np.setdiff1d(np.arange(n), serving)
    hot = set(temp.order(non_serving)[:n_hot].tolist())
    loads, evictions = [], []

    def evict(a):
        nonlocal used
        res[a] = False
        used -= int(size[a])
        strategy[a] = E2
        if int(a) in loads:              # brought in earlier in this step
            loads.remove(int(a))
        else:
            evictions.append(int(a))

    def load(a):
        nonlocal used
        res[a] = True
        used += int(size[a])
        strategy[a] = E1
        if int(a) in evictions:          # dropped earlier in this step: keep it
            evictions.remove(int(a))
        else:
            loads.append(int(a))

    def cost_with(a, e, strategy_now):
        s = strategy_now.copy()
        s[a] = e
        return lora_time(B, ranks, s, h_in, h_out, hw)

    placed = set()
    for a in serving:
        placed.add(int(a))
        if res[a]:
            strategy[a] = E1            # cached already: E1 costs no memory
            continue
        c1, c2 = cost_with(a, E1, strategy), cost_with(a, E2, strategy)
        if c2 <= c1:
            strategy[a] = E2
            continue
        need = used + int(size[a]) - budget
        if need <= 0:
            load(a)
            continue
        # cold adapters: cached, not serving, not hot; coldest first
        cold = [c for c in temp.order(np.nonzero(res)[0])[::-1]
                if c not in hot and B[c] == 0]
        if sum(int(size[c]) for c in cold) >= need:
            freed = 0
            for c in cold:
                if freed >= need:
                    break
                freed += int(size[c])
                evict(c)
            load(a)
            continue
        # not enough cold bytes: re-rank E2, E1 evicting hot adapters, E1
        # evicting other cached serving adapters (not yet placed ones first:
        # lowest batch first), by the cost model
        cands = [(c2, 0, "E2", [])]
        hot_cached = [h for h in temp.order(np.nonzero(res)[0])[::-1] if h in hot]
        for label, pool_, rank_ in (("hot", cold + hot_cached, 1),
                                    ("serving", None, 2)):
            if pool_ is None:
                others = [s for s in np.nonzero(res)[0] if B[s] > 0 and s != a]
                others.sort(key=lambda s: (int(s) in placed, B[s], -s))
                pool_ = cold + hot_cached + others
            freed, victims = 0, []
            for c in pool_:
                if freed >= need:
                    break
                freed += int(size[c])
                victims.append(int(c))
            if freed < need:
                continue
            s = strategy.copy()
            for v in victims:
                s[v] = E2
            s[a] = E1
            cands.append((lora_time(B, ranks, s, h_in, h_out, hw), rank_, label, victims))
        cands.sort(key=lambda c: (c[0], c[1]))
        _, _, label, victims = cands[0]
        if label == "E2":
            strategy[a] = E2
            continue
        for v in victims:
            evict(v)
        load(a)
    # pre-cache the hottest non-serving adapters into what budget is left
    for h in temp.order(non_serving)[:n_hot]:
        if res[h]:
            continue
        if used + int(size[h]) <= budget:
            load(h)
    for a in range(n):
        if B[a] == 0:
            strategy[a] = E1 if res[a] else E2
    assert used <= budget
    cost = lora_time(B, ranks, strategy, h_in, h_out, hw)
    return Decision(strategy=np.array(strategy, dtype=object), resident=res, loads=loads,
                    evictions=evictions, cost=cost)


class HbmCache:
    """The device side of the decisions: a slab of HBM of `budget` bytes that
    holds the cached adapters' A and B blocks, first fit over free ranges;
    A_pool / B_pool (pinned host tensors) hold every adapter at its pool
    offsets.  offsets() gives the a_off / b_off arrays plora_adapters takes
    (slab element offsets, or -1 - pool offset)."""

    def __init__(self, A_pool, B_pool, a_pool_off, b_pool_off, ranks, h_in: int, h_out: int,
                 budget: int, device="cuda"):
        import torch
        self.A_pool, self.B_pool = A_pool, B_pool
        self.a_pool_off = np.asarray(a_pool_off, np.int64)
        self.b_pool_off = np.asarray(b_pool_off, np.int64)
        self.ranks = np.asarray(ranks, np.int64)
        self.h_in, self.h_out = int(h_in), int(h_out)
        # A blocks take h_in / (h_in + h_out) of an adapter's bytes; one largest
        # block of slack per slab absorbs first-fit fragmentation of mixed ranks
        rmax = int(self.ranks.max()) if self.ranks.size else 8
        up8 = lambda v: (int(v) + 7) // 8 * 8
        ea = up8(int(budget) // 2 * self.h_in // (self.h_in + self.h_out)) + self.h_in * rmax
        eb = up8(int(budget) // 2 * self.h_out // (self.h_in + self.h_out)) + self.h_out * rmax
        self.A = torch.zeros(ea, dtype=torch.int16, device=device)
        self.B = torch.zeros(eb, dtype=torch.int16, device=device)
        self.free = [(0, ea)]               # free (start, length) ranges, in elements
        self.free_b = [(0, eb)]
        self.slot = {}                      # adapter -> (a start, b start)

    @staticmethod
    def _take(free, n):
        for k, (s, l) in enumerate(free):
            if l >= n:
                free[k] = (s + n, l - n)
                if free[k][1] == 0:
                    free.pop(k)
                return s
        return None

    @staticmethod
    def _give(free, s, n):
        free.append((s, n))
        free.sort()
        merged = []
        for a, l in free:
            if merged and merged[-1][0] + merged[-1][1] == a:
                merged[-1] = (merged[-1][0], merged[-1][1] + l)
            else:
                merged.append((a, l))
        free[:] = merged

    def apply(self, d: Decision, stream=None) -> None:
        """Evict, then copy the loaded adapters' blocks from the pools into
        the slab (on the current stream)."""
        for a in d.evictions:
            sa, sb = self.slot.pop(a)
            na, nb = self.h_in * int(self.ranks[a]), self.h_out * int(self.ranks[a])
            self._give(self.free, sa, (na + 7) // 8 * 8)
            self._give(self.free_b, sb, (nb + 7) // 8 * 8)
        for a in d.loads:
            na, nb = self.h_in * int(self.ranks[a]), self.h_out * int(self.ranks[a])
            sa = self._take(self.free, (na + 7) // 8 * 8)
            sb = self._take(self.free_b, (nb + 7) // 8 * 8)
            if sa is None or sb is None:
                raise RuntimeError("HBM slab fragmented: no free range for adapter %d" % a)
            pa, pb = int(self.a_pool_off[a]), int(self.b_pool_off[a])
            self.A[sa:sa + na].copy_(self.A_pool[pa:pa + na], non_blocking=True)
            self.B[sb:sb + nb].copy_(self.B_pool[pb:pb + nb], non_blocking=True)
            self.slot[a] = (sa, sb)

    def offsets(self):
        a_off = -1 - self.a_pool_off
        b_off = -1 - self.b_pool_off
        for a, (sa, sb) in self.slot.items():
            a_off[a] = sa
            b_off[a] = sb
        return a_off.astype(np.int64), b_off.astype(np.int64)
