#!/usr/bin/env python3
"""Benchmark: the batched heterogeneous-adapter LoRA apply on one MI355X.

One step = one pass of the whole hot path over one batch already resident in
HBM: plora_segment_apply, which groups the batch's tokens by adapter (the
plora_segment outputs) and applies y += s_i (x A_i) B_i for every token.  For
batches of up to 256 tokens that is one launch; larger batches take
plora_segment then plora_apply.  With --projections > 1 a step is
plora_segment then one plora_apply_multi.  Each step takes a fresh
token-to-adapter draw from a pool drawn up front, a different replica of the
adapter stack and a different replica of the activations, so that neither an
adapter's bytes nor x and y are still sitting in the 256 MB Infinity Cache
from an earlier step (a served model revisits one projection's stack only
after every other LoRA projection of every layer).

Prints ONE JSON line.  The top level is the headline configuration (--config,
the 1000-adapter Llama-7B-shaped decode batch by default); ``configs`` holds
the same measurements for the other workloads (large decode batch, ragged
ranks, prefill + decode), taken in the same run.  ``value`` is whole-job
tokens/s over the timed steps (wall clock), the K steps launched as one
captured HIP graph (``--eager``: one launch per call from Python).
``roofline`` prices the dominant kernel: algorithmic bytes per step
(distinct adapters' A_i and B_i, 2 r_i (h_in + h_out) bytes each, plus x
read, y read and written, and the token ids) over that kernel's average
duration.  Where a step is one launch, that is the step graph's duration
between two HIP events recorded on the stream the kernels run on; otherwise
it is the apply's: K plora_apply calls captured as one graph and replayed
between two such events.  ``read_ceiling`` is a plain 128-bit read of exactly
the adapter blocks each step touches, timed the same way (K launches in one
graph).  ``cpu_baseline`` times the CPU oracle on a bounded sample of the
headline workload.
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

HBM_PEAK_GBPS = 8000.0
MALL_BYTES = 256 << 20
ROOT = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(ROOT, "paper_2608_05483_amd", "csrc")
PROFILES = os.path.join(ROOT, "profiles")
EXTRA_DEFAULT = ("large", "ragged", "prefill")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="decode",
                    choices=["tiny", "decode", "large", "ragged", "prefill"],
                    help="the headline workload (top level of the JSON line)")
    ap.add_argument("--also", default="auto",
                    help="comma-separated workloads also measured in this run and reported "
                         "under 'configs' ('auto': large, ragged and prefill next to the "
                         "decode headline, none otherwise; 'none')")
    ap.add_argument("--draws", type=int, default=64,
                    help="distinct token-to-adapter draws cycled through")
    ap.add_argument("--replicas", type=int, default=0,
                    help="adapter-stack replicas rotated per step (0 = auto)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-ceiling", action="store_true")
    ap.add_argument("--projections", type=int, default=1,
                    help="LoRA-injected projections of one layer sharing x, applied "
                         "by one plora_apply_multi call (1: plora_apply)")
    ap.add_argument("--pool-from", type=int, default=-1, metavar="K",
                    help="also time the apply with adapters K.. read from a pinned host "
                         "pool (strategy E2) and the rest from HBM (E1), next to the "
                         "all-HBM apply, with the cost model's prediction for both")
    ap.add_argument("--workload", default="apply", choices=["apply", "attention"],
                    help="attention: the split-KV decode attention (plora_attn_decode) at "
                         "Llama-2-7B decode shape instead of the LoRA apply")
    ap.add_argument("--eager", action="store_true",
                    help="time the steps as individual launches instead of one graph")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run 10 plain device copies of MIB MiB (the reference "
                         "kernel for scaling HBM byte counters) and exit")
    return ap.parse_args()


def kernel_sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.h")))


def source_digest() -> str:
    """sha256 over every kernel source file (names and contents)."""
    h = hashlib.sha256()
    for path in kernel_sources():
        h.update(os.path.basename(path).encode())
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(stem: str):
    """HBM bytes per launch of the priced kernel from the committed counter
    summary (profiles/<stem>_traffic.txt, stem = kernel and workload), or
    None when there is none or the kernel sources have changed since the
    counters were taken."""
    path = os.path.join(PROFILES, f"{stem}_traffic.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        parts = line.split()
        if len(parts) == 2 and parts[0].endswith(":"):
            kv[parts[0][:-1]] = parts[1]
    if kv.get("source_sha256") != source_digest():
        return None
    try:
        return int(kv["fetch_bytes_per_launch"]) + int(kv["write_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def copy_calibration(mib: int):
    import torch
    dev = torch.device("cuda:0")
    n = mib << 20
    src = torch.ones(n // 4, dtype=torch.int32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(10):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration": {"bytes_read_per_copy": n,
                                           "bytes_written_per_copy": n, "copies": 10}}),
          flush=True)


def describe(name, c):
    if name == "prefill":
        return (f"prefill+decode: {c.n_req} requests of U{{1..{c.max_len}}} tokens, "
                f"one adapter each of N={c.N}; h_in={c.h_in}, h_out={c.h_out}, "
                f"r={c.rank}, bf16")
    rank = "U{" + ",".join(map(str, c.rank)) + "}" if isinstance(c.rank, tuple) else c.rank
    dist = f"Zipf({c.alpha})" if c.dist == "zipf" else c.dist
    return (f"{name}: T={c.T} tokens, h_in={c.h_in}, h_out={c.h_out}, r={rank}, "
            f"N={c.N} bf16 adapters, ids {dist}")


def graph_seconds(torch, calls, K, eager=False, wall=None):
    """K calls (calls(k) enqueues call k) captured as one HIP graph, replayed
    once untimed and once between two events recorded on the stream it is
    replayed on; seconds for the K calls.  eager: the K calls issued from
    Python instead (which floors at the host's launch rate).  wall, a list,
    receives the host's wall-clock seconds of the timed pass, from a
    synchronized device to a synchronized device."""
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    g = None
    if not eager:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for k in range(K):
                calls(k)
        g.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record()
    if eager:
        for k in range(K):
            calls(k)
    else:
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    if wall is not None:
        wall.append(time.perf_counter() - t0)
    return e0.elapsed_time(e1) / 1e3


class ReadProbe:
    """The same-footprint plain-read ceiling (csrc/read_ceiling.hip)."""

    def __init__(self, torch, dev, draws, N):
        import ctypes
        from paper_2608_05483_amd import build as B
        self.torch = torch
        pl = ctypes.CDLL(B.PROBE_LIB)
        pl.plora_probe_read.argtypes = [ctypes.c_void_p] * 6 + [ctypes.c_int32] * 3 + \
            [ctypes.c_void_p] * 2
        pl.plora_probe_sink_words.argtypes = [ctypes.c_int32]
        self.pl = pl
        self.uniq = [torch.from_numpy(np.unique(d[(d >= 0) & (d < N)]).astype(np.int32)).to(dev)
                     for d in draws]
        self.sink = torch.empty(pl.plora_probe_sink_words(max(1, max(u.numel()
                                                                     for u in self.uniq))),
                                dtype=torch.int32, device=dev)

    def read(self, ad, d, h_in, h_out):
        # the stream is looked up at call time, so that a call made under graph
        # capture is captured
        rc = self.pl.plora_probe_read(ad.A.data_ptr(), ad.B.data_ptr(), ad.a_off.data_ptr(),
                                      ad.b_off.data_ptr(), ad.ranks.data_ptr(),
                                      self.uniq[d].data_ptr(), self.uniq[d].numel(), h_in, h_out,
                                      self.sink.data_ptr(),
                                      self.torch.cuda.current_stream().cuda_stream)
        assert rc == 0


class ApplyBench:
    """One workload on the device: adapter-stack replicas, activation
    replicas, a pool of token draws and their segmentations."""

    def __init__(self, torch, P, W, dev, name, args, n_proj=1):
        self.torch, self.P, self.W, self.dev, self.name = torch, P, W, dev, name
        self.args = args
        c = W.CONFIGS[name]
        self.c = c
        seed = 1000 + W.CONFIG_NAMES.index(name)
        w = W.make_workload(name)
        self.w = w
        N = self.N = w.n_adapters
        self.n_proj = n_proj
        wps = [w] if n_proj == 1 else W.make_projections(name, n_proj=n_proj)
        if len(wps) != n_proj:
            print(f"bench.py: config {name} defines {len(wps)} projections", file=sys.stderr)
            sys.exit(2)
        self.wps = wps
        draws = [W.draw_idx(name, seed, d) for d in range(args.draws)]
        self.draws = draws
        Tmax = self.Tmax = max(d.size for d in draws)
        self.act_bytes = lambda T: T * (2 * w.h_in + sum(4 * wp.h_out for wp in wps)) + 4 * T
        self.ad_bytes = [sum(W.adapter_bytes(wp.ranks, d, wp.h_in, wp.h_out, N) for wp in wps)
                         for d in draws]
        self.tot_bytes = [a + self.act_bytes(d.size) for a, d in zip(self.ad_bytes, draws)]

        bases = [P.Adapters.from_workload(wp, device=dev) for wp in wps]
        self.bases = bases
        stack_bytes = sum(2 * (b.A.numel() + b.B.numel()) for b in bases)
        R = args.replicas
        if R <= 0:
            per_step = max(1, int(np.mean(self.ad_bytes)))
            R = max(2, min(64, math.ceil(3 * MALL_BYTES / per_step)))
            R = max(1, min(R, int((96 << 30) // max(stack_bytes, 1))))
        self.R = R
        self.reps = [bases]
        for _ in range(R - 1):
            self.reps.append([P.Adapters(b.A.clone(), b.B.clone(), b.a_off, b.b_off, b.ranks,
                                         b.scales, b.h_in, b.h_out, b.max_rank) for b in bases])
        # activation replicas: enough that x and y of earlier steps have left
        # the Infinity Cache too
        act_step = max(1, int(np.mean([self.act_bytes(d.size) for d in draws])))
        RA = max(1, min(64, math.ceil(3 * MALL_BYTES / act_step)))
        self.RA = RA
        xw = w if Tmax == w.T else W.with_idx(w, np.zeros(Tmax, np.int32))
        x0 = torch.from_numpy(xw.x).view(torch.int16).to(dev)
        self.xs = [x0] + [x0.clone() for _ in range(RA - 1)]
        self.ys = []                        # [projection][activation replica]
        for wp in wps:
            y_host = np.zeros((Tmax, wp.h_out), np.uint16)
            n = min(Tmax, wp.T)
            y_host[:n] = wp.y_base[:n]
            y0 = torch.from_numpy(y_host).view(torch.int16).to(dev)
            self.ys.append([y0] + [y0.clone() for _ in range(RA - 1)])
        self.ws = P.Workspace(Tmax, bases if n_proj > 1 else bases[0])
        self.idx_dev = [torch.from_numpy(d).to(dev) for d in draws]
        self.segs = [P.Segments(d.size, N, device=dev) for d in draws]
        self.apply_call = self._apply_call

    def _apply_call(self, k, separate=False):
        P = self.P
        d = k % len(self.draws)
        T = self.draws[d].size
        rp = self.reps[k % self.R]
        a = k % self.RA
        x = self.xs[a][:T]
        if self.n_proj == 1:
            P.apply(x, rp[0], self.segs[d], self.ys[0][a][:T], self.ws)
        elif separate:
            for q in range(self.n_proj):
                P.apply(x, rp[q], self.segs[d], self.ys[q][a][:T], self.ws)
        else:
            P.apply_multi(x, rp, self.segs[d], [yq[a][:T] for yq in self.ys], self.ws)

    def step(self, k, ev=None):
        P = self.P
        d = k % len(self.draws)
        if ev is not None:
            ev[0].record()
        if self.n_proj == 1:
            # segmentation and apply in one call (one launch for batches of up to
            # 256 tokens; plora_segment then plora_apply otherwise)
            T = self.draws[d].size
            a = k % self.RA
            P.segment_apply(self.idx_dev[d], self.xs[a][:T], self.reps[k % self.R][0],
                            self.segs[d], self.ys[0][a][:T], self.ws)
        else:
            P.segment(self.idx_dev[d], self.segs[d])
            self.apply_call(k)
        if ev is not None:
            ev[1].record()

    def one_launch(self):
        return self.n_proj == 1 and all(
            self.P.plora_segment_apply_launches(d.size, self.bases[0].struct) == 1
            for d in self.draws)

    def measure(self, K, warmup, eager=False, isolated=False, warm=False, ceiling=True):
        torch, P, args = self.torch, self.P, self.args
        for k in range(warmup):
            self.step(k)
        torch.cuda.synchronize()
        out = {}
        # eager steps with events around each (only where asked: the host
        # floors each such step at its launch rate)
        if isolated:
            evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                   for _ in range(K)]
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for k in range(K):
                self.step(warmup + k, evs[k])
            torch.cuda.synchronize()
            out["wall_eager"] = time.perf_counter() - t0
            ms = np.array([a.elapsed_time(b) for a, b in evs])
            out["isolated_us"] = {"mean": round(float(ms.mean()) * 1e3, 3),
                                  "p10": round(float(np.percentile(ms, 10)) * 1e3, 3),
                                  "p90": round(float(np.percentile(ms, 90)) * 1e3, 3)}
        # the K steps as one graph (or eager): wall clock and events
        wall = []
        step_s = graph_seconds(torch, lambda k: self.step(warmup + k), K, eager, wall)
        out["wall"] = wall[0]
        out["step_s"] = step_s
        ks = [(warmup + k) % len(self.draws) for k in range(K)]
        out["tokens"] = sum(self.draws[d].size for d in ks)
        out["bytes_total"] = sum(self.tot_bytes[d] for d in ks)
        out["bytes_adapter"] = sum(self.ad_bytes[d] for d in ks)
        # the apply's own duration: the same draws, stacks and activations,
        # segments made beforehand
        for d in range(len(self.draws)):
            P.segment(self.idx_dev[d], self.segs[d])
        torch.cuda.synchronize()
        out["apply_s"] = graph_seconds(torch, lambda k: self.apply_call(warmup + k), K, eager)
        if warm and self.n_proj == 1 and self.R > 1:
            # one stack replica and one activation replica: the adapters stay in
            # the Infinity Cache from call to call (reported, never priced)
            R, RA = self.R, self.RA
            self.R, self.RA = 1, 1
            out["warm_s"] = graph_seconds(torch, lambda k: self.apply_call(warmup + k), K, eager)
            self.R, self.RA = R, RA
        if self.n_proj > 1:
            out["separate_s"] = graph_seconds(
                torch, lambda k: self.apply_call(warmup + k, True), K, eager)
        if ceiling and self.n_proj == 1:
            probe = ReadProbe(torch, self.dev, self.draws, self.N)
            w = self.w
            rd = lambda k: probe.read(self.reps[(warmup + k) % self.R][0],
                                      (warmup + k) % len(self.draws), w.h_in, w.h_out)
            for k in range(warmup):
                rd(k)
            out["read_s"] = graph_seconds(torch, rd, K, eager)
        one = self.one_launch() and not eager
        out["one_launch"] = one
        out["priced_s"] = step_s if one else out["apply_s"]
        out["kernel"] = ("segment_apply_kernel (plora_segment_apply)" if one else
                         "plora_apply" if self.n_proj == 1 else "plora_apply_multi")
        stem = ("plora_segment_apply_" if one else "plora_apply_") + self.name
        out["traffic"] = measured_traffic(stem) if self.n_proj == 1 else None
        return out


def summary(b, m, K):
    """The per-workload record of the 'configs' object."""
    bt = m["bytes_total"] / K
    achieved = m["bytes_total"] / m["priced_s"] / 1e9
    rec = {
        "workload": describe(b.name, b.c),
        "tokens_per_step": round(m["tokens"] / K, 1),
        "tokens_per_s": round(m["tokens"] / m["wall"], 1),
        "step_us": round(m["step_s"] / K * 1e6, 3),
        "kernel": m["kernel"],
        "us_per_launch": round(m["priced_s"] / K * 1e6, 3),
        "bytes_per_launch": int(bt),
        "adapter_bytes_per_launch": int(m["bytes_adapter"] / K),
        "frac": round(achieved / HBM_PEAK_GBPS, 4),
        "traffic": m["traffic"],
        "traffic_over_algorithmic": (None if m["traffic"] is None
                                     else round(m["traffic"] / bt, 3)),
        "apply_us": round(m["apply_s"] / K * 1e6, 3),
        "adapter_GBps": round(m["bytes_adapter"] / m["apply_s"] / 1e9, 1),
        "stack_replicas": b.R, "activation_replicas": b.RA,
    }
    if "read_s" in m:
        rec["read_ceiling_us"] = round(m["read_s"] / K * 1e6, 3)
        rec["read_ceiling_frac"] = round(m["bytes_adapter"] / m["read_s"] / 1e9 /
                                         HBM_PEAK_GBPS, 4)
    return rec


def bench_attention(args):
    """plora_attn_decode on 64 requests x 32 heads x head dim 128 with caches
    of U{512..4096} keys (seeded), one HBM-resident bf16 KV cache per step
    replica; K steps captured as one graph and replayed between HIP events."""
    import torch
    from paper_2608_05483_amd import plora as P
    dev = torch.device("cuda:0")
    Bn, H, D, Lmax = 64, 32, P.ATTN_HEAD_DIM, 4096
    rng = np.random.default_rng(2024)
    lens_np = rng.integers(512, Lmax + 1, Bn).astype(np.int32)
    g = torch.Generator(device=dev).manual_seed(2024)
    bits = lambda t: t.to(torch.bfloat16).view(torch.int16)
    R = 2                                     # 2 x 4.3 GB of caches: far past the 256 MB MALL
    caches = [(bits(torch.randn((Bn, H, Lmax, D), device=dev, generator=g)),
               bits(torch.randn((Bn, H, Lmax, D), device=dev, generator=g))) for _ in range(R)]
    q = bits(torch.randn((Bn, H, D), device=dev, generator=g))
    lens = torch.from_numpy(lens_np).to(dev)
    out = torch.zeros((Bn, H, D), dtype=torch.int16, device=dev)
    ws = torch.empty(P.attn_workspace_bytes(Bn, H, Lmax), dtype=torch.uint8, device=dev)
    scale = 1.0 / math.sqrt(D)

    def step(k):
        K, V = caches[k % R]
        P.attn_decode(q, K, V, lens, scale, out, ws)

    for k in range(args.warmup):
        step(k)
    torch.cuda.synchronize()
    Ks = args.steps
    walls = []
    ev = graph_seconds(torch, step, Ks, wall=walls)
    wall = walls[0]
    kv_bytes = int(lens_np.sum()) * H * D * 2 * 2
    step_bytes = kv_bytes + 2 * Bn * H * D * 2
    achieved = step_bytes / (ev / Ks) / 1e9
    cpu = None
    if not args.no_cpu_baseline:
        sys.path.insert(0, ROOT)
        from oracle import attention as OA
        Kh = caches[0][0][:2].cpu().numpy().view(np.uint16)
        Vh = caches[0][1][:2].cpu().numpy().view(np.uint16)
        qh = q[:2].cpu().numpy().view(np.uint16)
        n_done, t_cpu = 0, 0.0
        while t_cpu < args.cpu_seconds:
            t1 = time.perf_counter()
            OA.attention(qh, Kh, Vh, lens_np[:2], scale)
            t_cpu += time.perf_counter() - t1
            n_done += 1
        cpu = {"value": round(n_done * 2 / t_cpu, 2), "unit": "requests/s (32 heads each)",
               "cores": 1, "kind": "oracle",
               "sample": f"{n_done} passes over requests 0 and 1 of this batch "
                         f"(caches of {int(lens_np[0])} and {int(lens_np[1])} keys), "
                         f"float64 numpy oracle, {t_cpu:.1f} s"}
    print(json.dumps({
        "metric": "decode attention KV-cache GB/s (% of HBM peak), split-KV with exact merge",
        "value": round(Bn * Ks / wall, 1), "unit": "requests/s (32 heads each)",
        "n_gpus": 1, "steps": Ks, "warmup": args.warmup,
        "ms_per_step": round(wall / Ks * 1e3, 5), "launch": "hip graph of the K steps",
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"decode attention: {Bn} requests x {H} heads x head dim {D}, "
                               f"caches U{{512..{Lmax}}} keys (seeded), bf16",
                   "batch": Bn, "heads": H, "head_dim": D, "max_len": Lmax,
                   "kv_keys": int(lens_np.sum()), "cache_replicas": R},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": None, "kernel": "attn_partial_kernel + attn_merge_kernel",
                     "us_per_launch": round(ev / Ks * 1e6, 3)},
        "bytes_per_step": step_bytes,
        "cpu_baseline": cpu}), flush=True)


def placement_split(torch, P, b, args, K):
    """The apply with adapters K.. read from the pinned host pool (E2) and
    the rest from HBM (E1), next to the cost model's prediction."""
    from paper_2608_05483_amd import placement as PL
    w, N, dev = b.w, b.N, b.dev
    Kp = args.pool_from
    A_pool = torch.from_numpy(w.A.view(np.int16)).pin_memory()
    B_pool = torch.from_numpy(w.B.view(np.int16)).pin_memory()
    in_pool = np.arange(N) >= Kp
    a_off = torch.from_numpy(np.where(in_pool, -1 - w.a_off, w.a_off).astype(np.int64)).to(dev)
    b_off = torch.from_numpy(np.where(in_pool, -1 - w.b_off, w.b_off).astype(np.int64)).to(dev)
    pool_reps = [P.Adapters(rp[0].A, rp[0].B, a_off, b_off, rp[0].ranks, rp[0].scales,
                            w.h_in, w.h_out, w.max_rank, A_pool=A_pool, B_pool=B_pool)
                 for rp in b.reps]

    def pool_call(k):
        d = k % len(b.draws)
        T = b.draws[d].size
        a = k % b.RA
        P.apply(b.xs[a][:T], pool_reps[k % b.R], b.segs[d], b.ys[0][a][:T], b.ws)

    pool_s = graph_seconds(torch, lambda k: pool_call(args.warmup + k), K, args.eager)
    apply_s = graph_seconds(torch, lambda k: b.apply_call(args.warmup + k), K, args.eager)
    hw = PL.Hardware()
    model_split, model_hbm, pool_bytes = [], [], []
    for d in b.draws:
        ok = (d >= 0) & (d < N)
        Bc = np.bincount(d[ok], minlength=N)
        st = np.where(in_pool, PL.E2, PL.E1).astype(object)
        model_split.append(PL.lora_time(Bc, w.ranks, st, w.h_in, w.h_out, hw))
        model_hbm.append(PL.lora_time(Bc, w.ranks, np.full(N, PL.E1, dtype=object),
                                      w.h_in, w.h_out, hw))
        pool_bytes.append(sum(PL.adapter_bytes(w.ranks[a], w.h_in, w.h_out)
                              for a in np.unique(d[ok]) if a >= Kp))
    return {
        "pool_from": Kp,
        "apply_us_split": round(pool_s / K * 1e6, 3),
        "apply_us_all_hbm": round(apply_s / K * 1e6, 3),
        "pool_bytes_per_call": int(np.mean(pool_bytes)),
        "model_us_split": round(float(np.mean(model_split)) * 1e6, 3),
        "model_us_all_hbm": round(float(np.mean(model_hbm)) * 1e6, 3),
        "model_hardware": {"C_gpu": hw.C_gpu, "W_gpu": hw.W_gpu, "W_link": hw.W_link,
                           "L_link": hw.L_link},
    }


def cpu_baseline(W, b, args):
    """The CPU oracle, as it stands, on a bounded sample of the workload."""
    sys.path.insert(0, ROOT)
    import oracle
    w, wps, draws = b.w, b.wps, b.draws
    cores = len(os.sched_getaffinity(0))

    def run(seconds, threads):
        n_done, toks, t_cpu = 0, 0, 0.0
        while t_cpu < seconds:
            d = draws[n_done % len(draws)]
            wd = w if d.size == w.T else W.with_idx(w, d)
            t1 = time.perf_counter()
            for wp in wps:
                oracle.apply(wd.x, d, wp.A, wp.a_off, wp.B, wp.b_off, wp.ranks, wp.scales,
                             np.zeros((d.size, wp.h_out), np.uint16), w.h_in, wp.h_out,
                             n_threads=threads)
            t_cpu += time.perf_counter() - t1
            toks += d.size
            n_done += 1
        return n_done, toks, t_cpu

    n_done, toks, t_cpu = run(args.cpu_seconds, cores)
    k1, toks1, t1_cpu = run(args.cpu_seconds / 10, 1)
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"value": round(toks / t_cpu, 1), "unit": "tokens/s", "cores": cores,
            "kind": "oracle", "value_1_thread": round(toks1 / t1_cpu, 1), "cpu_model": model,
            "sample": f"{n_done} batches of this workload, cycling its "
                      f"{len(draws)} token draws ({toks} tokens, {t_cpu:.1f} s), "
                      f"fp32 C oracle, OpenMP over tokens on {cores} threads; "
                      f"one thread: {k1} batches ({toks1} tokens, {t1_cpu:.1f} s)"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported: the "
              "apply runs on a single GPU (how it would shard is a design note only).",
              file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration > 0:
        copy_calibration(args.copy_calibration)
        return
    if args.workload == "attention":
        bench_attention(args)
        return

    import torch
    from paper_2608_05483_amd import plora as P
    from paper_2608_05483_amd import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    name = args.config
    K = args.steps
    n_proj = args.projections
    if args.also == "auto":
        extra = list(EXTRA_DEFAULT) if name == "decode" and n_proj == 1 else []
    elif args.also in ("", "none"):
        extra = []
    else:
        extra = [e for e in args.also.split(",") if e and e != name]

    b = ApplyBench(torch, P, W, dev, name, args, n_proj)
    print(f"bench: {name} ({b.R} stack replicas, {b.RA} activation replicas)",
          file=sys.stderr, flush=True)
    m = b.measure(K, args.warmup, eager=args.eager, isolated=True, warm=True,
                  ceiling=not args.no_ceiling)
    placement = placement_split(torch, P, b, args, K) \
        if args.pool_from >= 0 and n_proj == 1 else None
    cpu = None if args.no_cpu_baseline else cpu_baseline(W, b, args)
    rec = summary(b, m, K)
    w, N, R, Tmax = b.w, b.N, b.R, b.Tmax
    wps = b.wps
    achieved = m["bytes_total"] / m["priced_s"] / 1e9
    adapter_gbps = m["bytes_adapter"] / m["apply_s"] / 1e9
    del b
    torch.cuda.empty_cache()

    configs = {}
    for e in extra:
        print(f"bench: {e}", file=sys.stderr, flush=True)
        be = ApplyBench(torch, P, W, dev, e, args, 1)
        me = be.measure(K, args.warmup, eager=args.eager, ceiling=not args.no_ceiling)
        configs[e] = summary(be, me, K)
        del be
        torch.cuda.empty_cache()

    out = {
        "metric": "tokens/s and effective adapter GB/s (% of HBM peak) for plora_apply",
        "value": round(m["tokens"] / m["wall"], 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(m["wall"] / K * 1e3, 5),
        "launch": "eager" if args.eager else "hip graph of the K steps",
        "ms_per_step_eager": round(m["wall_eager"] / K * 1e3, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": describe(name, W.CONFIGS[name]) + (
                       "" if n_proj == 1 else
                       f"; {n_proj} projections sharing x, h_out "
                       f"{[wp.h_out for wp in wps]}, one plora_apply_multi call"),
                   "T": int(Tmax),
                   "h_in": w.h_in,
                   "h_out": w.h_out if n_proj == 1 else [wp.h_out for wp in wps],
                   "max_rank": w.max_rank, "n_adapters": N,
                   "draws": args.draws, "stack_replicas": R,
                   "activation_replicas": rec["activation_replicas"]},
        "adapter_GBps": round(adapter_gbps, 1),
        "adapter_frac_of_peak": round(adapter_gbps / HBM_PEAK_GBPS, 4),
        "apply_us": rec["apply_us"],
        "apply_us_warm": None if "warm_s" not in m else round(m["warm_s"] / K * 1e6, 3),
        "step_us_events": round(m["step_s"] / K * 1e6, 3),
        "step_us_isolated_events": m["isolated_us"],
        "bytes_per_launch": rec["bytes_per_launch"],
        "adapter_bytes_per_launch": rec["adapter_bytes_per_launch"],
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": m["traffic"],
                     "kernel": m["kernel"], "us_per_launch": rec["us_per_launch"]},
        "read_ceiling": (None if "read_s" not in m else {
            "kernel": "plain 128-bit read of the same adapter blocks, K launches in one graph",
            "GBps": round(m["bytes_adapter"] / m["read_s"] / 1e9, 1),
            "us_per_launch": rec["read_ceiling_us"],
            "frac_of_peak": rec["read_ceiling_frac"]}),
        "separate_calls_us": (None if "separate_s" not in m
                              else round(m["separate_s"] / K * 1e6, 3)),
        "placement": placement,
        "configs": configs,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
