#!/usr/bin/env python3
"""Benchmark: the batched heterogeneous-adapter LoRA apply on one MI355X.

One step = one pass of the whole hot path over one batch already resident in
HBM: plora_segment_apply, which groups the batch's tokens by adapter (the
plora_segment outputs) and applies y += s_i (x A_i) B_i for every token.  For
decode-sized batches that is one launch; larger batches take plora_segment
then plora_apply.  With --projections > 1 a step is plora_segment then one
plora_apply_multi.  Each step takes a fresh token-to-adapter draw from a pool
drawn up front, and a different replica of the adapter stack, so that an
adapter's bytes are never still sitting in the 256 MB Infinity Cache from an
earlier step (a served model revisits one projection's stack only after every
other LoRA projection of every layer).

Prints ONE JSON line.  ``value`` is whole-job tokens/s over the timed steps
(wall clock), the K steps launched as one captured HIP graph (``--eager``:
one launch per call from Python; the eager time is reported too).
``roofline`` prices the dominant kernel: algorithmic bytes per step
(distinct adapters' A_i and B_i, 2 r_i (h_in + h_out) bytes each, plus x
read, y read and written, and the token ids) over that kernel's average
duration.  Where a step is one launch, that is the step graph's duration
between two HIP events recorded on the stream the kernels run on; otherwise
it is the apply's: K plora_apply calls captured as one graph and replayed
between two such events.  ``cpu_baseline`` times the CPU oracle on a bounded
sample of the same workload.
"""
from __future__ import annotations

import argparse
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
KERNEL_SOURCE = os.path.join(ROOT, "paper_2608_05483_amd", "csrc", "plora.hip")
PROFILES = os.path.join(ROOT, "profiles")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="decode",
                    choices=["tiny", "decode", "large", "ragged", "prefill"])
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


def source_digest() -> str:
    with open(KERNEL_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic(stem: str):
    """HBM bytes per launch of the priced kernel from the committed counter
    summary (profiles/<stem>_traffic.txt, stem = kernel and workload), or
    None when there is none or the kernel source has changed since the
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
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for k in range(Ks):
            step(k)
    graph.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    graph.replay()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ev = e0.elapsed_time(e1) / 1e3
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
    c = W.CONFIGS[name]
    seed = 1000 + W.CONFIG_NAMES.index(name)
    w = W.make_workload(name)
    N = w.n_adapters
    n_proj = args.projections
    # the projections of one layer that share x (projection 0 is the config's
    # own workload); one projection is the plain plora_apply
    wps = [w] if n_proj == 1 else W.make_projections(name, n_proj=n_proj)
    if len(wps) != n_proj:
        print(f"bench.py: config {name} defines {len(wps)} projections", file=sys.stderr)
        sys.exit(2)

    # ---- token-to-adapter draws -------------------------------------------------
    draws = [W.draw_idx(name, seed, d) for d in range(args.draws)]
    Tmax = max(d.size for d in draws)
    act_bytes = lambda T: T * (2 * w.h_in + sum(4 * wp.h_out for wp in wps)) + 4 * T
    ad_bytes = [sum(W.adapter_bytes(wp.ranks, d, wp.h_in, wp.h_out, N) for wp in wps)
                for d in draws]
    tot_bytes = [a + act_bytes(d.size) for a, d in zip(ad_bytes, draws)]

    # ---- device buffers -----------------------------------------------------------
    bases = [P.Adapters.from_workload(wp, device=dev) for wp in wps]
    stack_bytes = sum(2 * (b.A.numel() + b.B.numel()) for b in bases)
    R = args.replicas
    if R <= 0:
        per_step = max(1, int(np.mean(ad_bytes)))
        R = max(2, min(64, math.ceil(3 * MALL_BYTES / per_step)))
        R = max(1, min(R, int((96 << 30) // max(stack_bytes, 1))))
    reps = [bases]
    for _ in range(R - 1):
        reps.append([P.Adapters(b.A.clone(), b.B.clone(), b.a_off, b.b_off, b.ranks, b.scales,
                                b.h_in, b.h_out, b.max_rank) for b in bases])
    xw = w if Tmax == w.T else W.with_idx(w, np.zeros(Tmax, np.int32))
    x = torch.from_numpy(xw.x).view(torch.int16).to(dev)
    ys = []
    for wp in wps:
        y_host = np.zeros((Tmax, wp.h_out), np.uint16)
        n = min(Tmax, wp.T)
        y_host[:n] = wp.y_base[:n]
        ys.append(torch.from_numpy(y_host).view(torch.int16).to(dev))
    ws = P.Workspace(Tmax, bases if n_proj > 1 else bases[0])
    idx_dev = [torch.from_numpy(d).to(dev) for d in draws]
    segs = [P.Segments(d.size, N, device=dev) for d in draws]

    def apply_call(k, separate=False):
        d = k % len(draws)
        T = draws[d].size
        rp = reps[k % R]
        if n_proj == 1:
            P.apply(x[:T], rp[0], segs[d], ys[0][:T], ws)
        elif separate:
            for q in range(n_proj):
                P.apply(x[:T], rp[q], segs[d], ys[q][:T], ws)
        else:
            P.apply_multi(x[:T], rp, segs[d], [yq[:T] for yq in ys], ws)

    def step(k, ev=None):
        d = k % len(draws)
        if ev is not None:
            ev[0].record()
        if n_proj == 1:
            # segmentation and apply in one call (one launch for decode-sized
            # batches; plora_segment then plora_apply otherwise)
            T = draws[d].size
            P.segment_apply(idx_dev[d], x[:T], reps[k % R][0], segs[d], ys[0][:T], ws)
        else:
            P.segment(idx_dev[d], segs[d])
            apply_call(k)
        if ev is not None:
            ev[1].record()

    for k in range(args.warmup):
        step(k)
    torch.cuda.synchronize()

    K = args.steps
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(K)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(K):
        step(args.warmup + k, evs[k])
    torch.cuda.synchronize()
    wall_eager = time.perf_counter() - t0
    wall = wall_eager
    step_event_s = None

    # ---- the same K steps launched as one HIP graph ------------------------------
    # At decode size a step's two kernels take less GPU time than Python needs
    # to issue them, so the eager loop measures the host.  The K steps (same
    # draws, same stack replicas) are captured once and the graph is replayed:
    # once untimed, then once timed.
    if not args.eager:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for k in range(K):
                step(args.warmup + k)
        graph.replay()
        torch.cuda.synchronize()
        s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        s0.record()
        graph.replay()
        s1.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        step_event_s = s0.elapsed_time(s1) / 1e3

    apply_ms = np.array([a.elapsed_time(b) for a, b in evs])
    ks = [(args.warmup + k) % len(draws) for k in range(K)]
    tokens = sum(draws[d].size for d in ks)

    # ---- the apply's own duration: K launches back to back -------------------
    # (segments already built; the same draws and stack replicas as the steps).
    # Events around single launches add several microseconds of their own at
    # this size, so the launch stream is bracketed once around all K.
    for k in range(K):
        P.segment(idx_dev[k % len(draws)], segs[k % len(draws)])
    torch.cuda.synchronize()
    b0, b1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(separate=False):
        # K calls captured as one graph (unless --eager), replayed once untimed
        # and once between two events on the stream the kernels run on: at
        # this size a Python loop of launches would time the host
        if args.eager:
            b0.record()
            for k in range(K):
                apply_call(k, separate)
            b1.record()
        else:
            ga = torch.cuda.CUDAGraph()
            with torch.cuda.graph(ga):
                for k in range(K):
                    apply_call(k, separate)
            ga.replay()
            torch.cuda.synchronize()
            b0.record()
            ga.replay()
            b1.record()
        torch.cuda.synchronize()
        return b0.elapsed_time(b1) / 1e3

    apply_s = timed()
    # warm: the same K calls on one stack replica, whose adapters stay in the
    # 256 MB Infinity Cache from call to call (reported, never priced)
    warm_s = None
    if n_proj == 1 and R > 1:
        saved_R, saved_reps = R, reps
        R, reps = 1, reps[:1]
        warm_s = timed()
        R, reps = saved_R, saved_reps
    separate_s = None
    if n_proj > 1:                           # the same work as one call per projection
        separate_s = timed(separate=True)
    bytes_total = sum(tot_bytes[k % len(draws)] for k in range(K))
    bytes_adapter = sum(ad_bytes[k % len(draws)] for k in range(K))
    # the kernel the roofline prices: where a step is a single launch
    # (plora_segment_apply's one-launch form) that launch, timed over the
    # step graph; otherwise the apply's own launches
    one_launch = (n_proj == 1 and step_event_s is not None and
                  all(P.plora_segment_apply_launches(d.size, bases[0].struct) == 1
                      for d in draws))
    priced_s = step_event_s if one_launch else apply_s
    kernel = ("segment_apply_kernel (plora_segment_apply)" if one_launch else
              "plora_apply" if n_proj == 1 else "plora_apply_multi")
    achieved = bytes_total / priced_s / 1e9
    traffic = (measured_traffic(("plora_segment_apply_" if one_launch else "plora_apply_") + name)
               if n_proj == 1 else None)
    adapter_gbps = bytes_adapter / apply_s / 1e9

    # ---- placement split: adapters K.. from the pinned host pool ----------------
    placement = None
    if args.pool_from >= 0 and n_proj == 1:
        from paper_2608_05483_amd import placement as PL
        Kp = args.pool_from
        A_pool = torch.from_numpy(w.A.view(np.int16)).pin_memory()
        B_pool = torch.from_numpy(w.B.view(np.int16)).pin_memory()
        in_pool = np.arange(N) >= Kp
        a_off = torch.from_numpy(np.where(in_pool, -1 - w.a_off, w.a_off).astype(np.int64)).to(dev)
        b_off = torch.from_numpy(np.where(in_pool, -1 - w.b_off, w.b_off).astype(np.int64)).to(dev)
        pool_reps = [P.Adapters(rp[0].A, rp[0].B, a_off, b_off, rp[0].ranks, rp[0].scales,
                                w.h_in, w.h_out, w.max_rank, A_pool=A_pool, B_pool=B_pool)
                     for rp in reps]

        def pool_call(k, separate=False):
            d = k % len(draws)
            T = draws[d].size
            P.apply(x[:T], pool_reps[k % R], segs[d], ys[0][:T], ws)

        saved = apply_call
        apply_call = pool_call
        pool_s = timed()
        apply_call = saved
        hw = PL.Hardware()
        model_split, model_hbm, pool_bytes = [], [], []
        for d in draws:
            ok = (d >= 0) & (d < N)
            Bc = np.bincount(d[ok], minlength=N)
            st = np.where(in_pool, PL.E2, PL.E1).astype(object)
            model_split.append(PL.lora_time(Bc, w.ranks, st, w.h_in, w.h_out, hw))
            model_hbm.append(PL.lora_time(Bc, w.ranks, np.full(N, PL.E1, dtype=object),
                                          w.h_in, w.h_out, hw))
            pool_bytes.append(sum(PL.adapter_bytes(w.ranks[a], w.h_in, w.h_out)
                                  for a in np.unique(d[ok]) if a >= Kp))
        placement = {
            "pool_from": Kp,
            "apply_us_split": round(pool_s / K * 1e6, 3),
            "apply_us_all_hbm": round(apply_s / K * 1e6, 3),
            "pool_bytes_per_call": int(np.mean(pool_bytes)),
            "model_us_split": round(float(np.mean(model_split)) * 1e6, 3),
            "model_us_all_hbm": round(float(np.mean(model_hbm)) * 1e6, 3),
            "model_hardware": {"C_gpu": hw.C_gpu, "W_gpu": hw.W_gpu, "W_link": hw.W_link,
                               "L_link": hw.L_link},
        }

    # ---- same-footprint plain-read ceiling -------------------------------------
    ceiling = None
    if not args.no_ceiling and n_proj == 1:
        import ctypes
        from paper_2608_05483_amd import build as B
        pl = ctypes.CDLL(B.PROBE_LIB)
        pl.plora_probe_read.argtypes = [ctypes.c_void_p] * 6 + [ctypes.c_int32] * 3 + \
            [ctypes.c_void_p] * 2
        pl.plora_probe_sink_words.argtypes = [ctypes.c_int32]
        uniq = [torch.from_numpy(np.unique(d[(d >= 0) & (d < N)]).astype(np.int32)).to(dev)
                for d in draws]
        sink = torch.empty(pl.plora_probe_sink_words(max(u.numel() for u in uniq)),
                           dtype=torch.int32, device=dev)
        stream = torch.cuda.current_stream().cuda_stream

        def probe(k):
            d = k % len(draws)
            rp = reps[k % R][0]
            rc = pl.plora_probe_read(rp.A.data_ptr(), rp.B.data_ptr(), rp.a_off.data_ptr(),
                                     rp.b_off.data_ptr(), rp.ranks.data_ptr(),
                                     uniq[d].data_ptr(), uniq[d].numel(), w.h_in, w.h_out,
                                     sink.data_ptr(), stream)
            assert rc == 0

        for k in range(args.warmup):
            probe(k)
        torch.cuda.synchronize()
        p0, p1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        p0.record()
        for k in range(K):                   # back to back, as the apply is timed
            probe(k)
        p1.record()
        torch.cuda.synchronize()
        read_s = p0.elapsed_time(p1) / 1e3
        bytes_adapter = sum(ad_bytes[k % len(draws)] for k in range(K))
        ceiling = {"kernel": "plain 128-bit read of the same adapter blocks",
                   "GBps": round(bytes_adapter / read_s / 1e9, 1),
                   "us_per_launch": round(read_s / K * 1e6, 3),
                   "frac_of_peak": round(bytes_adapter / read_s / 1e9 / HBM_PEAK_GBPS, 4)}

    # ---- CPU oracle baseline ----------------------------------------------------
    cpu = None
    if not args.no_cpu_baseline:
        sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
        import oracle
        cores = len(os.sched_getaffinity(0))
        n_done, toks, t_cpu = 0, 0, 0.0
        # cycle through the draws until the time budget is spent
        while t_cpu < args.cpu_seconds:
            d = draws[n_done % len(draws)]
            wd = w if d.size == w.T else W.with_idx(w, d)
            t1 = time.perf_counter()
            for wp in wps:
                oracle.apply(wd.x, d, wp.A, wp.a_off, wp.B, wp.b_off, wp.ranks, wp.scales,
                             np.zeros((d.size, wp.h_out), np.uint16), w.h_in, wp.h_out,
                             n_threads=cores)
            t_cpu += time.perf_counter() - t1
            toks += d.size
            n_done += 1
        # the same oracle on one thread, over a tenth of the time
        t1_cpu, toks1, k1 = 0.0, 0, 0
        while t1_cpu < args.cpu_seconds / 10:
            d = draws[k1 % len(draws)]
            wd = w if d.size == w.T else W.with_idx(w, d)
            t1 = time.perf_counter()
            for wp in wps:
                oracle.apply(wd.x, d, wp.A, wp.a_off, wp.B, wp.b_off, wp.ranks, wp.scales,
                             np.zeros((d.size, wp.h_out), np.uint16), w.h_in, wp.h_out,
                             n_threads=1)
            t1_cpu += time.perf_counter() - t1
            toks1 += d.size
            k1 += 1
        model = "unknown"
        try:
            for line in open("/proc/cpuinfo"):
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
        except OSError:
            pass
        cpu = {"value": round(toks / t_cpu, 1), "unit": "tokens/s", "cores": cores,
               "kind": "oracle",
               "value_1_thread": round(toks1 / t1_cpu, 1),
               "cpu_model": model,
               "sample": f"{n_done} batches of this workload, cycling its "
                         f"{len(draws)} token draws ({toks} tokens, {t_cpu:.1f} s), "
                         f"fp32 C oracle, OpenMP over tokens on {cores} threads; "
                         f"one thread: {k1} batches ({toks1} tokens, {t1_cpu:.1f} s)"}

    out = {
        "metric": "tokens/s and effective adapter GB/s (% of HBM peak) for plora_apply",
        "value": round(tokens / wall, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(wall / K * 1e3, 5),
        "launch": "eager" if args.eager else "hip graph of the K steps",
        "ms_per_step_eager": round(wall_eager / K * 1e3, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": describe(name, c) + (
                       "" if n_proj == 1 else
                       f"; {n_proj} projections sharing x, h_out "
                       f"{[wp.h_out for wp in wps]}, one plora_apply_multi call"),
                   "T": int(Tmax), "h_in": w.h_in,
                   "h_out": w.h_out if n_proj == 1 else [wp.h_out for wp in wps],
                   "max_rank": w.max_rank, "n_adapters": N,
                   "draws": len(draws), "stack_replicas": R},
        "adapter_GBps": round(adapter_gbps, 1),
        "adapter_frac_of_peak": round(adapter_gbps / HBM_PEAK_GBPS, 4),
        "apply_us": round(apply_s / K * 1e6, 3),
        "apply_us_warm": None if warm_s is None else round(warm_s / K * 1e6, 3),
        "step_us_events": (None if step_event_s is None
                           else round(step_event_s / K * 1e6, 3)),
        "step_us_isolated_events": {
            "mean": round(float(apply_ms.mean()) * 1e3, 3),
            "p10": round(float(np.percentile(apply_ms, 10)) * 1e3, 3),
            "p90": round(float(np.percentile(apply_ms, 90)) * 1e3, 3)},
        "bytes_per_launch": int(bytes_total / K),
        "adapter_bytes_per_launch": int(bytes_adapter / K),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": traffic,
                     "kernel": kernel, "us_per_launch": round(priced_s / K * 1e6, 3)},
        "read_ceiling": ceiling,
        "separate_calls_us": (None if separate_s is None
                              else round(separate_s / K * 1e6, 3)),
        "placement": placement,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
