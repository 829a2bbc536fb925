"""GPU parity across the paper's rank range (section V-A: ranks 2..128; the
evaluation of section VII-A draws from {8, 16, 32, 64, 128}): every rank
from 1 to 128 must give the oracle's y, through every form of the apply.

Ranks that are multiples of 8 run the vector and matrix-core paths of the
next power of two with their own row stride; the others take the LDS-staged
shrink.  The batches below mix segment lengths so that one call exercises
single-token tiles, the vector path's token widths 1, 2 and 4, matrix-path
tiles of one and two 16-token tiles, and segments split over several tiles.
Bars are those of test_gpu_parity (the benchmark spec's tolerance, the rigorous
fp32 bound against float64, agreement with the oracle's bf16, and the
relative L2 error of the delta on unit-scale inputs), plus: no exchange
give-ups and no skipped tokens in the workspace counters.
"""
from __future__ import annotations

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import refs  # noqa: E402
from paper_2608_05483_amd import workloads as W  # noqa: E402
from test_gpu_parity import (ORACLE_THREADS, Run, bits16, check_segments, check_y,  # noqa: E402
                             dev, gamma, oracle_y, say)

# every kernel shape: below 8, odd, multiples of 4 and 8 that are not powers
# of two, each power of two, and the ends of the range
RANKS = [1, 2, 3, 4, 7, 8, 12, 16, 20, 24, 32, 40, 48, 56, 64, 72, 96, 100, 120, 127, 128]
# segment lengths of the mixed batch (175 tokens)
LENGTHS = (1, 1, 1, 2, 2, 3, 4, 5, 7, 8, 12, 16, 17, 31, 32, 33)


@pytest.fixture(scope="module")
def P():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2608_05483_amd import plora
    return plora


def lengths_idx(rng, N, lengths):
    ids = rng.choice(N, len(lengths), replace=False)
    idx = np.repeat(ids, lengths).astype(np.int32)
    rng.shuffle(idx)
    return idx


def check_counters(run):
    give_ups, skipped = run.ws.counters()
    assert give_ups == 0, f"{give_ups} work items computed v alone"
    assert skipped == 0, f"{skipped} tokens skipped"


def check_v(w, v, idx):
    """v within 2 gamma_{h_in} sum_k |x_k A_kc| of the oracle's, per element."""
    vref = oracle.shrink(w.x, idx, w.A, w.a_off, w.ranks, w.h_in, ldv=v.shape[1],
                         n_threads=ORACLE_THREADS)
    valid = (idx >= 0) & (idx < w.n_adapters)
    toks = np.nonzero(valid)[0]
    if toks.size > 48:
        toks = np.sort(np.random.default_rng(0).choice(toks, 48, replace=False))
    for t in toks:
        i = int(idx[t])
        r = int(w.ranks[i])
        if r == 0:
            continue
        Ai = refs.dec(w.A[w.a_off[i]:w.a_off[i] + w.h_in * r]).reshape(w.h_in, r)
        S = np.abs(refs.dec(w.x[t])) @ np.abs(Ai)
        assert (np.abs(v[t, :r] - vref[t, :r]) <= 2 * gamma(w.h_in) * S).all(), t


@pytest.mark.parametrize("r", RANKS)
def test_rank_matches_oracle_in_every_form(P, r):
    rng = np.random.default_rng(100 + r)
    N = 64
    idx = lengths_idx(rng, N, LENGTHS)
    w = W.make_workload("decode", scale="parity", ranks=r, n_adapters=N, idx=idx)
    say(f"rank {r}: T={w.T} max_rank={max(8, (r + 7) // 8 * 8)}")
    yref, yout = oracle_y(w)
    # plora_apply on a segmentation from plora_segment
    run = Run(P, w).segment()
    check_segments(P, run, N)
    y = run.apply()
    check_y(y, yref, yout, w, strict_l2=True)
    # the split calls: v within its bound, and the same y bits as the apply
    v = run.shrink()
    check_v(w, v.cpu().numpy(), w.idx)
    assert (run.expand(v) == y).all()
    # plora_segment_apply (one launch where the batch allows it)
    run2 = Run(P, w)
    y2 = run2.segment_apply()
    check_segments(P, run2, N)
    assert (y2 == y).all()
    check_counters(run)
    check_counters(run2)
    # a decode batch of single tokens and short tiles (the exchange form)
    wd = W.with_idx(w, W.zipf_ids(rng, 64, N, 1.0))
    rd = Run(P, wd).segment()
    yd = rd.apply()
    ydr, ydo = oracle_y(wd)
    check_y(yd, ydr, ydo, wd, strict_l2=True)
    assert (rd.segment_apply() == yd).all()
    check_counters(rd)


@pytest.mark.parametrize("r", [3, 12, 48, 100, 128])
def test_rank_two_part_prefill_form(P, r):
    """Batches above 256 tokens take the two-part form (shrink work groups
    pass partial v per h_in slice through the workspace to the expand work
    groups, in one launch), here at the prefill shape (h_in = 8192,
    h_out = 1024) with requests of up to 300 tokens."""
    rng = np.random.default_rng(200 + r)
    N = 40
    lens = list(rng.integers(150, 300, size=8)) + [1, 2, 5, 33]
    idx = lengths_idx(rng, N, lens)
    w = W.make_workload("prefill", scale="parity", ranks=r, n_adapters=N, idx=idx)
    say(f"rank {r} two-part: T={w.T}")
    assert w.T > 1024
    run = Run(P, w).segment()
    y = run.apply()
    yref, yout = oracle_y(w)
    check_y(y, yref, yout, w, strict_l2=True)
    v = run.shrink()
    check_v(w, v.cpu().numpy(), w.idx)
    assert (run.expand(v) == y).all()
    check_counters(run)


def test_mixed_ranks_1_to_128_in_one_stack(P):
    """One stack whose adapters carry every rank from 0 to 128 side by side
    (ragged offsets), through a decode batch, a 256-token batch, a batch of
    mixed segment lengths and a two-part batch."""
    rng = np.random.default_rng(77)
    N = 300
    ranks = rng.integers(1, 129, size=N).astype(np.int32)
    ranks[rng.choice(N, 10, replace=False)] = 0
    ranks[:128] = np.arange(1, 129)
    base = W.make_workload("decode", scale="parity", ranks=ranks, n_adapters=N,
                           idx=np.zeros(1, np.int32))
    batches = [("zipf64", W.zipf_ids(rng, 64, N, 1.0)),
               ("uniform256", W.uniform_ids(rng, 256, N)),
               ("lengths", lengths_idx(rng, N, LENGTHS)),
               ("two_part", lengths_idx(rng, N, list(rng.integers(1, 200, size=12)) +
                                          [1] * 40))]
    for name, idx in batches:
        w = W.with_idx(base, idx)
        say(f"mixed ranks {name}: T={w.T}")
        run = Run(P, w).segment()
        y = run.apply()
        yref, yout = oracle_y(w)
        check_y(y, yref, yout, w, strict_l2=True)
        if w.T <= 256:
            run2 = Run(P, w)
            assert (run2.segment_apply() == y).all()
            check_counters(run2)
        assert (run.expand(run.shrink()) == y).all()
        check_counters(run)


@pytest.mark.parametrize("scale", ["paper", "parity"])
def test_rank128_thousand_adapters_large_shape(P, scale):
    """1000 rank-128 adapters at the large decode-batch shape (T = 256
    uniform ids, h = 4096, y_base ~ N(0, 1) at the paper scale), and a
    64-token Zipf batch on the same stack, which takes the exchange form with
    one work group per compute unit (82 KB of LDS each): every item of the
    launch is resident, so no partner is waited for and none gives up."""
    rng = np.random.default_rng(128)
    idx = W.uniform_ids(rng, 256, 1000)
    w = W.make_workload("large", scale=scale, ranks=128, idx=idx, only_used=True)
    say(f"rank 128 x 1000 adapters, T=256, {scale}")
    run = Run(P, w).segment()
    y = run.apply()
    yref, yout = oracle_y(w)
    check_y(y, yref, yout, w, strict_l2=(scale == "parity"))
    run2 = Run(P, w)
    assert (run2.segment_apply() == y).all()
    check_counters(run)
    check_counters(run2)
    wd = W.make_workload("large", scale=scale, ranks=128, idx=W.zipf_ids(rng, 64, 1000, 1.0),
                         only_used=True)
    say(f"rank 128 x 1000 adapters, T=64, {scale}")
    rd = Run(P, wd).segment()
    assert P.plora_segment_apply_launches(64, rd.ad.struct) == 1
    yd = rd.segment_apply()
    ydr, ydo = oracle_y(wd)
    check_y(yd, ydr, ydo, wd, strict_l2=(scale == "parity"))
    assert (rd.apply() == yd).all()
    check_counters(rd)


@pytest.mark.parametrize("reps", [1, 3])
def test_unusable_entries_are_counted(P, reps):
    """A rank above max_rank (or below 0) cannot be applied: those tokens keep
    y_base, the workspace counts them once per call, the rest of the batch is
    the oracle's, and plora_check_adapters names the first such entry.  With
    the lengths three times over (525 tokens) the apply takes its two-part
    form, whose expand work groups do the counting."""
    w = W.make_workload("decode", scale="parity", ranks=16, n_adapters=64,
                        idx=lengths_idx(np.random.default_rng(5), 64, LENGTHS * reps))
    bad = int(w.idx[0])
    ranks = w.ranks.copy()
    ranks[bad] = 24                            # above max_rank = 16
    ad = P.Adapters.from_arrays(w.A, w.B, w.a_off, w.b_off, ranks, w.scales, w.h_in,
                                w.h_out, max_rank=16)
    assert P.plora_check_adapters(ad.struct, P._stream()) == bad
    run = Run(P, w).segment()
    run.ad = ad
    y = run.apply()
    rows = w.idx == bad
    assert (y[rows] == w.y_base[rows]).all()
    yref, yout = oracle_y(w)
    assert (y[~rows] == run.expand(run.shrink())[~rows]).all()
    keep = ~rows
    wk = W.Workload(**{**w.__dict__, "idx": w.idx[keep], "T": int(keep.sum()),
                       "x": w.x[keep], "y_base": w.y_base[keep]})
    check_y(y[keep], yref[keep], yout[keep], wk, strict_l2=True)
    give_ups, skipped = run.ws.counters()
    assert give_ups == 0
    # apply, then shrink (which counts too): two calls
    assert skipped == 2 * int(rows.sum())


def test_overlong_one_launch_tile_is_skipped_and_counted(P):
    """A one-launch call (T <= 256) holds each tile's partial v in an
    exchange region sized for PLORA_SMALL_BATCH_TILE_TOKENS tokens; a tile
    longer than that (which plora_segment never writes for such a batch) is
    skipped, its tokens keep y_base and are counted, and every other tile
    gives the bits of the unmodified segmentation."""
    w = W.make_workload("decode", scale="parity", ranks=16, n_adapters=64,
                        idx=np.full(40, 7, np.int32))
    run = Run(P, w).segment()
    y_ref = run.apply()
    tiles = run.segs.tiles.view(-1, 4).cpu().numpy().copy()
    n = int(run.segs.meta[4].item())
    tl = P.tile_tokens(w.T)
    assert n == 40 // tl and (tiles[:n, 2] == tl).all()
    L = 2 * P.PLORA_SMALL_BATCH_TILE_TOKENS + 1     # longer than any one-launch tile
    keep = tiles[:n][tiles[:n, 1] >= L + 1]         # the tiles after positions 0..L
    new = [(7, 0, L, 0), (7, L, 1, 0)] + [tuple(t) for t in keep]
    tiles[:] = (-1, 0, 0, -1)
    tiles[:len(new)] = new
    run.segs.tiles.copy_(torch.from_numpy(tiles.reshape(-1)))
    run.segs.meta[4] = len(new)
    run.ws = P.Workspace(w.T, run.ad)
    y = run.apply()
    perm = run.segs.perm.cpu().numpy()
    skipped = perm[:L]
    rest = np.setdiff1d(np.arange(w.T), skipped)
    assert (y[skipped] == w.y_base[skipped]).all()
    assert (y[rest] == y_ref[rest]).all()
    give_ups, n_skipped = run.ws.counters()
    assert give_ups == 0 and n_skipped == L
