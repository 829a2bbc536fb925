"""The seeded input generator: determinism, shapes, layout and skew."""
import numpy as np
import pytest

from paper_2608_05483_amd import workloads as W


@pytest.mark.parametrize("name", ["tiny", "decode", "ragged", "prefill"])
def test_deterministic_and_shaped(name):
    a = W.make_workload(name, only_used=True)
    b = W.make_workload(name, only_used=True)
    for f in ("idx", "x", "y_base", "ranks", "a_off", "b_off", "A", "B", "scales"):
        assert np.array_equal(getattr(a, f), getattr(b, f)), f
    assert a.x.shape == (a.T, a.h_in) and a.y_base.shape == (a.T, a.h_out)
    assert a.x.dtype == np.uint16 and a.idx.dtype == np.int32
    # A_i / B_i blocks are contiguous, 16-byte aligned and non-overlapping
    assert (a.a_off % 8 == 0).all() and (a.b_off % 8 == 0).all()
    ends = a.a_off + a.ranks.astype(np.int64) * a.h_in
    assert (ends[:-1] <= a.a_off[1:]).all() and ends[-1] <= a.A.size


def test_only_used_matches_full_draw():
    full = W.make_workload("tiny")
    part = W.make_workload("tiny", only_used=True)
    for i in np.unique(full.idx):
        r = full.ranks[i]
        sl = slice(full.a_off[i], full.a_off[i] + full.h_in * r)
        assert np.array_equal(full.A[sl], part.A[sl])


def test_zipf_mass_and_uniform_range():
    rng = np.random.default_rng(0)
    ids = W.zipf_ids(rng, 200_000, 1000, 1.0)
    top50 = np.mean(ids < 50)
    w = np.arange(1, 1001, dtype=np.float64) ** -1.0
    assert abs(top50 - w[:50].sum() / w.sum()) < 0.01
    assert ids.min() >= 0 and ids.max() < 1000
    u = W.uniform_ids(rng, 10_000, 7)
    assert set(np.unique(u)) == set(range(7))


def test_prefill_requests_are_contiguous_runs():
    idx = W.draw_idx("prefill", 1004)
    changes = np.count_nonzero(np.diff(idx)) + 1
    assert changes <= 32 and 32 <= idx.size <= 32 * 512


def test_ragged_ranks_and_scales():
    w = W.make_workload("ragged", only_used=True)
    assert set(np.unique(w.ranks)) <= {8, 16, 32, 64}
    l = W.make_workload("large", only_used=True)
    assert set(np.unique(l.scales)) <= {0.5, 1.0, 2.0}


def test_bf16_rounding_of_draws():
    vals = np.array([1.0, 1.00390625, 1.005859375, -2.5], np.float32)
    bits = W.to_bf16_bits(vals)
    assert bits.tolist() == [0x3F80, 0x3F80, 0x3F81, 0xC020]
