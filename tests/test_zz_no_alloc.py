"""plora_segment_apply_noalloc, the entry point for callers that cannot
allocate: through the C ABI, two calls in a row (the second on a smaller
batch) against plora_segment_apply with a workspace of its own, bit for bit,
and against the oracle's bars; the segmentation it writes is the oracle's."""
from __future__ import annotations

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from paper_2608_05483_amd import workloads as W  # noqa: E402
from test_gpu_parity import Run, bits16, check_segments, check_y, dev, oracle_y, say  # noqa: E402


@pytest.fixture(scope="module")
def P():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2608_05483_amd import plora
    return plora


def _noalloc(P, run):
    y = dev(run.y0.view(np.int16))
    P.plora_segment_apply_noalloc(run.idx_d.data_ptr(), run.x.data_ptr(), run.x.stride(0),
                                  run.ad.struct, run.segs.struct, y.data_ptr(), y.stride(0),
                                  P._stream())
    torch.cuda.synchronize()
    return bits16(y)[:, :run.w.h_out]


@pytest.mark.parametrize("cfg,scale", [("decode", "parity"), ("decode", "paper"),
                                       ("large", "parity"), ("ragged", "parity")])
def test_noalloc_equals_segment_apply(P, cfg, scale):
    w0 = W.make_workload(cfg, scale=scale)
    rng = np.random.default_rng(17)
    # two calls in a row, the second with a smaller batch; for the ragged and
    # large stacks the batches are cut to the 256 tokens the call takes
    sizes = {"decode": (64, 24), "large": (256, 100), "ragged": (256, 40)}[cfg]
    for k, T in enumerate(sizes):
        idx = w0.idx[:T] if k == 0 else W.zipf_ids(rng, T, w0.n_adapters, 1.0)
        w = W.with_idx(w0, np.ascontiguousarray(idx))
        say(f"noalloc {cfg}/{scale} call {k}: T={T}")
        ours = Run(P, w)
        ours.segs.perm.fill_(-9)
        y_na = _noalloc(P, ours)
        check_segments(P, ours, w.n_adapters)
        ref = Run(P, w)
        y_ws = ref.segment_apply()
        assert (y_na == y_ws).all()
        yref, yout = oracle_y(w)
        check_y(y_na, yref, yout, w, strict_l2=(scale == "parity"))


def test_noalloc_refuses_more_than_256_tokens(P):
    w = W.make_workload("decode", scale="paper", idx=np.zeros(257, np.int32))
    run = Run(P, w)
    with pytest.raises(P.PloraError) as e:
        _noalloc(P, run)
    assert e.value.status == P.PLORA_ERR_UNSUPPORTED
