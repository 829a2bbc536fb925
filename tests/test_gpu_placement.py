"""The placement decision driving the kernels (strategies E1 / E2): over a
sequence of decode batches, an HBM budget of a fraction of the adapter bytes,
adapters cached by the selection and the rest read from a pinned host pool.
Every step's y must meet the oracle's bars, and be the all-HBM result bit for
bit (the same kernels read the same values, wherever they live)."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from paper_2608_05483_amd import placement as PL  # noqa: E402
from paper_2608_05483_amd import workloads as W  # noqa: E402
from test_gpu_parity import check_y, oracle_y  # noqa: E402


@pytest.fixture(scope="module")
def P():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2608_05483_amd import plora
    return plora


def bits16(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


@pytest.mark.parametrize("budget_frac", [0.0, 0.02, 0.2])
def test_placed_adapters_give_the_all_hbm_result(P, budget_frac):
    w = W.make_workload("decode", scale="parity")
    seed = 1000 + W.CONFIG_NAMES.index("decode")
    print(f"placement decode budget {budget_frac}", flush=True)
    full = P.Adapters.from_workload(w)
    A_pool = torch.from_numpy(w.A.view(np.int16)).pin_memory()
    B_pool = torch.from_numpy(w.B.view(np.int16)).pin_memory()
    total = int(sum(PL.adapter_bytes(r, w.h_in, w.h_out) for r in w.ranks))
    budget = int(budget_frac * total)
    cache = PL.HbmCache(A_pool, B_pool, w.a_off, w.b_off, w.ranks, w.h_in, w.h_out, budget)
    temp = PL.Temperature(w.n_adapters)
    res = np.zeros(w.n_adapters, bool)
    hw = PL.Hardware()
    x = torch.from_numpy(w.x.view(np.int16)).cuda()
    y0 = torch.from_numpy(w.y_base.view(np.int16)).cuda()
    ws = P.Workspace(w.T, full)
    n_e1 = 0
    for step in range(8):
        idx = W.draw_idx("decode", seed, step)
        temp.request(idx[(idx >= 0) & (idx < w.n_adapters)])
        Bc = np.bincount(idx[(idx >= 0) & (idx < w.n_adapters)], minlength=w.n_adapters)
        d = PL.choose(Bc, w.ranks, w.h_in, w.h_out, hw, budget, res, temp)
        cache.apply(d)
        a_off, b_off = cache.offsets()
        ad = P.Adapters(cache.A, cache.B, torch.from_numpy(a_off).cuda(),
                        torch.from_numpy(b_off).cuda(), full.ranks, full.scales, w.h_in,
                        w.h_out, full.max_rank, A_pool=A_pool, B_pool=B_pool)
        assert P.plora_check_adapters(ad.struct, P._stream()) == -1
        idx_d = torch.from_numpy(idx).cuda()
        segs_p, segs_f = P.Segments(idx.size, w.n_adapters), P.Segments(idx.size, w.n_adapters)
        y_p, y_f = y0.clone(), y0.clone()
        P.segment_apply(idx_d, x, ad, segs_p, y_p, ws)
        P.segment_apply(idx_d, x, full, segs_f, y_f, ws)
        torch.cuda.synchronize()
        wk = W.with_idx(w, idx)
        yref, yout = oracle_y(wk)
        check_y(bits16(y_p), yref, yout, wk, strict_l2=True)
        assert (bits16(y_p) == bits16(y_f)).all(), step
        served = Bc > 0
        n_e1 += int((served & d.resident).sum())
        if budget == 0:
            assert not d.resident.any()
        res = d.resident
        temp.step()
    if budget_frac >= 0.2:
        assert n_e1 > 0      # the hot adapters were served from HBM
    assert ws.counters() == (0, 0)
