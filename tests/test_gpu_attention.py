"""GPU parity of the split-KV decode attention (section V-B) against the
float64 oracle: partials, merge, the whole call, any arrival order, and the
edge lengths (empty, one key, partition boundaries, the full cache)."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
from oracle import attention as OA  # noqa: E402

D = 128
C = 256


@pytest.fixture(scope="module")
def P():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2608_05483_amd import plora
    return plora


def bits(a):
    return oracle.f32_to_bf16(np.asarray(a, np.float32))


def case(seed, Bn, H, Lmax, lens):
    rng = np.random.default_rng(seed)
    q = bits(rng.normal(0, 1, (Bn, H, D)))
    K = bits(rng.normal(0, 1, (Bn, H, Lmax, D)))
    V = bits(rng.normal(0, 1, (Bn, H, Lmax, D)))
    return q, K, V, np.asarray(lens, np.int32)


def dev(a):
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).cuda()


def run_partial(P, q, K, V, lens, scale):
    Bn, H, Lmax = K.shape[:3]
    Pn = P.attn_partitions(Lmax)
    m = torch.full((Bn, H, Pn), float("nan"), device="cuda")
    l = torch.full((Bn, H, Pn), float("nan"), device="cuda")
    o = torch.full((Bn, H, Pn, D), float("nan"), device="cuda")
    P.attn_partial(dev(q), dev(K), dev(V), dev(lens), scale, m, l, o)
    torch.cuda.synchronize()
    return m, l, o


def check_out(out_bits, ref):
    got = oracle.bf16_to_f32(out_bits).astype(np.float64)
    assert np.isfinite(got).all()
    assert (np.abs(got - ref) <= 1e-2 * (1 + np.abs(ref))).all()
    # bf16 output: half an ulp (2^-9 relative) plus fp32 accumulation
    assert (np.abs(got - ref) <= 2.0 ** -8 * np.abs(ref) + 1e-4).all()


EDGE_LENS = [0, 1, 255, 256, 257, 700, 1024]


@pytest.mark.parametrize("scale", [1 / np.sqrt(D), 0.5])
def test_partials_match_the_oracle(P, scale):
    q, K, V, lens = case(1, 7, 3, 1024, EDGE_LENS)
    m, l, o = run_partial(P, q, K, V, lens, scale)
    mr, lr, orf = OA.partial(q, K, V, lens, scale, C)
    m, l, o = m.cpu().numpy(), l.cpu().numpy(), o.cpu().numpy()
    for b, n in enumerate(lens):
        np_ = -(-int(n) // C)
        assert np.isnan(m[b, :, np_:]).all()                  # past len: not written
        if np_ == 0:
            continue
        mm, mrr = m[b, :, :np_], mr[b, :, :np_]
        # scores: 128 exact products summed in fp32
        assert np.allclose(mm, mrr, rtol=1e-5, atol=1e-5)
        # the shifted sums and outputs, relative to their magnitude
        w = np.exp(mm.astype(np.float64) - mrr)               # anchors differ in the last bits
        assert np.allclose(l[b, :, :np_], lr[b, :, :np_] * w, rtol=2e-5, atol=1e-6)
        assert np.allclose(o[b, :, :np_], orf[b, :, :np_] * w[..., None], rtol=2e-4,
                           atol=2e-4 * np.abs(orf[b, :, :np_]).max())


def test_decode_matches_the_definition(P):
    q, K, V, lens = case(2, 7, 3, 1024, EDGE_LENS)
    scale = 1 / np.sqrt(D)
    out = torch.zeros((7, 3, D), dtype=torch.int16, device="cuda")
    ws = torch.empty(P.attn_workspace_bytes(7, 3, 1024), dtype=torch.uint8, device="cuda")
    P.attn_decode(dev(q), dev(K), dev(V), dev(lens), scale, out, ws)
    torch.cuda.synchronize()
    ob = out.cpu().numpy().view(np.uint16)
    ref = OA.attention(q, K, V, lens, scale)
    check_out(ob, ref)
    assert (ob[0] == 0).all()                                 # len 0: zeros
    # relative L2 error of the whole output
    got = oracle.bf16_to_f32(ob).astype(np.float64)
    assert np.linalg.norm(got - ref) / np.linalg.norm(ref) <= 4e-3


def test_merge_of_the_oracles_partials(P):
    q, K, V, lens = case(3, 4, 2, 900, [900, 300, 1, 513])
    scale = 0.2
    mr, lr, orf = OA.partial(q, K, V, lens, scale, C)
    out = torch.zeros((4, 2, D), dtype=torch.int16, device="cuda")
    f32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()
    P.attn_merge(f32(mr), f32(lr), f32(orf), dev(lens), out, 900)
    torch.cuda.synchronize()
    check_out(out.cpu().numpy().view(np.uint16), OA.attention(q, K, V, lens, scale))


def test_any_arrival_order(P):
    """The partials of a full-length request permuted along the partition
    axis (as if they had arrived in another order) merge to the same output
    within rounding."""
    q, K, V, lens = case(4, 2, 4, 2048, [2048, 2048])
    m, l, o = run_partial(P, q, K, V, lens, 0.1)
    out0 = torch.zeros((2, 4, D), dtype=torch.int16, device="cuda")
    P.attn_merge(m, l, o, dev(lens), out0, 2048)
    ref = OA.attention(q, K, V, lens, 0.1)
    rng = np.random.default_rng(0)
    for _ in range(3):
        perm = torch.from_numpy(rng.permutation(m.shape[2])).cuda()
        out = torch.zeros_like(out0)
        P.attn_merge(m[:, :, perm].contiguous(), l[:, :, perm].contiguous(),
                     o[:, :, perm].contiguous(), dev(lens), out, 2048)
        torch.cuda.synchronize()
        check_out(out.cpu().numpy().view(np.uint16), ref)
    check_out(out0.cpu().numpy().view(np.uint16), ref)


def test_deterministic(P):
    q, K, V, lens = case(5, 3, 2, 600, [600, 17, 256])
    ws = torch.empty(P.attn_workspace_bytes(3, 2, 600), dtype=torch.uint8, device="cuda")
    outs = []
    for _ in range(3):
        out = torch.zeros((3, 2, D), dtype=torch.int16, device="cuda")
        P.attn_decode(dev(q), dev(K), dev(V), dev(lens), 0.3, out, ws)
        torch.cuda.synchronize()
        outs.append(out.cpu())
    assert all(torch.equal(outs[0], x) for x in outs[1:])


def test_llama7b_decode_shape(P):
    """32 heads, caches of up to 4096 keys, 8 requests (two of them full, at
    4096 keys): every head of the two full requests and of one more, and four
    sampled (request, head) pairs of the others, checked element-wise against
    the oracle."""
    rng = np.random.default_rng(6)
    Bn, H, Lmax = 8, 32, 4096
    lens = rng.integers(512, Lmax + 1, Bn).astype(np.int32)
    lens[0] = lens[3] = Lmax
    g = torch.Generator(device="cuda").manual_seed(6)
    to_bits = lambda t: t.to(torch.bfloat16).view(torch.int16)
    q = to_bits(torch.randn((Bn, H, D), device="cuda", generator=g))
    K = to_bits(torch.randn((Bn, H, Lmax, D), device="cuda", generator=g))
    V = to_bits(torch.randn((Bn, H, Lmax, D), device="cuda", generator=g))
    out = torch.zeros((Bn, H, D), dtype=torch.int16, device="cuda")
    ws = torch.empty(P.attn_workspace_bytes(Bn, H, Lmax), dtype=torch.uint8, device="cuda")
    scale = 1 / np.sqrt(D)
    P.attn_decode(q, K, V, dev(lens), scale, out, ws)
    torch.cuda.synchronize()
    ob = out.cpu().numpy().view(np.uint16)
    u16 = lambda t: t.cpu().numpy().view(np.uint16)
    for b in (0, 3, 6):
        print(f"attention request {b}: all {H} heads, {int(lens[b])} keys", flush=True)
        ref = OA.attention(u16(q[b:b + 1]), u16(K[b:b + 1]), u16(V[b:b + 1]), lens[b:b + 1],
                           scale)
        check_out(ob[b:b + 1], ref)
    for b, h in [(1, 0), (2, 17), (7, 31), (5, 8)]:
        ref = OA.attention(u16(q[b:b + 1, h:h + 1]), u16(K[b:b + 1, h:h + 1]),
                           u16(V[b:b + 1, h:h + 1]), lens[b:b + 1], scale)
        check_out(ob[b:b + 1, h:h + 1], ref)
