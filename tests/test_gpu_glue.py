"""Per-operator parity of the decode-step glue at Llama-3-70B dimensions
(batch 8): each kernel gets the same inputs as the oracle function it
implements."""
import numpy as np
import pytest

import synth
from oracle import decode_step as ods
from oracle.gemv import bf16_to_f32, f32_to_bf16
from paper_2609_13592_amd import binding as bd
from tests.gpu_util import host_u16, slices_sum, stream, sync, to_dev_u16

pytestmark = pytest.mark.gpu
B, D_MODEL, HQ, HKV, HD, FFN, VOCAB = 8, 8192, 64, 8, 128, 28672, 128256


def dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def assert_bf16_close(got_u16, want_u16, frac_exact=0.995):
    """bf16 outputs: every value within one bf16 ulp of the oracle's, and
    almost all bit-identical (the two sides round fp32 and fp64 values that
    can straddle a rounding boundary)."""
    g = bf16_to_f32(got_u16).astype(np.float64)
    w = bf16_to_f32(want_u16).astype(np.float64)
    ulp = np.maximum(np.abs(w), 1e-30) * 2.0 ** -7
    assert np.all(np.abs(g - w) <= ulp)
    assert np.mean(got_u16 == want_u16) >= frac_exact


def test_rmsnorm_70b(gpu_ctx):
    import torch
    rng = np.random.default_rng(0)
    x = (rng.standard_normal((B, D_MODEL)) * 3).astype(np.float32)
    w = synth.round_bf16((1 + 0.1 * rng.standard_normal(D_MODEL)).astype(np.float32))
    out = torch.empty((B, D_MODEL), dtype=torch.int16, device="cuda")
    bd.boost_rmsnorm(gpu_ctx, dev(x), to_dev_u16(w), B, D_MODEL, 1e-5, out, stream())
    sync()
    assert_bf16_close(host_u16(out), ods.to_bf16(ods.rmsnorm(x.astype(np.float64), w)))


@pytest.mark.parametrize("d", [4096, 12288, 1026, 36])
def test_rmsnorm_widths(gpu_ctx, d):
    """Vector path (d % 4 == 0, d <= 8192) and the plain loop (wider rows,
    d % 4 != 0), ragged against 256 lanes."""
    import torch
    rng = np.random.default_rng(d)
    x = (rng.standard_normal((3, d)) * 2).astype(np.float32)
    w = synth.round_bf16((1 + 0.1 * rng.standard_normal(d)).astype(np.float32))
    out = torch.empty((3, d), dtype=torch.int16, device="cuda")
    bd.boost_rmsnorm(gpu_ctx, dev(x), to_dev_u16(w), 3, d, 1e-5, out, stream())
    sync()
    assert_bf16_close(host_u16(out), ods.to_bf16(ods.rmsnorm(x.astype(np.float64), w)))


@pytest.mark.parametrize("V", [1001, 7, 4100])
def test_argmax_lengths(gpu_ctx, V):
    """Plain loop (V % 4 != 0) and the float4 path with a ragged tail; the
    maximum planted at the last index and a tie planted early."""
    rng = np.random.default_rng(V)
    s = rng.standard_normal((4, V)).astype(np.float32)
    s[0, V - 1] = 50.0
    s[1, 2] = s[1, V - 2] = 60.0
    ids = dev(np.zeros(4, np.int32))
    bd.boost_argmax(gpu_ctx, dev(s), 4, V, ids, stream())
    sync()
    got = ids.cpu().numpy().tolist()
    assert got == ods.argmax_lowest(s.astype(np.float64)).tolist()
    assert got[:2] == [V - 1, 2]


def test_rope_qkv_70b(gpu_ctx):
    import torch
    rng = np.random.default_rng(1)
    heads = HQ + 2 * HKV
    qkv = rng.standard_normal((B, heads * HD)).astype(np.float32)
    pos = np.array([0, 1, 15, 16, 1000, 2047, 4095, 8191], dtype=np.int32)
    q = torch.empty((B, HQ, HD), dtype=torch.int16, device="cuda")
    k = torch.empty((B, HKV, HD), dtype=torch.int16, device="cuda")
    v = torch.empty((B, HKV, HD), dtype=torch.int16, device="cuda")
    bd.boost_rope_qkv(gpu_ctx, dev(qkv), dev(pos), B, HQ, HKV, HD, 500000.0, q, k, v, stream())
    sync()
    x = qkv.astype(np.float64)
    want_q = ods.to_bf16(ods.rope(x[:, :HQ * HD].reshape(B, HQ, HD), pos))
    want_k = ods.to_bf16(ods.rope(x[:, HQ * HD:(HQ + HKV) * HD].reshape(B, HKV, HD), pos))
    want_v = ods.to_bf16(x[:, (HQ + HKV) * HD:].reshape(B, HKV, HD))
    assert_bf16_close(host_u16(q), want_q)
    assert_bf16_close(host_u16(k), want_k)
    assert np.array_equal(host_u16(v), want_v)


def test_silu_mul_70b(gpu_ctx):
    import torch
    rng = np.random.default_rng(2)
    gu = (rng.standard_normal((B, 2 * FFN)) * 4).astype(np.float32)
    out = torch.empty((B, FFN), dtype=torch.int16, device="cuda")
    bd.boost_silu_mul(gpu_ctx, dev(gu), B, FFN, out, stream())
    sync()
    g = gu[:, :FFN].astype(np.float64)
    u = gu[:, FFN:].astype(np.float64)
    assert_bf16_close(host_u16(out), ods.to_bf16(ods.silu(g) * u))


def test_embed_gather_through_tiered_pages(gpu_ctx):
    import torch
    g = torch.Generator(device="cuda")
    g.manual_seed(3)
    e = torch.randn((VOCAB, D_MODEL), generator=g, device="cuda").to(torch.bfloat16)
    E = bd.boost_place_weights(gpu_ctx, e.view(torch.int16), VOCAB * D_MODEL * 2, 6)
    try:
        assert bd.boost_tensor_tiers(E).sum() > 0
        tok = np.array([0, 1, 127, 128, 640, 65535, VOCAB - 1, VOCAB], dtype=np.int32)
        out = torch.empty((B, D_MODEL), dtype=torch.float32, device="cuda")
        bd.boost_embed_gather(gpu_ctx, E, VOCAB, D_MODEL, dev(tok), B, out, stream())
        sync()
        got = out.cpu().numpy()
        rows = e.view(torch.int16)[torch.from_numpy(tok[:-1].astype(np.int64)).cuda()]
        want = bf16_to_f32(rows.cpu().numpy().view(np.uint16))
        assert np.array_equal(got[:-1], want)
        assert np.all(got[-1] == 0)          # token outside the vocabulary
    finally:
        bd.boost_tensor_free(E)


def test_residual_and_argmax(gpu_ctx):
    rng = np.random.default_rng(4)
    x = rng.standard_normal((B, VOCAB)).astype(np.float32)
    y = rng.standard_normal((B, VOCAB)).astype(np.float32)
    xd = dev(x)
    bd.boost_residual_add(gpu_ctx, xd, dev(y), B * VOCAB, stream())
    sync()
    s = xd.cpu().numpy()
    assert np.array_equal(s, x + y)
    # ties: plant equal maxima, the lowest index must win
    s[0, 5] = s[0, 77] = s[0, 100000] = 1e6
    s[1, :] = 0.0
    s[2, VOCAB - 1] = 1e7
    ids = dev(np.zeros(B, np.int32))
    bd.boost_argmax(gpu_ctx, dev(s), B, VOCAB, ids, stream())
    sync()
    assert ids.cpu().numpy().tolist() == ods.argmax_lowest(s.astype(np.float64)).tolist()
    assert ids.cpu().numpy()[:3].tolist() == [5, 0, VOCAB - 1]


@pytest.mark.parametrize("d", [8192, 4096, 12288, 1026])
def test_add_rmsnorm_equals_add_then_norm(gpu_ctx, d):
    """The fused residual add + RMSNorm leaves the same x and writes the same
    bits as the residual add followed by the norm (vector path and plain
    loop), and x + r meets the oracle's norm."""
    import torch
    rng = np.random.default_rng(100 + d)
    x = (rng.standard_normal((5, d)) * 2).astype(np.float32)
    r = (rng.standard_normal((5, d)) * 2).astype(np.float32)
    w = synth.round_bf16((1 + 0.1 * rng.standard_normal(d)).astype(np.float32))
    wd = to_dev_u16(w)
    x1, x2 = dev(x), dev(x)
    o1 = torch.empty((5, d), dtype=torch.int16, device="cuda")
    o2 = torch.empty((5, d), dtype=torch.int16, device="cuda")
    bd.boost_residual_add(gpu_ctx, x1, dev(r), 5 * d, stream())
    bd.boost_rmsnorm(gpu_ctx, x1, wd, 5, d, 1e-5, o1, stream())
    bd.boost_add_rmsnorm(gpu_ctx, x2, dev(r), wd, 5, d, 1e-5, o2, stream())
    sync()
    assert np.array_equal(x2.cpu().numpy(), x + r)
    assert np.array_equal(x1.cpu().numpy(), x2.cpu().numpy())
    assert np.array_equal(host_u16(o1), host_u16(o2))
    assert_bf16_close(host_u16(o2), ods.to_bf16(ods.rmsnorm((x + r).astype(np.float64), w)))
    with pytest.raises(bd.BoostError) as e:
        bd.boost_add_rmsnorm(gpu_ctx, x2, None, wd, 5, d, 1e-5, o2, stream())
    assert e.value.code == bd.EINVAL


def random_slices(rng, S, B, N, K):
    """A slice buffer in the GEMV's layout: S random slices [S][B][N] and, for
    the rows of an [N, K] matrix that cross a page, random parts after them."""
    pages = -(-N * K // (1 << 20))
    tail = (pages + 1) * 2 * S * B if S > 1 else 0
    return (rng.standard_normal(S * B * N + tail) * 2).astype(np.float32)


@pytest.mark.parametrize("d,S,K", [(4096, 1, 4096), (4096, 4, 4096), (8192, 8, 8192),
                                   (1026, 3, 4096), (4096, 4, 14336), (4096, 8, 14336),
                                   (1026, 2, 3000)])
def test_add_rmsnorm_slices_equals_sum_then_fused(gpu_ctx, d, S, K):
    """With the residual handed over as S split-K slices of a [d, K] matrix
    (K = 14336 and 3000: rows cut by pages, whose parts follow the slices), x
    and the norm get the same bits as the fused call on the sum the header
    defines (vector path and plain loop); bad slice counts are refused."""
    import torch
    rng = np.random.default_rng(200 + d + S + K)
    Bn = 6
    x = (rng.standard_normal((Bn, d)) * 2).astype(np.float32)
    flat = random_slices(rng, S, Bn, d, K)
    r = slices_sum(flat, S, Bn, d, K)
    w = synth.round_bf16((1 + 0.1 * rng.standard_normal(d)).astype(np.float32))
    wd = to_dev_u16(w)
    x1, x2 = dev(x), dev(x)
    o1 = torch.empty((Bn, d), dtype=torch.int16, device="cuda")
    o2 = torch.empty((Bn, d), dtype=torch.int16, device="cuda")
    bd.boost_add_rmsnorm(gpu_ctx, x1, dev(r), wd, Bn, d, 1e-5, o1, stream())
    bd.boost_add_rmsnorm_slices(gpu_ctx, x2, dev(flat), S, K, wd, Bn, d, 1e-5, o2, stream())
    sync()
    assert np.array_equal(x2.cpu().numpy().view(np.uint32), (x + r).view(np.uint32))
    assert np.array_equal(x1.cpu().numpy().view(np.uint32), x2.cpu().numpy().view(np.uint32))
    assert np.array_equal(host_u16(o1), host_u16(o2))
    assert_bf16_close(host_u16(o2), ods.to_bf16(ods.rmsnorm((x + r).astype(np.float64), w)))
    for bad_s, bad_k in ((0, K), (bd.MAX_GEMV_SLICES + 1, K), (S, 0)):
        with pytest.raises(bd.BoostError) as e:
            bd.boost_add_rmsnorm_slices(gpu_ctx, x2, dev(flat), bad_s, bad_k, wd, Bn, d, 1e-5,
                                        o2, stream())
        assert e.value.code == bd.EINVAL


@pytest.mark.parametrize("S,K", [(1, 8192), (2, 8192), (8, 8192), (4, 14336)])
def test_rope_kv_append_slices_equals_sum(gpu_ctx, S, K):
    """RoPE + KV append of S qkv slices (K = 14336: rows cut by pages) writes
    the same q and pool slots as the call on their sum (attention over the two
    pools agrees bitwise)."""
    import torch
    rng = np.random.default_rng(30 + S + K)
    heads = HQ + 2 * HKV
    mb = 8
    pos = np.array([0, 3, 15, 16, 40, 77, 100, 127], dtype=np.int32)
    flat = random_slices(rng, S, B, heads * HD, K)
    qkv = slices_sum(flat, S, B, heads * HD, K)
    pools, outs, qs = [], [], []
    try:
        for sliced in (False, True):
            pool = bd.boost_kv_pool_create(gpu_ctx, 1, HKV, HD, B * mb, 0, bd.KV_ALL_HBM,
                                           q_heads=HQ, max_batch=B, max_blocks_per_seq=mb)
            pools.append(pool)
            tables = np.stack([bd.boost_kv_alloc(pool, b, mb) for b in range(B)]).astype(np.int32)
            td, pd = dev(tables), dev(pos)
            q = torch.empty((B, HQ, HD), dtype=torch.int16, device="cuda")
            if sliced:
                bd.boost_rope_kv_append_slices(gpu_ctx, pool, 0, dev(flat), S, K, pd, B, HQ,
                                               500000.0, td, mb, q, stream())
            else:
                bd.boost_rope_kv_append(gpu_ctx, pool, 0, dev(qkv), pd, B, HQ, 500000.0, td, mb,
                                        q, stream())
            lens = (pos + 1).astype(np.int32)
            out = torch.empty((B, HQ, HD), dtype=torch.float32, device="cuda")
            bd.boost_paged_attn_decode(gpu_ctx, pool, 0, q, B, HQ, td, mb, dev(lens), 0.0, out,
                                       bd.DTYPE_F32, stream())
            sync()
            qs.append(host_u16(q))
            outs.append(out.cpu().numpy())
        assert np.array_equal(qs[0], qs[1])
        assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))
        with pytest.raises(bd.BoostError) as e:
            bd.boost_rope_kv_append_slices(gpu_ctx, pools[1], 0, dev(flat), 0, K, dev(pos), B,
                                           HQ, 500000.0, dev(np.zeros((B, mb), np.int32)), mb,
                                           dev(qs[1]), stream())
        assert e.value.code == bd.EINVAL
    finally:
        for p in pools:
            bd.boost_kv_pool_destroy(p)


def test_rope_kv_append_equals_pair(gpu_ctx):
    """The fused RoPE + KV append writes the same q as the RoPE call and the
    same pool slots as the KV append (two identical all-HBM pools, one filled
    each way: attention over them agrees bitwise; a one-token context returns
    the appended value head exactly); a position outside the table is
    skipped by both."""
    import torch
    rng = np.random.default_rng(7)
    heads = HQ + 2 * HKV
    G = HQ // HKV
    mb = 32  # blocks per request in the table (512 positions)
    pos = np.array([0, 1, 15, 16, 100, 255, 511, mb * 16], dtype=np.int32)  # last: outside
    qkv = rng.standard_normal((B, heads * HD)).astype(np.float32)
    pools, outs, qs = [], [], []
    try:
        for fused in (False, True):
            pool = bd.boost_kv_pool_create(gpu_ctx, 2, HKV, HD, B * mb, 0, bd.KV_ALL_HBM,
                                           q_heads=HQ, max_batch=B, max_blocks_per_seq=mb)
            pools.append(pool)
            tables = np.stack([bd.boost_kv_alloc(pool, b, mb) for b in range(B)]).astype(np.int32)
            td, pd = dev(tables), dev(pos)
            q = torch.empty((B, HQ, HD), dtype=torch.int16, device="cuda")
            if fused:
                bd.boost_rope_kv_append(gpu_ctx, pool, 1, dev(qkv), pd, B, HQ, 500000.0, td,
                                        mb, q, stream())
            else:
                k = torch.empty((B, HKV, HD), dtype=torch.int16, device="cuda")
                v = torch.empty((B, HKV, HD), dtype=torch.int16, device="cuda")
                bd.boost_rope_qkv(gpu_ctx, dev(qkv), pd, B, HQ, HKV, HD, 500000.0, q, k, v,
                                  stream())
                bd.boost_kv_append(gpu_ctx, pool, 1, td, mb, pd, k, v, B, stream())
            lens = np.minimum(pos + 1, mb * 16).astype(np.int32)
            out = torch.empty((B, HQ, HD), dtype=torch.float32, device="cuda")
            bd.boost_paged_attn_decode(gpu_ctx, pool, 1, q, B, HQ, td, mb, dev(lens), 0.0, out,
                                       bd.DTYPE_F32, stream())
            sync()
            qs.append(host_u16(q))
            outs.append(out.cpu().numpy())
        assert np.array_equal(qs[0], qs[1])
        assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))
        # request 0 has one token: its output is the appended value head itself
        want_v = bf16_to_f32(ods.to_bf16(qkv[0, (HQ + HKV) * HD:].astype(np.float64)))
        want_v = want_v.reshape(HKV, HD)
        for h in range(HQ):
            assert np.array_equal(outs[1][0, h], want_v[h // G])
        with pytest.raises(bd.BoostError) as e:
            bd.boost_rope_kv_append(gpu_ctx, pools[1], 2, dev(qkv), dev(pos), B, HQ, 500000.0,
                                    dev(np.zeros((B, mb), np.int32)), mb, dev(qs[1]),
                                    stream())
        assert e.value.code == bd.EINVAL
    finally:
        for p in pools:
            bd.boost_kv_pool_destroy(p)
