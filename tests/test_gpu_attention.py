"""GPU parity of the paged-attention decode over a tiered KV pool."""
import numpy as np
import pytest

import synth
from oracle import attention as oa
from oracle import gemv as og
from oracle import kvpool as okv
from paper_2609_13592_amd import binding as bd
from tests.gpu_util import dev_f32, dev_u16, fill_pool, host_u16, stream, sync, to_dev_u16

pytestmark = pytest.mark.gpu
TOL = 2e-2


def run_attn(ctx, pool, layer, q, tables, lens, out_dtype=bd.DTYPE_F32, scale=0.0):
    import torch
    B, Hq, D = q.shape
    qd = to_dev_u16(q)
    td = torch.from_numpy(np.ascontiguousarray(tables, dtype=np.int32)).cuda()
    ld = torch.from_numpy(np.asarray(lens, dtype=np.int32)).cuda()
    out = dev_f32(B, Hq, D) if out_dtype == bd.DTYPE_F32 else dev_u16(B, Hq, D)
    bd.boost_paged_attn_decode(ctx, pool, layer, qd, B, Hq, td, tables.shape[1], ld,
                               scale, out, out_dtype, stream())
    sync()
    return out.cpu().numpy() if out_dtype == bd.DTYPE_F32 else host_u16(out)


def new_pool(ctx, H, Hq, nb, M, mode, layers=1, max_batch=64, max_blocks=256,
             budget=0):
    return bd.boost_kv_pool_create(ctx, layers, H, 128, nb, M, mode, q_heads=Hq,
                                   max_batch=max_batch, max_blocks_per_seq=max_blocks,
                                   hbm_budget_bytes=budget)


@pytest.mark.parametrize("Hq,H", [(32, 8), (64, 8), (8, 8), (16, 8)])
def test_small_parity_and_placement_invariance(gpu_ctx, Hq, H):
    lengths = np.array([1, 15, 16, 17, 300, 1000, 0, 2049])
    _, q, ks, vs = synth.attention_inputs(len(lengths), Hq, H, 128, 0, 0, seed=4,
                                          kv_seed=5, lengths=lengths)
    ref = oa.decode_attention(q, ks, vs)
    outs = []
    # the budget leaves 9 of each tensor's 32 pages in HBM: blocks carry 5 or
    # 6 host heads of 8
    budget = 2 * 9 * bd.PAGE_BYTES
    for mode, M in ((bd.KV_ALL_HBM, 0), (bd.KV_LPP, 3), (bd.KV_ALL_HOST, 0),
                    (bd.KV_BUDGET, 0)):
        pool = new_pool(gpu_ctx, H, Hq, 2000, M, mode, max_blocks=160, budget=budget)
        try:
            if mode == bd.KV_BUDGET:
                info = bd.boost_kv_pool_info(pool)
                assert info["host_pages_per_tensor"] == 23
                assert (info["local_host_heads"], info["shh_host_heads"]) == (5, 6)
            tables = fill_pool(bd, gpu_ctx, pool, 0, lengths, ks, vs)
            o = run_attn(gpu_ctx, pool, 0, q, tables, lengths)
            assert og.rel_err(o, ref) <= TOL
            assert np.max(np.abs(o - ref)) < 1e-4
            assert np.all(o[6] == 0)             # empty context: zero row
            outs.append(o)
        finally:
            bd.boost_kv_pool_destroy(pool)
    for o in outs[1:]:
        assert np.array_equal(o.view(np.uint32), outs[0].view(np.uint32))


@pytest.mark.parametrize("Hq,H", [(4, 2), (8, 1), (32, 8)])
def test_more_than_256_requests(gpu_ctx, Hq, H):
    """300 requests: each workgroup finds its work item from the context
    lengths with sums, prefix scans and a counting sort over chunks of 256
    requests, so the second chunk is exercised; empty contexts and partial
    partitions of every size (16-block partitions) are included, and the
    LPP pool gives the same bits as the all-HBM one."""
    rng = np.random.default_rng(31)
    B = 300
    lengths = rng.integers(1, 700, size=B)
    lengths[::17] = 0
    _, q, ks, vs = synth.attention_inputs(B, Hq, H, 128, 0, 0, seed=32, kv_seed=33,
                                          lengths=lengths)
    ref = oa.decode_attention(q, ks, vs)
    nb = int(sum((int(L) + 15) // 16 for L in lengths)) + 64
    outs = []
    for mode, M in ((bd.KV_ALL_HBM, 0), (bd.KV_LPP, 3)):
        pool = new_pool(gpu_ctx, H, Hq, nb, M, mode, max_batch=B, max_blocks=48)
        try:
            tables = fill_pool(bd, gpu_ctx, pool, 0, lengths, ks, vs)
            o = run_attn(gpu_ctx, pool, 0, q, tables, lengths)
            assert og.rel_err(o, ref) <= TOL
            assert np.max(np.abs(o - ref)) < 1e-4
            assert np.all(o[lengths == 0] == 0)
            outs.append(o)
        finally:
            bd.boost_kv_pool_destroy(pool)
    assert np.array_equal(outs[1].view(np.uint32), outs[0].view(np.uint32))


def test_host_heads_follow_block_types(gpu_ctx):
    """LPP with H = 8 and a modulus above H: the tail lies in head 7, so an SHH
    request has exactly its head-7 data on host; output still exact."""
    H, Hq, M = 8, 32, 12
    pool = new_pool(gpu_ctx, H, Hq, 4096, M, bd.KV_LPP)
    try:
        info = bd.boost_kv_pool_info(pool)
        g = okv.kv_geometry(4096, H, 128, M)
        assert info["host_pages_per_tensor"] == g.host_pages
        assert info["shh_host_heads"] == 1 and info["local_host_heads"] == 0
        lengths = synth.context_lengths(9, 16, 200, 900)
        _, q, ks, vs = synth.attention_inputs(16, Hq, H, 128, 0, 0, seed=9, kv_seed=10,
                                              lengths=lengths)
        tables = fill_pool(bd, gpu_ctx, pool, 0, lengths, ks, vs)
        types = [bd.boost_kv_request_type(pool, b) for b in range(16)]
        assert bd.KV_SHH in types and bd.KV_LOCAL in types
        o = run_attn(gpu_ctx, pool, 0, q, tables, lengths)
        assert og.rel_err(o, oa.decode_attention(q, ks, vs)) <= TOL
    finally:
        bd.boost_kv_pool_destroy(pool)


def test_two_layers_and_bf16_output(gpu_ctx):
    H, Hq = 8, 32
    pool = new_pool(gpu_ctx, H, Hq, 1024, 5, bd.KV_LPP, layers=2)
    try:
        lengths = np.array([33, 400, 129])
        _, q, k0, v0 = synth.attention_inputs(3, Hq, H, 128, 0, 0, seed=1, kv_seed=2,
                                              lengths=lengths)
        _, _, k1, v1 = synth.attention_inputs(3, Hq, H, 128, 0, 0, seed=1, kv_seed=3,
                                              lengths=lengths)
        tables = fill_pool(bd, gpu_ctx, pool, 0, lengths, k0, v0)
        fill_pool(bd, gpu_ctx, pool, 1, lengths, k1, v1, tables=tables)
        o0 = run_attn(gpu_ctx, pool, 0, q, tables, lengths)
        o1 = run_attn(gpu_ctx, pool, 1, q, tables, lengths)
        assert og.rel_err(o0, oa.decode_attention(q, k0, v0)) <= TOL
        assert og.rel_err(o1, oa.decode_attention(q, k1, v1)) <= TOL
        ob = run_attn(gpu_ctx, pool, 1, q, tables, lengths, bd.DTYPE_BF16)
        assert np.array_equal(ob, og.f32_to_bf16(o1))
        # an explicit scale replaces 1/sqrt(D)
        o2 = run_attn(gpu_ctx, pool, 0, q, tables, lengths, scale=0.05)
        assert og.rel_err(o2, oa.decode_attention(q, k0, v0, scale=0.05)) <= TOL
    finally:
        bd.boost_kv_pool_destroy(pool)


def test_bad_arguments(gpu_ctx):
    import torch
    pool = new_pool(gpu_ctx, 8, 32, 512, 4, bd.KV_LPP, max_batch=4, max_blocks=8)
    q = dev_u16(4, 32, 128)
    t = torch.zeros((4, 8), dtype=torch.int32, device="cuda")
    lens = torch.zeros(4, dtype=torch.int32, device="cuda")
    out = dev_f32(4, 32, 128)
    try:
        for args in ((0, 5, 32, 8), (0, 4, 16, 8), (0, 4, 32, 9), (1, 4, 32, 8)):
            layer, B, Hq, mb = args
            with pytest.raises(bd.BoostError) as e:
                bd.boost_paged_attn_decode(gpu_ctx, pool, layer, q, B, Hq, t, mb, lens,
                                           0.0, out, bd.DTYPE_F32, stream())
            assert e.value.code == bd.EINVAL
    finally:
        bd.boost_kv_pool_destroy(pool)


def test_config3_full_size_sampled(gpu_ctx):
    """Batch 64, 32/8 heads, lengths U[512, 4096] (seed 0), admitted through
    the allocator after a seeded churn warm-up, pool modulus 111: sampled
    (request, head) pairs against the oracle; the all-HBM pool agrees bitwise."""
    B, Hq, H = 64, 32, 8
    lengths, q, ks, vs = synth.attention_inputs(B, Hq, H, 128, 512, 4096, seed=0,
                                                kv_seed=1)
    need = sum((int(L) + 15) // 16 for L in lengths)
    nb = need + 16384
    outs = []
    for mode, M in ((bd.KV_LPP, 111), (bd.KV_ALL_HBM, 0)):
        pool = new_pool(gpu_ctx, H, Hq, nb, M, mode, max_batch=64, max_blocks=256)
        try:
            # churn warm-up (replace events: retire the victim, admit a new
            # request) so block ids are scattered as in a live pool; a quarter
            # of the churn requests stay alive
            live = set()
            for victim, L in synth.churn_trace(2, 256, 48, 512, 4096):
                r = 1000 + victim
                if r in live:
                    bd.boost_kv_free(pool, r)
                    live.discard(r)
                if bd.boost_kv_alloc(pool, r, (L + 15) // 16) != bd.EAGAIN:
                    live.add(r)
            for r in sorted(live):
                if r % 4:
                    bd.boost_kv_free(pool, r)
            tables = fill_pool(bd, gpu_ctx, pool, 0, lengths, ks, vs, max_blocks=256)
            st = bd.boost_kv_stats(pool)
            assert st["used_blocks"] >= need
            outs.append(run_attn(gpu_ctx, pool, 0, q, tables, lengths))
        finally:
            bd.boost_kv_pool_destroy(pool)
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))
    rng = np.random.default_rng(0)
    pairs = [(int(b), int(h)) for b, h in zip(rng.integers(0, B, 48), rng.integers(0, Hq, 48))]
    pairs += [(0, 0), (B - 1, Hq - 1)]
    ref = oa.decode_attention(q, ks, vs, heads=pairs)
    got = np.array([outs[0][b, h] for b, h in pairs])
    exp = np.array([ref[p] for p in pairs])
    assert og.rel_err(got, exp) <= TOL
    assert np.max(np.abs(got - exp)) < 1e-4


def test_batch256_long_contexts_full_size_sampled(gpu_ctx):
    """The largest configuration: batch 256, 32/8 heads, contexts U[1024,
    8192] (up to 512 blocks, several partitions per request), K/V drawn on
    the device (seeded torch generator) and written through the allocator's
    blocks; an LPP pool at modulus 126 and an all-HBM pool agree bitwise, and
    sampled (request, head) pairs meet the bar against the oracle (their K/V
    copied back from the generator's output, not from the pool)."""
    import torch
    B, Hq, H, D = 256, 32, 8, 128
    lengths = synth.context_lengths(3, B, 1024, 8192)
    rng = np.random.default_rng(4)
    q = synth.normal_bf16(rng, (B, Hq, D), 1.0)
    k, v, offs = synth.attention_kv_torch(lengths, H, D, kv_seed=5, device="cuda")
    need = [(int(L) + 15) // 16 for L in lengths]
    mb = max(need)
    outs = []
    for mode, M in ((bd.KV_LPP, 126), (bd.KV_ALL_HBM, 0)):
        pool = new_pool(gpu_ctx, H, Hq, sum(need), M, mode, max_batch=B, max_blocks=mb)
        try:
            tables = np.full((B, mb), -1, dtype=np.int32)
            for b in range(B):
                got = bd.boost_kv_alloc(pool, b, need[b])
                assert got != bd.EAGAIN
                tables[b, :need[b]] = got
            if mode == bd.KV_LPP:
                assert bd.boost_kv_stats(pool)["shh_requests"] > 0
            slots = np.concatenate([tables[b, np.arange(L) // 16] * 16 + np.arange(L) % 16
                                    for b, L in enumerate(lengths)]).astype(np.int32)
            s = torch.from_numpy(slots).cuda()
            bd.boost_kv_write(gpu_ctx, pool, 0, s, k.view(torch.int16), v.view(torch.int16),
                              int(s.numel()), stream())
            sync()
            outs.append(run_attn(gpu_ctx, pool, 0, q, tables, lengths))
        finally:
            bd.boost_kv_pool_destroy(pool)
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))
    # sampled pairs: the longest request, the last one and seeded draws
    bl = int(np.argmax(lengths))
    reqs = sorted({bl, B - 1, *[int(x) for x in rng.integers(0, B, 6)]})
    pairs = [(b, int(h)) for b in reqs for h in rng.integers(0, Hq, 4)] + [(bl, Hq - 1)]
    ks, vs = {}, {}
    for b in reqs:
        a, L = int(offs[b]), int(lengths[b])
        ks[b] = k[a:a + L].view(torch.int16).cpu().numpy().view(np.uint16)
        vs[b] = v[a:a + L].view(torch.int16).cpu().numpy().view(np.uint16)
    got, exp = [], []
    for b, h in pairs:
        r = oa.decode_attention(q[b:b + 1], [ks[b]], [vs[b]], heads=[(0, h)])
        exp.append(r[(0, h)])
        got.append(outs[0][b, h])
    got, exp = np.array(got), np.array(exp)
    assert og.rel_err(got, exp) <= TOL
    assert np.max(np.abs(got - exp)) < 1e-4


def test_block_ids_outside_pool_are_skipped(gpu_ctx):
    """Block-table entries outside [0, nb_pool) at positions inside the
    context leave their 16 tokens out of the softmax: the output equals the
    oracle's attention over the remaining tokens (checked on the CPU), for
    entries in the unmasked main loop (the first blocks), in the partial
    last block, for a whole group of blocks, and for a request whose every
    block is invalid (zero row).  Under LPP and all-HBM pools alike."""
    H, Hq = 8, 32
    lengths = np.array([100, 300, 700, 40, 2049])
    _, q, ks, vs = synth.attention_inputs(len(lengths), Hq, H, 128, 0, 0, seed=14,
                                          kv_seed=15, lengths=lengths)
    bad = {0: [0, 6], 1: [5, 18], 2: [1, 2, 3, 4, 43], 3: [0, 1, 2], 4: [7, 64, 128]}
    keep_k, keep_v = [], []
    for b, L in enumerate(lengths):
        tok = np.arange(int(L))
        keep = ~np.isin(tok // 16, bad[b])
        keep_k.append(ks[b][keep])
        keep_v.append(vs[b][keep])
    ref = oa.decode_attention(q, keep_k, keep_v)
    outs = []
    for mode, M in ((bd.KV_LPP, 3), (bd.KV_ALL_HBM, 0)):
        pool = new_pool(gpu_ctx, H, Hq, 2000, M, mode, max_blocks=160)
        try:
            tables = fill_pool(bd, gpu_ctx, pool, 0, lengths, ks, vs)
            nb = bd.boost_kv_pool_info(pool)["nb_pool"]
            for b, blks in bad.items():
                for j, blk in enumerate(blks):
                    tables[b, blk] = -1 if j % 2 == 0 else nb + 5 * j
            o = run_attn(gpu_ctx, pool, 0, q, tables, lengths)
            assert np.all(o[3] == 0)             # every block skipped
            assert og.rel_err(o, ref) <= TOL
            assert np.max(np.abs(o - ref)) < 1e-4
            outs.append(o)
        finally:
            bd.boost_kv_pool_destroy(pool)
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))
