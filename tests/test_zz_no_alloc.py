"""The allocation-free attention entry point (partials in the library's static
device scratch) against the pool-scratch entry point: the same bits, on two
calls in a row (the second smaller), both within the bar of the oracle; calls
beyond the scratch's size are refused."""
import numpy as np
import pytest

import synth
from oracle import attention as oa
from oracle import gemv as og
from paper_2609_13592_amd import binding as bd
from tests.gpu_util import dev_f32, fill_pool, stream, sync, to_dev_u16

pytestmark = pytest.mark.gpu


def _call(fn, ctx, pool, q, tables, lens):
    import torch
    B, Hq, D = q.shape
    out = dev_f32(B, Hq, D)
    out.fill_(np.nan)
    fn(ctx, pool, 0, to_dev_u16(q), B, Hq,
       torch.from_numpy(np.ascontiguousarray(tables, np.int32)).cuda(), tables.shape[1],
       torch.from_numpy(np.asarray(lens, np.int32)).cuda(), 0.0, out, bd.DTYPE_F32, stream())
    sync()
    return out.cpu().numpy()


def test_noalloc_attention_matches_pool_scratch(gpu_ctx):
    H, Hq = 8, 32
    pool = bd.boost_kv_pool_create(gpu_ctx, 1, H, 128, 6000, 3, bd.KV_LPP, q_heads=Hq,
                                   max_batch=64, max_blocks_per_seq=256)
    try:
        cases = [synth.context_lengths(31, 24, 100, 4096),      # first call: larger
                 np.array([1, 17, 300])]                          # second: smaller
        for i, lengths in enumerate(cases):
            _, q, ks, vs = synth.attention_inputs(len(lengths), Hq, H, 128, 0, 0,
                                                  seed=40 + i, kv_seed=50 + i,
                                                  lengths=lengths)
            tables = fill_pool(bd, gpu_ctx, pool, 0, lengths, ks, vs, rid_base=1000 * i)
            o_static = _call(bd.boost_paged_attn_decode_noalloc, gpu_ctx, pool, q, tables,
                             lengths)
            o_pool = _call(bd.boost_paged_attn_decode, gpu_ctx, pool, q, tables, lengths)
            assert np.array_equal(o_static.view(np.uint32), o_pool.view(np.uint32)), i
            heads = [(b, h) for b in range(len(lengths)) for h in (0, 13, 31)]
            ref = oa.decode_attention(q, ks, vs, heads=heads)
            got = np.stack([o_static[b, h] for b, h in heads])
            exp = np.stack([ref[k] for k in heads])
            assert og.rel_err(got, exp) <= 2e-2
            assert np.max(np.abs(got - exp)) < 1e-4
    finally:
        bd.boost_kv_pool_destroy(pool)


def test_noalloc_attention_refuses_beyond_scratch(gpu_ctx):
    """65 requests x 64 query heads x 8 partitions = 33280 partial rows, over
    the 32768 the static scratch holds: EINVAL before any launch (the pool's
    own scratch serves the same call)."""
    import torch
    H, Hq, B, mb = 8, 64, 65, 2048
    pool = bd.boost_kv_pool_create(gpu_ctx, 1, H, 128, 600, 3, bd.KV_LPP, q_heads=Hq,
                                   max_batch=B, max_blocks_per_seq=mb)
    try:
        q = torch.zeros((B, Hq, 128), dtype=torch.int16, device="cuda")
        tables = torch.full((B, mb), -1, dtype=torch.int32, device="cuda")
        lens = torch.zeros(B, dtype=torch.int32, device="cuda")
        out = dev_f32(B, Hq, 128)
        with pytest.raises(bd.BoostError) as e:
            bd.boost_paged_attn_decode_noalloc(gpu_ctx, pool, 0, q, B, Hq, tables, mb, lens,
                                               0.0, out, bd.DTYPE_F32, stream())
        assert e.value.code == bd.EINVAL
        bd.boost_paged_attn_decode(gpu_ctx, pool, 0, q, B, Hq, tables, mb, lens, 0.0, out,
                                   bd.DTYPE_F32, stream())
        sync()
        assert torch.all(out == 0)
    finally:
        bd.boost_kv_pool_destroy(pool)
