"""The decode calls inside a captured HIP graph: every replay (with eager
work and synchronisations between the replays) gives the bits of the eager
calls.  Covers the GEMV with a page-boundary fix-up (rows cut between pages
of different tiers), the split-K matrix-core GEMM with its reduction, and
paged attention with its partition merge."""
import numpy as np
import pytest

import synth
from oracle import placement as opl
from paper_2609_13592_amd import binding as bd
from tests.gpu_util import dev_f32, fill_pool, stream, sync, to_dev_u16

pytestmark = pytest.mark.gpu


def test_graph_replays_match_eager(gpu_ctx):
    import torch
    # GEMV: K = 14336 rows are cut by page boundaries; alternating tiers put
    # every cut between an HBM and a host page (split_fixup runs)
    w1, x1 = synth.gemv_inputs(31, 300, 14336, 1)
    n1 = opl.n_pages(w1.nbytes)
    t1 = bd.boost_place_weights_map(gpu_ctx, w1, w1.nbytes, (np.arange(n1) % 2).astype(np.uint8))
    # matrix-core GEMM at batch 64 with K split over workgroups
    w2, x2 = synth.gemv_inputs(32, 4096, 4096, 64)
    t2 = bd.boost_place_weights(gpu_ctx, w2, w2.nbytes, 3)
    B, Hq, H = 16, 32, 8
    lengths, q, ks, vs = synth.attention_inputs(B, Hq, H, 128, 100, 3000, seed=33, kv_seed=34)
    need = sum((int(L) + 15) // 16 for L in lengths)
    pool = bd.boost_kv_pool_create(gpu_ctx, 1, H, 128, need + 512, 3, bd.KV_LPP, q_heads=Hq,
                                   max_batch=B, max_blocks_per_seq=256)
    try:
        tables = fill_pool(bd, gpu_ctx, pool, 0, lengths, ks, vs, max_blocks=256)
        xd1, xd2, qd = to_dev_u16(x1), to_dev_u16(x2), to_dev_u16(q)
        td = torch.from_numpy(tables).cuda()
        ld = torch.from_numpy(lengths.astype(np.int32)).cuda()
        y1, y2, o = dev_f32(1, 300), dev_f32(64, 4096), dev_f32(B, Hq, 128)

        def calls(s):
            bd.boost_decode_gemv(gpu_ctx, t1, 300, 14336, xd1, 1, y1, bd.DTYPE_F32, s)
            bd.boost_decode_gemv(gpu_ctx, t2, 4096, 4096, xd2, 64, y2, bd.DTYPE_F32, s)
            bd.boost_paged_attn_decode(gpu_ctx, pool, 0, qd, B, Hq, td, 256, ld, 0.0, o,
                                       bd.DTYPE_F32, s)

        calls(stream())
        sync()
        eager = [t.cpu().numpy().copy() for t in (y1, y2, o)]
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            calls(torch.cuda.current_stream().cuda_stream)
        for rep in range(3):
            for t in (y1, y2, o):
                t.fill_(float("nan"))
            # eager work between replays: the same calls into other buffers
            bd.boost_decode_gemv(gpu_ctx, t2, 4096, 4096, xd2, 64, dev_f32(64, 4096),
                                 bd.DTYPE_F32, stream())
            sync()
            g.replay()
            sync()
            for want, got in zip(eager, (y1, y2, o)):
                assert np.array_equal(got.cpu().numpy().view(np.uint32), want.view(np.uint32)), rep
        del g
    finally:
        bd.boost_kv_pool_destroy(pool)
        bd.boost_tensor_free(t1)
        bd.boost_tensor_free(t2)
