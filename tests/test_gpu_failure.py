"""Failure injection on the GPU: a forced host-allocation failure while placing
a tensor or creating a KV pool returns BOOST_ENOMEM and frees the HBM it had
already taken."""
import numpy as np
import pytest

import synth
from oracle import placement as opl
from paper_2609_13592_amd import binding as bd

pytestmark = pytest.mark.gpu


def test_forced_host_alloc_failure_frees_hbm(gpu_ctx, monkeypatch):
    import torch
    torch.cuda.synchronize()
    w, _ = synth.gemv_inputs(3, 4096, 4096, 1)          # 16 pages
    free0 = torch.cuda.mem_get_info()[0]
    monkeypatch.setenv("BOOST_FAULT_HOST_ALLOC", "1")
    for _ in range(3):
        with pytest.raises(bd.BoostError) as e:
            bd.boost_place_weights(gpu_ctx, w, w.nbytes, 4)     # 4 host pages
        assert e.value.code == bd.ENOMEM
        with pytest.raises(bd.BoostError) as e:
            bd.boost_kv_pool_create(gpu_ctx, 2, 8, 128, 4096, 3, bd.KV_LPP, q_heads=32,
                                    max_batch=4, max_blocks_per_seq=64)
        assert e.value.code == bd.ENOMEM
    # an all-HBM tensor needs no host memory and still places
    t = bd.boost_place_weights_map(gpu_ctx, w, w.nbytes, np.zeros(16, np.uint8))
    bd.boost_tensor_free(t)
    torch.cuda.synchronize()
    assert torch.cuda.mem_get_info()[0] >= free0 - (4 << 20)
    monkeypatch.delenv("BOOST_FAULT_HOST_ALLOC")
    t = bd.boost_place_weights(gpu_ctx, w, w.nbytes, 4)
    try:
        assert np.array_equal(bd.boost_tensor_tiers(t), opl.mpp_tier_map(w.nbytes, 4))
    finally:
        bd.boost_tensor_free(t)
