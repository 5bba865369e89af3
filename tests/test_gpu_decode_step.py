"""GPU parity of a full decode step (glue + GEMV + attention) against the
oracle, and its invariance to where the weights and the KV live."""
import numpy as np
import pytest

import synth
from oracle import decode_step as ods
from oracle import gemv as og
from paper_2609_13592_amd import binding as bd
from paper_2609_13592_amd.step import DecodeModel, Dims
from tests.gpu_util import fill_pool, sync, to_dev_u16

pytestmark = pytest.mark.gpu
TOL = 2e-2


def model_weights(dims, seed):
    rng = np.random.default_rng(seed)
    d, Hq, H, D, F, V = dims.d, dims.hq, dims.hkv, dims.hd, dims.ffn, dims.vocab
    bfv = lambda a: synth.round_bf16(np.asarray(a, np.float32))
    w = {"embed": synth.normal_bf16(rng, (V, d), 1.0),
         "lm_head": synth.normal_bf16(rng, (V, d), 0.05),
         "norm_f": bfv(1 + 0.1 * rng.standard_normal(d))}
    for l in range(dims.layers):
        w[f"norm1.{l}"] = bfv(1 + 0.1 * rng.standard_normal(d))
        w[f"norm2.{l}"] = bfv(1 + 0.1 * rng.standard_normal(d))
        for name, N, K in dims.shapes():
            w[f"{name}.{l}"] = synth.normal_bf16(rng, (N, K), 0.05)
    return w


def build(ctx, dims, w, lengths, host_weights, pool_mode, M=3, kv_seed=11):
    import torch
    B = len(lengths)
    mats = {}
    for name, arr in w.items():
        if name.startswith("norm"):
            continue
        n = -(-arr.nbytes // bd.PAGE_BYTES)
        tiers = np.ones(n, np.uint8) if host_weights else np.zeros(n, np.uint8)
        mats[name] = bd.boost_place_weights_map(ctx, arr, arr.nbytes, tiers)
    norms = {k: to_dev_u16(v) for k, v in w.items() if k.startswith("norm")}
    need = [(int(L) + 15) // 16 for L in lengths]
    mb = max(need)
    pool = bd.boost_kv_pool_create(ctx, dims.layers, dims.hkv, dims.hd, max(sum(need), 1536), M,
                                   pool_mode, q_heads=dims.hq, max_batch=B,
                                   max_blocks_per_seq=mb)
    rng = np.random.default_rng(kv_seed)
    kc = [[synth.normal_bf16(rng, (int(L) - 1, dims.hkv, dims.hd), 1.0) for L in lengths]
          for _ in range(dims.layers)]
    vc = [[synth.normal_bf16(rng, (int(L) - 1, dims.hkv, dims.hd), 1.0) for L in lengths]
          for _ in range(dims.layers)]
    tables = None
    for l in range(dims.layers):
        # allocate blocks for the full length (the new token's slot included),
        # write the context before it
        if tables is None:
            tables = np.full((B, mb), -1, np.int32)
            for b in range(B):
                tables[b, :need[b]] = bd.boost_kv_alloc(pool, b, need[b])
        fill_pool(bd, ctx, pool, l, [int(L) - 1 for L in lengths], kc[l], vc[l],
                  tables=tables)
    model = DecodeModel(ctx, dims, B, mb, pool, mats, norms)
    return model, pool, mats, tables, kc, vc


def run(model, tokens, lengths, tables):
    import torch
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()
    ids, logits = model.step(dev(tokens), dev(np.asarray(lengths) - 1), dev(lengths),
                             dev(tables), torch.cuda.current_stream().cuda_stream)
    sync()
    return ids.cpu().numpy(), logits.cpu().numpy()


def free(pool, mats):
    for t in mats.values():
        bd.boost_tensor_free(t)
    bd.boost_kv_pool_destroy(pool)


def rms(a):
    return float(np.sqrt(np.mean(np.asarray(a, np.float64) ** 2)))


# Bars of the composed step, relative to the rms of the logits.  A step
# re-rounds about six operands per layer to bf16; where the kernels' fp32
# value and the oracle's fp64 value straddle a rounding boundary (a fraction
# of roughly sqrt(K) * 2^-16 of the elements for a K-term sum) the operand
# differs by one bf16 ulp (2^-8 relative), and these flips propagate.  For
# two layers that is a mean deviation of order 2 * 6 * 2^-8 * sqrt(3e-3)
# ~ 2.5e-3 of the rms, with single elements about ten times that.  Wiring
# errors (wrong buffer, layer, position or residual) give deviations of the
# order of the rms itself.  Each operator separately meets the element-wise
# bar (tests/test_gpu_glue.py, test_gpu_gemv.py, test_gpu_attention.py).
STEP_MEAN_BAR = 5e-3
STEP_MAX_BAR = 5e-2


def check_logits(logits, ref_logits):
    err = np.abs(np.asarray(logits, np.float64) - ref_logits)
    r = rms(ref_logits)
    assert err.mean() <= STEP_MEAN_BAR * r, err.mean() / r
    assert err.max() <= STEP_MAX_BAR * r, err.max() / r


def check_ids(ids, ref_logits):
    ref_ids = ods.argmax_lowest(ref_logits)
    r = rms(ref_logits)
    for b in range(len(ids)):
        if ids[b] != ref_ids[b]:
            # only a near tie (within the logits bar) may pick another index
            assert ref_logits[b, ref_ids[b]] - ref_logits[b, ids[b]] <= STEP_MAX_BAR * r, \
                (b, ids[b], ref_ids[b])


def test_small_model_step_parity_and_invariance(gpu_ctx):
    dims = Dims(layers=2, d=256, hq=4, hkv=2, hd=128, ffn=384, vocab=1000)
    w = model_weights(dims, 3)
    lengths = np.array([1, 17, 300])
    tokens = np.array([5, 999, 0])
    outs = []
    for host_weights, pool_mode in ((False, bd.KV_ALL_HBM), (True, bd.KV_LPP),
                                    (True, bd.KV_ALL_HOST)):
        model, pool, mats, tables, kc, vc = build(gpu_ctx, dims, w, lengths, host_weights,
                                                  pool_mode)
        try:
            outs.append(run(model, tokens, lengths, tables))
        finally:
            free(pool, mats)
    ref_logits, ref_ids, _ = ods.decode_step(w, tokens, kc, vc, lengths, dims.__dict__)
    for ids, logits in outs:
        assert og.rel_err(logits, ref_logits) <= TOL   # short contexts: element-wise bar
        check_logits(logits, ref_logits)
        check_ids(ids, ref_logits)
    for ids, logits in outs[1:]:
        assert np.array_equal(logits.view(np.uint32), outs[0][1].view(np.uint32))
        assert np.array_equal(ids, outs[0][0])


def test_split_projection_fold_matches_reduction(gpu_ctx):
    """A batch of 24 on d = 2048 splits K of the qkv, o and down projections
    over workgroups (down's rows, K = 3072, cross page boundaries); handing
    the slices to the RoPE + KV append and to the residual norms gives the
    same ids and logits, bit for bit, as reducing each projection first, and
    both meet the oracle."""
    dims = Dims(layers=2, d=2048, hq=16, hkv=4, hd=128, ffn=3072, vocab=1000)
    w = model_weights(dims, 8)
    lengths = synth.context_lengths(21, 24, 1, 200)
    tokens = synth.context_lengths(22, 24, 0, dims.vocab - 1)
    model, pool, mats, tables, kc, vc = build(gpu_ctx, dims, w, lengths, True, bd.KV_LPP)
    try:
        assert model.fold
        folded = run(model, tokens, lengths, tables)
        plain = DecodeModel(gpu_ctx, dims, len(lengths), model.mb, pool, mats, model.norms,
                            fold_slices=False)
        assert not plain.fold
        reduced = run(plain, tokens, lengths, tables)
    finally:
        free(pool, mats)
    assert np.array_equal(folded[1].view(np.uint32), reduced[1].view(np.uint32))
    assert np.array_equal(folded[0], reduced[0])
    ref_logits, _, _ = ods.decode_step(w, tokens, kc, vc, lengths, dims.__dict__)
    check_logits(folded[1], ref_logits)
    check_ids(folded[0], ref_logits)


def test_bad_glue_arguments(gpu_ctx):
    import torch
    x = torch.zeros((2, 64), dtype=torch.float32, device="cuda")
    w = torch.zeros(64, dtype=torch.int16, device="cuda")
    o = torch.zeros((2, 64), dtype=torch.int16, device="cuda")
    with pytest.raises(bd.BoostError):
        bd.boost_rmsnorm(gpu_ctx, x, w, 0, 64, 1e-5, o)
    with pytest.raises(bd.BoostError):
        bd.boost_rope_qkv(gpu_ctx, x, x, 1, 1, 1, 63, 500000.0, o, o, o)
    with pytest.raises(bd.BoostError):
        bd.boost_argmax(gpu_ctx, x, 2, 0, w)
    with pytest.raises(bd.BoostError):
        bd.boost_silu_mul(gpu_ctx, x, 2, 0, o)


@pytest.mark.timeout(900)
def test_llama70b_shaped_two_layer_step(gpu_ctx):
    """70B shapes (d 8192, FFN 28672, GQA 64/8, head_dim 128, vocab 128256),
    two layers, batch 8, context 2048; weights placed by MPP at the modulus
    of the 120 GB budget (M = 6, host pages in the large tensors); logits and
    argmax against the oracle."""
    import torch
    dims = Dims(layers=2, d=8192, hq=64, hkv=8, hd=128, ffn=28672, vocab=128256)
    B, L = 8, 2048
    lengths = np.full(B, L)
    tokens = synth.context_lengths(5, B, 0, dims.vocab - 1).astype(np.int64)
    # weights drawn on the device (seeded), copied to the host for the oracle
    w, mats = {}, {}
    for name, N, K, seed in ([("embed", dims.vocab, dims.d, 9998), ("lm_head", dims.vocab, dims.d, 9999)]
                             + [(f"{n}.{l}", N_, K_, 1000 + 10 * l + i)
                                for l in range(dims.layers)
                                for i, (n, N_, K_) in enumerate(dims.shapes())]):
        g = torch.Generator(device="cuda")
        g.manual_seed(seed)
        t = (torch.randn((N, K), generator=g, device="cuda") * (1.0 if name == "embed" else 0.02)
             ).to(torch.bfloat16).view(torch.int16)
        mats[name] = bd.boost_place_weights(gpu_ctx, t, N * K * 2, 6)
        w[name] = t.cpu().numpy().view(np.uint16)
        del t
    rng = np.random.default_rng(4)
    for k in ["norm_f"] + [f"norm{j}.{l}" for l in range(dims.layers) for j in (1, 2)]:
        w[k] = synth.round_bf16((1 + 0.1 * rng.standard_normal(dims.d)).astype(np.float32))
    norms = {k: to_dev_u16(v) for k, v in w.items() if k.startswith("norm")}
    host_pages = sum(int(bd.boost_tensor_tiers(t).sum()) for t in mats.values())
    assert host_pages > 0
    need = L // 16
    pool = bd.boost_kv_pool_create(gpu_ctx, dims.layers, dims.hkv, dims.hd, B * need, 0,
                                   bd.KV_ALL_HBM, q_heads=dims.hq, max_batch=B,
                                   max_blocks_per_seq=need)
    try:
        tables = np.full((B, need), -1, np.int32)
        for b in range(B):
            tables[b] = bd.boost_kv_alloc(pool, b, need)
        kr = np.random.default_rng(12)
        kc = [[synth.normal_bf16(kr, (L - 1, dims.hkv, dims.hd), 1.0) for _ in range(B)]
              for _ in range(dims.layers)]
        vc = [[synth.normal_bf16(kr, (L - 1, dims.hkv, dims.hd), 1.0) for _ in range(B)]
              for _ in range(dims.layers)]
        for l in range(dims.layers):
            fill_pool(bd, gpu_ctx, pool, l, [L - 1] * B, kc[l], vc[l], tables=tables)
        model = DecodeModel(gpu_ctx, dims, B, need, pool, mats, norms)
        ids, logits = run(model, tokens, lengths, tables)
    finally:
        for t in mats.values():
            bd.boost_tensor_free(t)
        bd.boost_kv_pool_destroy(pool)
        torch.cuda.empty_cache()
    ref_logits, _, _ = ods.decode_step(w, tokens, kc, vc, lengths, dims.__dict__)
    check_logits(logits, ref_logits)
    check_ids(ids, ref_logits)
