"""GPU parity of the tiered-page GEMV against the oracle (through the C-ABI)."""
import numpy as np
import pytest

import synth
from oracle import gemv as og
from oracle import placement as opl
from paper_2609_13592_amd import binding as bd
from tests.gpu_util import dev_f32, dev_u16, host_u16, slices_sum, stream, sync, to_dev_u16

pytestmark = pytest.mark.gpu
TOL = 2e-2          # stated bar for bf16 inputs (max rel err)


def assert_f32_bound(y, w, x, rows=None):
    """Internal gate: every output within the worst-case fp32 summation error
    K * 2^-24 * sum_k |w x| of the fp64 result (any summation order)."""
    wf = og.bf16_to_f32(w).astype(np.float64)
    xf = og.bf16_to_f32(x).astype(np.float64)
    ref = xf @ wf.T
    mag = np.abs(xf) @ np.abs(wf).T
    K = wf.shape[1]
    yy = y if rows is None else y[:, rows]
    assert np.all(np.abs(yy - ref) <= K * 2.0 ** -24 * mag + 1e-30)


def run_gemv(ctx, t, N, K, x_dev, B, y_dtype=bd.DTYPE_F32):
    y = dev_f32(B, N) if y_dtype == bd.DTYPE_F32 else dev_u16(B, N)
    bd.boost_decode_gemv(ctx, t, N, K, x_dev, B, y, y_dtype, stream())
    sync()
    return y.cpu().numpy() if y_dtype == bd.DTYPE_F32 else host_u16(y)


def irregular_map(n):
    """Host pages at 0, 3, 5, 8, 10, ... (two per five, unevenly spaced): a map
    with no modulo closed form, so the kernels read the page tables."""
    return ((np.arange(n) * 7) % 5 < 2).astype(np.uint8)


def place(ctx, w, tiers=None, M=None):
    nbytes = w.nbytes
    if tiers is not None:
        return bd.boost_place_weights_map(ctx, w, nbytes, tiers)
    return bd.boost_place_weights(ctx, w, nbytes, M)


def test_calibration(gpu_ctx):
    hbm, host, alpha = bd.boost_calibrate(gpu_ctx, 2 << 30, 512 << 20, 3)
    print(f"calibration: hbm {hbm:.1f} GB/s host {host:.1f} GB/s alpha {alpha:.5f}")
    assert 1000 < hbm < 8200
    assert 2 < host < 200
    assert 0 < alpha < 0.1
    M = bd.boost_modulus_from_alpha(alpha)
    assert M == opl.modulus_from_alpha(alpha)


def test_cap_probe_points(gpu_ctx):
    """The concurrent streaming probe: every layout variant runs, reports rates
    inside the physical range, and rejects points outside its contract."""
    T, H = 256 << 20, 32 << 20
    pts = [dict(hbm_bytes=T, hbm_wgs=1024),
           dict(host_bytes=H, host_wgs=8, host_depth=2),
           dict(hbm_bytes=T - (4 << 20), hbm_wgs=1024, host_bytes=4 << 20, host_wgs=4,
                host_depth=1, host_policy=2),
           dict(hbm_bytes=T - (4 << 20), hbm_wgs=1024, host_bytes=4 << 20, host_wgs=4,
                host_stride=8, host_policy=1),
           dict(hbm_bytes=T - (4 << 20), hbm_wgs=1024, host_bytes=4 << 20, dma=1),
           dict(hbm_bytes=T - (4 << 20) - 16, hbm_wgs=1020, host_bytes=4 << 20, host_wgs=4,
                host_stride=8, hbm_chunk_kib=256),
           dict(hbm_bytes=T, hbm_wgs=3000, hbm_chunk_kib=64),
           dict(hbm_bytes=T - 16, hbm_wgs=1000, hbm_chunk_kib=256, chunk_static=1),
           dict(hbm_bytes=T - 16, hbm_wgs=1000, host_bytes=4 << 20, host_wgs=8,
                hbm_chunk_kib=256, chunk_static=2),
           dict(hbm_bytes=T - (4 << 20) - 16, hbm_wgs=240, host_bytes=4 << 20, host_wgs=16,
                host_stride=8, hbm_chunk_kib=64, chunk_static=3)]
    r = bd.boost_cap_sweep(gpu_ctx, T, H, pts, 2)
    assert r.shape == (10, 16)
    assert 500 < r[7, 2] < 9000 and 500 < r[8, 2] < 9000 and 1 < r[8, 3] < 200
    # round robin on compute units of their own, host workgroups on one XCD
    assert 500 < r[9, 2] < 9000 and 1 < r[9, 3] < 200
    # queue-fed HBM workers (a ragged last chunk; more workers than slots)
    assert 500 < r[5, 2] < 9000 and 1 < r[5, 3] < 200
    assert 500 < r[6, 2] < 9000
    # every XCD ran HBM workgroups, none ended after the last one
    assert np.all(r[0, 8:16] > 0) and np.all(r[0, 8:16] <= r[0, 7] + 1e-6)
    assert 500 < r[0, 2] < 9000 and r[0, 3] == 0
    assert 1 < r[1, 3] < 200 and r[1, 2] == 0
    for i in (2, 3):
        assert 500 < r[i, 2] < 9000 and 1 < r[i, 3] < 200
        assert 0 < r[i, 5] <= r[i, 7] <= r[i, 4] + 1e-6
    assert r[4, 6] > 0 and 1 < r[4, 3] < 200
    for bad in (dict(hbm_bytes=T, hbm_wgs=16, host_depth=3),
                dict(hbm_bytes=T, hbm_wgs=16, hbm_chunk_kib=6),
                dict(hbm_bytes=T, hbm_wgs=16, hbm_chunk_kib=64, chunk_static=4),
                dict(hbm_bytes=T, hbm_wgs=16, chunk_static=1),
                dict(hbm_bytes=T, hbm_wgs=16, hbm_chunk_kib=64, chunk_static=3, host_depth=2),
                dict(hbm_bytes=T, hbm_wgs=16, host_bytes=H, host_wgs=1, dma=1),
                dict(hbm_bytes=T + 16, hbm_wgs=16),
                dict(hbm_bytes=T, hbm_wgs=4, host_bytes=H, host_wgs=2, host_stride=8),
                dict(host_bytes=H, host_wgs=0)):
        with pytest.raises(bd.BoostError) as e:
            bd.boost_cap_sweep(gpu_ctx, T, H, [bad], 1)
        assert e.value.code == bd.EINVAL


def test_single_layer_parity(gpu_ctx):
    """4096 x 4096 bf16 layer, 16 pages, page 15 on host (M = 16)."""
    w, x = synth.single_layer_inputs()
    t = place(gpu_ctx, w, M=16)
    try:
        tiers = bd.boost_tensor_tiers(t)
        assert np.array_equal(tiers, opl.mpp_tier_map(w.nbytes, 16))
        assert np.flatnonzero(tiers).tolist() == [15]
        # bytes of the host page and of an HBM page read back unchanged
        for page in (0, 15):
            got = bd.boost_tensor_read(t, page * opl.PAGE, opl.PAGE)
            assert np.array_equal(got, w.view(np.uint8).reshape(-1)[
                page * opl.PAGE:(page + 1) * opl.PAGE])
        xd = to_dev_u16(x)
        r64, r32 = og.gemv_f64(w, x), og.gemv_f32(w, x)
        for sched in (bd.SCHED_CAP, bd.SCHED_ADDRESS):
            bd.boost_gemv_set_schedule(gpu_ctx, sched)
            y = run_gemv(gpu_ctx, t, 4096, 4096, xd, 1)
            assert og.rel_err(y, r64) <= TOL
            assert og.rel_err(y, r32) <= TOL
            assert_f32_bound(y, w, x)
    finally:
        bd.boost_gemv_set_schedule(gpu_ctx, bd.SCHED_CAP)
        bd.boost_tensor_free(t)


@pytest.mark.parametrize("N,K,B", [(4096, 4096, 1), (300, 14336, 1), (5000, 520, 3),
                                   (1000, 8, 8), (257, 4104, 2), (77, 28672, 5)])
def test_placement_invariance_and_parity(gpu_ctx, N, K, B):
    """Bitwise-equal y under all-HBM, alternating, MPP and all-host maps, both
    schedules and any number of host workers; every result within the bar
    of the oracle."""
    w, x = synth.gemv_inputs(11 + N + K + B, N, K, B)
    n = opl.n_pages(w.nbytes)
    maps = {"hbm": np.zeros(n, np.uint8), "host": np.ones(n, np.uint8),
            "alt": (np.arange(n) % 2).astype(np.uint8),
            "mpp3": opl.mpp_tier_map(w.nbytes, 3), "irregular": irregular_map(n)}
    xd = to_dev_u16(x)
    r64 = og.gemv_f64(w, x)
    r32 = og.gemv_f32(w, x)
    outs = []
    for name, tiers in maps.items():
        t = place(gpu_ctx, w, tiers=tiers)
        try:
            # CAP with 3 host workers, with the default count, and with more
            # workers than host units; address order
            for sched, hw in ((bd.SCHED_CAP, 3), (bd.SCHED_CAP, 0), (bd.SCHED_CAP, 999),
                              (bd.SCHED_ADDRESS, 0)):
                bd.boost_gemv_set_schedule(gpu_ctx, sched, hw)
                y = run_gemv(gpu_ctx, t, N, K, xd, B)
                assert og.rel_err(y, r64) <= TOL, (name, sched)
                assert og.rel_err(y, r32) <= TOL, (name, sched)
                assert_f32_bound(y, w, x)
                outs.append(y)
        finally:
            bd.boost_gemv_set_schedule(gpu_ctx, bd.SCHED_CAP)
            bd.boost_tensor_free(t)
    for y in outs[1:]:
        assert np.array_equal(y.view(np.uint32), outs[0].view(np.uint32))


@pytest.mark.parametrize("N,K,B", [(300, 14336, 7), (5000, 520, 16), (2400, 14336, 12),
                                   (257, 4104, 20),
                                   (257, 4104, 33), (77, 28672, 64), (300, 14336, 64),
                                   (1000, 8, 100), (600, 4096, 128), (300, 14336, 128),
                                   (130, 14336, 256), (40, 56, 200)])
def test_mfma_placement_invariance_and_parity(gpu_ctx, N, K, B):
    """Batches from 7 up run on the matrix cores: bitwise-equal y under every
    map and schedule, every result within the bar of the oracle (ragged
    batch tiles, rows cut by page boundaries, pages of both tiers).  Up to
    B = 16 one batch tile with weights staged through LDS, in one row tile
    or (B = 12 on a matrix of 2^25 elements) two.  From B = 17 the GEMM
    covers 2, 4, 8 and 16 batch tiles with 64-row units (B = 20, 33, 64,
    100, 128, 200) and 128-row units (K = 14336 at B = 64, 128 and 256, on
    eight wavefronts), each with its own wavefront grid, and the host pages
    of the "host", "alt" and "mpp3" maps run as 16-row sub-units: the
    bitwise comparison across maps checks that they sum in the same
    order."""
    w, x = synth.gemv_inputs(17 + N + K + B, N, K, B)
    n = opl.n_pages(w.nbytes)
    maps = {"hbm": np.zeros(n, np.uint8), "host": np.ones(n, np.uint8),
            "alt": (np.arange(n) % 2).astype(np.uint8),
            "mpp3": opl.mpp_tier_map(w.nbytes, 3), "irregular": irregular_map(n)}
    xd = to_dev_u16(x)
    r64 = og.gemv_f64(w, x)
    outs = []
    for name, tiers in maps.items():
        t = place(gpu_ctx, w, tiers=tiers)
        try:
            # CAP with 3 host workers, with the default count, and with more
            # workers than host units; address order
            for sched, hw in ((bd.SCHED_CAP, 3), (bd.SCHED_CAP, 0), (bd.SCHED_CAP, 999),
                              (bd.SCHED_ADDRESS, 0)):
                bd.boost_gemv_set_schedule(gpu_ctx, sched, hw)
                y = run_gemv(gpu_ctx, t, N, K, xd, B)
                assert og.rel_err(y, r64) <= TOL, (name, sched)
                assert_f32_bound(y, w, x)
                outs.append(y)
        finally:
            bd.boost_gemv_set_schedule(gpu_ctx, bd.SCHED_CAP)
            bd.boost_tensor_free(t)
    for y in outs[1:]:
        assert np.array_equal(y.view(np.uint32), outs[0].view(np.uint32))


@pytest.mark.parametrize("B", [9, 16, 256])
def test_mfma_exact_pins(gpu_ctx, B):
    """W = I gives x back exactly on the matrix-core path; bf16 output of it
    is x's bits."""
    n = 1024
    eye = synth.round_bf16(np.eye(n, dtype=np.float32))
    rng = np.random.default_rng(B)
    x = synth.normal_bf16(rng, (B, n), 1.0)
    t = place(gpu_ctx, eye, tiers=(np.arange(opl.n_pages(eye.nbytes)) % 2).astype(np.uint8))
    try:
        xd = to_dev_u16(x)
        assert np.array_equal(run_gemv(gpu_ctx, t, n, n, xd, B), og.bf16_to_f32(x))
        assert np.array_equal(run_gemv(gpu_ctx, t, n, n, xd, B, bd.DTYPE_BF16), x)
    finally:
        bd.boost_tensor_free(t)


def test_exact_pins(gpu_ctx):
    """W = I gives x back, all-ones gives K: exact in fp32."""
    n = 1024
    eye = synth.round_bf16(np.eye(n, dtype=np.float32))
    rng = np.random.default_rng(5)
    x = synth.normal_bf16(rng, (2, n), 1.0)
    t = place(gpu_ctx, eye, tiers=(np.arange(opl.n_pages(eye.nbytes)) % 2).astype(np.uint8))
    try:
        y = run_gemv(gpu_ctx, t, n, n, to_dev_u16(x), 2)
        assert np.array_equal(y, og.bf16_to_f32(x))
    finally:
        bd.boost_tensor_free(t)
    K = 4096
    ones = synth.round_bf16(np.ones((520, K), np.float32))
    t = place(gpu_ctx, ones, M=2)
    try:
        y = run_gemv(gpu_ctx, t, 520, K, to_dev_u16(ones[:1]), 1)
        assert np.all(y == K)
    finally:
        bd.boost_tensor_free(t)


def test_bf16_output(gpu_ctx):
    N, K = 2000, 4096
    w, x = synth.gemv_inputs(21, N, K, 2)
    t = place(gpu_ctx, w, M=3)
    try:
        xd = to_dev_u16(x)
        yb = run_gemv(gpu_ctx, t, N, K, xd, 2, bd.DTYPE_BF16)
        yf = run_gemv(gpu_ctx, t, N, K, xd, 2, bd.DTYPE_F32)
        assert og.rel_err(og.bf16_to_f32(yb), og.gemv_f64(w, x)) <= TOL
        # bf16 output is the round-to-nearest-even of the fp32 result
        assert np.array_equal(yb, og.f32_to_bf16(yf))
    finally:
        bd.boost_tensor_free(t)


def test_bad_arguments(gpu_ctx):
    w, x = synth.gemv_inputs(1, 64, 512, 1)
    t = place(gpu_ctx, w, M=2)
    xd = to_dev_u16(x)
    y = dev_f32(257, 64)
    try:
        for args in ((64, 520, 1), (63, 512, 1), (64, 512, 257), (64, 512, 0)):
            N, K, B = args
            with pytest.raises(bd.BoostError) as e:
                bd.boost_decode_gemv(gpu_ctx, t, N, K, xd, B, y, bd.DTYPE_F32, stream())
            assert e.value.code == bd.EINVAL
        with pytest.raises(bd.BoostError):
            bd.boost_decode_gemv(gpu_ctx, t, 64, 512, xd, 1, y, 7, stream())
    finally:
        bd.boost_tensor_free(t)


@pytest.mark.parametrize("kind,B", [(0, 1), (1, 1), (2, 1), (3, 1), (9, 1),
                                    (0, 256), (3, 256), (2, 64)])
def test_full_size_chain_tensor_sampled(gpu_ctx, kind, B):
    """Full-size Llama-3-8B-shaped tensors (fused qkv, o, gate_up, down,
    lm_head) placed by MPP at M = 11, at batch 1 (GEMV) and at the
    high-throughput batches (matrix cores): sampled rows against the oracle."""
    import torch
    per_layer, head = synth.chain_shapes(synth.LLAMA8B)
    shapes = {k: (n, kk) for _, k, n, kk in per_layer}
    shapes[9] = head[2:]
    N, K = shapes[kind]
    wt = synth.chain_weight_torch(3, kind, N, K, "cuda")
    w_dev = wt.view(torch.int16)
    rng = np.random.default_rng(kind)
    x = synth.normal_bf16(rng, (B, K), 1.0)
    t = bd.boost_place_weights(gpu_ctx, w_dev, N * K * 2, 11)
    try:
        tiers = bd.boost_tensor_tiers(t)
        assert np.array_equal(tiers, opl.mpp_tier_map(N * K * 2, 11))
        y = run_gemv(gpu_ctx, t, N, K, to_dev_u16(x), B)
        rows = np.unique(np.concatenate([rng.integers(0, N, 200), [0, N - 1],
                                         (np.arange(0, N * K, opl.PAGE // 2) // K)]))
        w_rows = w_dev[torch.from_numpy(rows).cuda()].cpu().numpy().view(np.uint16)
        ref = og.gemv_rows_f64(w_rows, rows, x)
        assert og.rel_err(y[:, rows], ref) <= TOL
        assert_f32_bound(y, w_rows, x, rows)
    finally:
        bd.boost_tensor_free(t)
        del wt, w_dev
        torch.cuda.empty_cache()


def test_prefetch_staged_view(gpu_ctx):
    """The prefetch baseline's staged view reads the copied host pages from
    HBM staging and gives the same bits as the tiered tensor."""
    import torch
    N, K = 3000, 4096
    w, x = synth.gemv_inputs(31, N, K, 1)
    t = place(gpu_ctx, w, M=2)
    n_host = int(bd.boost_tensor_tiers(t).sum())
    staging = torch.empty(n_host * opl.PAGE, dtype=torch.uint8, device="cuda")
    v = bd.boost_staged_view(gpu_ctx, t, staging, staging.numel())
    try:
        assert not bd.boost_tensor_tiers(v).any()
        assert bd.boost_tensor_layout(v)[0] == -1  # staged pages: no closed form
        xd = to_dev_u16(x)
        bd.boost_prefetch(gpu_ctx, v, stream())
        yv = run_gemv(gpu_ctx, v, N, K, xd, 1)
        yt = run_gemv(gpu_ctx, t, N, K, xd, 1)
        assert np.array_equal(yv.view(np.uint32), yt.view(np.uint32))
        assert og.rel_err(yv, og.gemv_f64(w, x)) <= TOL
        with pytest.raises(bd.BoostError):
            bd.boost_staged_view(gpu_ctx, t, staging, staging.numel() - 16)
        with pytest.raises(bd.BoostError):
            bd.boost_prefetch(gpu_ctx, t, stream())
    finally:
        bd.boost_tensor_free(v)
        bd.boost_tensor_free(t)


@pytest.mark.parametrize("kind", [0, 1, 2, 3, 9])
def test_full_size_70b_tensor_sampled_batch8(gpu_ctx, kind):
    """Full-size Llama-3-70B-shaped tensors (fused qkv 10240 x 8192, o
    8192 x 8192, fused gate_up 57344 x 8192, down 8192 x 28672, lm_head
    128256 x 8192: 80 to 1002 pages) placed by MPP at M = 6, the modulus of
    the 120e9-byte HBM weight budget, at batch 8: the matrix-core kernel with
    weights staged through LDS, one K slice, many host units per CAP worker,
    and (down) rows cut by page boundaries through split_fixup.  Sampled rows,
    including every row a page boundary cuts, element by element against the
    oracle at the stated bar and within the fp32 summation bound."""
    import torch
    per_layer, head = synth.chain_shapes(synth.LLAMA70B)
    shapes = {k: (n, kk) for _, k, n, kk in per_layer}
    shapes[9] = head[2:]
    N, K = shapes[kind]
    B = 8
    wt = synth.chain_weight_torch(5, kind, N, K, "cuda")
    w_dev = wt.view(torch.int16)
    rng = np.random.default_rng(70 + kind)
    x = synth.normal_bf16(rng, (B, K), 1.0)
    t = bd.boost_place_weights(gpu_ctx, w_dev, N * K * 2, 6)
    try:
        tiers = bd.boost_tensor_tiers(t)
        assert np.array_equal(tiers, opl.mpp_tier_map(N * K * 2, 6))
        assert tiers.sum() == len(tiers) // 6
        y = run_gemv(gpu_ctx, t, N, K, to_dev_u16(x), B)
        cut = np.arange(0, N * K, opl.PAGE // 2) // K        # row at each page start
        rows = np.unique(np.concatenate([rng.integers(0, N, 300), [0, N - 1], cut]))
        w_rows = w_dev[torch.from_numpy(rows).cuda()].cpu().numpy().view(np.uint16)
        ref = og.gemv_rows_f64(w_rows, rows, x)
        assert og.rel_err(y[:, rows], ref) <= TOL
        assert_f32_bound(y, w_rows, x, rows)
        assert np.all(np.isfinite(y))
    finally:
        bd.boost_tensor_free(t)
        del wt, w_dev
        torch.cuda.empty_cache()


@pytest.mark.parametrize("N,K,B,split", [(6144, 4096, 64, True), (4096, 4096, 64, True),
                                         (128, 16384, 64, True), (600, 4096, 128, None),
                                         (3072, 2048, 24, True), (2048, 2048, 24, True),
                                         (300, 2048, 3, False), (1000, 8, 100, None),
                                         (4096, 14336, 64, True), (2048, 3072, 24, True),
                                         (300, 14336, 7, None), (130, 14336, 256, None)])
def test_slices_sum_to_y(gpu_ctx, N, K, B, split):
    """The slices entry point writes split-K partials (and the parts of rows
    cut by page boundaries) whose sum, in the order the header states, is
    boost_decode_gemv's y bit for bit, under the HBM, alternating and MPP
    maps; caps of one and two slices give a y within the oracle's bar.
    `split` says whether the shape must split (None: either)."""
    w, x = synth.gemv_inputs(91 + N + K + B, N, K, B)
    n = opl.n_pages(w.nbytes)
    maps = {"hbm": np.zeros(n, np.uint8), "alt": (np.arange(n) % 2).astype(np.uint8),
            "mpp3": opl.mpp_tier_map(w.nbytes, 3)}
    xd = to_dev_u16(x)
    r64 = og.gemv_f64(w, x)
    size = bd.boost_gemv_slices_floats(N, K, B, bd.MAX_GEMV_SLICES)
    ys = []
    for name, tiers in maps.items():
        t = place(gpu_ctx, w, tiers=tiers)
        try:
            y = run_gemv(gpu_ctx, t, N, K, xd, B)
            sl = dev_f32(size)
            sl.fill_(float("nan"))  # the unwritten entries must not reach y
            S = bd.boost_decode_gemv_slices(gpu_ctx, t, N, K, xd, B, sl, bd.MAX_GEMV_SLICES,
                                            stream())
            sync()
            assert 1 <= S <= bd.MAX_GEMV_SLICES
            if split is not None:
                assert (S > 1) == split, (name, S)
            got = slices_sum(sl.cpu().numpy(), S, B, N, K)
            assert np.array_equal(got.view(np.uint32), y.view(np.uint32)), name
            ys.append(y)
            for cap in (1, 2):
                sl.fill_(float("nan"))
                S2 = bd.boost_decode_gemv_slices(gpu_ctx, t, N, K, xd, B, sl, cap, stream())
                sync()
                assert 1 <= S2 <= cap
                y2 = slices_sum(sl.cpu().numpy(), S2, B, N, K)
                assert og.rel_err(y2, r64) <= TOL, (name, cap)
                assert_f32_bound(y2, w, x)
        finally:
            bd.boost_tensor_free(t)
    assert og.rel_err(ys[0], r64) <= TOL
    for y in ys[1:]:
        assert np.array_equal(y.view(np.uint32), ys[0].view(np.uint32))


def test_slices_calls_on_two_streams(gpu_ctx):
    """The slices entry point keeps its partials in the caller's buffer (the
    context's split-K workspace is not touched), so calls on two streams may
    overlap: two split shapes under MPP maps, each called five times on its
    own stream with the other's calls interleaved, sum to the serial
    boost_decode_gemv results bit for bit."""
    import torch
    B = 64
    shapes = [(6144, 4096), (4096, 14336)]
    size = max(bd.boost_gemv_slices_floats(N, K, B, bd.MAX_GEMV_SLICES) for N, K in shapes)
    ts, xs, ys, bufs = [], [], [], []
    try:
        for i, (N, K) in enumerate(shapes):
            w, x = synth.gemv_inputs(501 + i, N, K, B)
            t = place(gpu_ctx, w, tiers=opl.mpp_tier_map(w.nbytes, 3))
            ts.append(t)
            xs.append(to_dev_u16(x))
            ys.append(run_gemv(gpu_ctx, t, N, K, xs[-1], B))
            bufs.append([dev_f32(size) for _ in range(5)])
        torch.cuda.synchronize()
        streams = [torch.cuda.Stream(), torch.cuda.Stream()]
        S = [[0] * 5, [0] * 5]
        for r in range(5):
            for i, (N, K) in enumerate(shapes):
                S[i][r] = bd.boost_decode_gemv_slices(gpu_ctx, ts[i], N, K, xs[i], B, bufs[i][r],
                                                      bd.MAX_GEMV_SLICES,
                                                      streams[i].cuda_stream)
        torch.cuda.synchronize()
        for i, (N, K) in enumerate(shapes):
            for r in range(5):
                assert S[i][r] > 1, (N, K)
                got = slices_sum(bufs[i][r].cpu().numpy(), S[i][r], B, N, K)
                assert np.array_equal(got.view(np.uint32), ys[i].view(np.uint32)), (N, K, r)
    finally:
        for t in ts:
            bd.boost_tensor_free(t)


def test_slices_bad_arguments(gpu_ctx):
    """Slice caps outside [1, 8] and misaligned buffers are refused before
    anything runs."""
    w, x = synth.gemv_inputs(3, 256, 4096, 64)
    t = place(gpu_ctx, w, M=3)
    xd = to_dev_u16(x)
    sl = dev_f32(bd.boost_gemv_slices_floats(256, 4096, 64, bd.MAX_GEMV_SLICES) + 4)
    try:
        for cap in (0, bd.MAX_GEMV_SLICES + 1):
            with pytest.raises(bd.BoostError) as e:
                bd.boost_decode_gemv_slices(gpu_ctx, t, 256, 4096, xd, 64, sl, cap, stream())
            assert e.value.code == bd.EINVAL
        with pytest.raises(bd.BoostError) as e:
            bd.boost_decode_gemv_slices(gpu_ctx, t, 256, 4096, xd, 64, sl[1:], 8, stream())
        assert e.value.code == bd.EINVAL
    finally:
        bd.boost_tensor_free(t)


def test_host_pages_bound_to_a_numa_node(gpu_ctx):
    """Host pages pinned under a policy bound to node 0 (present on every
    host) serve the GEMV with the same bits as HIP's default node."""
    w, x = synth.gemv_inputs(5, 1024, 4096, 2)
    tiers = (np.arange(opl.n_pages(w.nbytes)) % 2).astype(np.uint8)
    xd = to_dev_u16(x)
    info = bd.boost_host_numa_info(gpu_ctx)
    assert info["n_nodes"] >= 1 and info["node"] == bd.NUMA_DEVICE
    assert info["device_node"] >= -1
    ys = []
    try:
        for node in (0, bd.NUMA_DEVICE):
            bd.boost_set_host_numa(gpu_ctx, node)
            t = place(gpu_ctx, w, tiers=tiers)
            try:
                assert int(bd.boost_tensor_tiers(t).sum()) == int(tiers.sum())
                ys.append(run_gemv(gpu_ctx, t, 1024, 4096, xd, 2))
            finally:
                bd.boost_tensor_free(t)
    finally:
        bd.boost_set_host_numa(gpu_ctx, bd.NUMA_DEVICE)
    assert og.rel_err(ys[0], og.gemv_f64(w, x)) <= TOL
    assert np.array_equal(ys[0].view(np.uint32), ys[1].view(np.uint32))


def test_closed_form_layouts(gpu_ctx):
    """Modulo maps get the closed form the kernels compute pages from (all
    HBM, all host, alternating, MPP with and without superpages); an
    irregular map and a staged view keep the tables; the GEMV gives the same
    bits either way."""
    w, x = synth.gemv_inputs(8, 2048, 4096, 3)   # 8 pages
    n = opl.n_pages(w.nbytes)
    xd = to_dev_u16(x)
    cases = [(np.zeros(n, np.uint8), (0, 1)), (np.ones(n, np.uint8), (1, n)),
             ((np.arange(n) % 2).astype(np.uint8), (2, 1)),
             (((np.arange(n) // 2) % 3 == 2).astype(np.uint8), (3, 2)),
             (irregular_map(n), (-1, 1))]
    ys = []
    for tiers, want in cases:
        t = place(gpu_ctx, w, tiers=tiers)
        try:
            assert bd.boost_tensor_layout(t) == want, (tiers, want)
            ys.append(run_gemv(gpu_ctx, t, 2048, 4096, xd, 3))
        finally:
            bd.boost_tensor_free(t)
    t = place(gpu_ctx, w, M=4)
    try:
        M, SP = bd.boost_tensor_layout(t)
        assert M == 4 or bd.boost_tensor_tiers(t).sum() == 0
    finally:
        bd.boost_tensor_free(t)
    for y in ys[1:]:
        assert np.array_equal(y.view(np.uint32), ys[0].view(np.uint32))
