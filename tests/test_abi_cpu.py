"""C-ABI checks that need no GPU: the library loads, exports every symbol the
headers declare, and its CPU-only planners match the oracle bit for bit."""
import glob
import os
import re

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import placement as opl
from paper_2609_13592_amd import binding as bd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        src = open(h).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        for m in re.finditer(r"\b(boost_[a-z0-9_]+)\s*\(", src):
            names.add(m.group(1))
    return sorted(names)


def test_library_loads_and_exports_every_declared_symbol():
    lib = bd.load()
    names = declared_symbols()
    assert len(names) >= 15
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing
    assert bd.boost_version() >= 100


def test_plan_only_context():
    ctx = bd.boost_init(-1)
    assert bd.boost_ctx_info(ctx) == (-1, 0)
    with pytest.raises(bd.BoostError) as e:
        bd.boost_place_weights(ctx, np.zeros(16, np.uint8), 16, 4)
    assert e.value.code == bd.ENODEV
    bd.boost_shutdown(ctx)


def _online_nodes():
    """Node ids listed in /sys/devices/system/node/online ("0", "0-3", "0,2")."""
    try:
        txt = open("/sys/devices/system/node/online").read().strip()
    except OSError:
        return [0]
    ids = []
    for part in txt.split(","):
        lo, _, hi = part.partition("-")
        ids += list(range(int(lo), int(hi or lo) + 1))
    return ids


def test_host_numa_setting():
    """The host-tier NUMA node: HIP's choice by default, any online node on
    request, anything else refused; a plan-only context has no device node."""
    ctx = bd.boost_init(-1)
    try:
        nodes = _online_nodes()
        info = bd.boost_host_numa_info(ctx)
        assert info == {"device_node": -1, "n_nodes": len(nodes), "node": bd.NUMA_DEVICE}
        for n in nodes:
            bd.boost_set_host_numa(ctx, n)
            assert bd.boost_host_numa_info(ctx)["node"] == n
        for bad in (-2, max(nodes) + 1, 5000):
            with pytest.raises(bd.BoostError) as e:
                bd.boost_set_host_numa(ctx, bad)
            assert e.value.code == bd.EINVAL
        assert bd.boost_host_numa_info(ctx)["node"] == nodes[-1]
        bd.boost_set_host_numa(ctx, bd.NUMA_DEVICE)
        assert bd.boost_host_numa_info(ctx)["node"] == bd.NUMA_DEVICE
    finally:
        bd.boost_shutdown(ctx)


def test_gemv_slices_floats():
    """Slice buffer size: max_slices * B * (N + 2 (pages + 1)) floats, pages of
    2^20 bf16 elements of the [N, K] matrix (the 8B o and down matrices)."""
    assert bd.boost_gemv_slices_floats(4096, 4096, 64, 8) == 8 * 64 * (4096 + 2 * 17)
    assert bd.boost_gemv_slices_floats(4096, 14336, 64, 4) == 4 * 64 * (4096 + 2 * 57)
    assert bd.boost_gemv_slices_floats(3, 8, 1, 1) == 1 * (3 + 2 * 2)
    for bad in ((0, 8, 1, 1), (8, 0, 1, 1), (8, 8, 0, 1), (8, 8, 1, 0)):
        with pytest.raises(bd.BoostError) as e:
            bd.boost_gemv_slices_floats(*bad)
        assert e.value.code == bd.EINVAL


def test_cap_sweep_needs_a_device():
    ctx = bd.boost_init(-1)
    try:
        with pytest.raises(bd.BoostError) as e:
            bd.boost_cap_sweep(ctx, 1 << 20, 1 << 20,
                               [dict(hbm_bytes=1 << 20, hbm_wgs=4)], 1)
        assert e.value.code == bd.ENODEV
    finally:
        bd.boost_shutdown(ctx)


def test_bad_arguments():
    for bad in (0.0, -1.0, 1.5):
        with pytest.raises(bd.BoostError) as e:
            bd.boost_modulus_from_alpha(bad)
        assert e.value.code == bd.EINVAL
    with pytest.raises(bd.BoostError):
        bd.boost_plan_mpp(0, 4)
    with pytest.raises(bd.BoostError):
        bd.boost_plan_mpp(100, 1)
    with pytest.raises(bd.BoostError) as e:
        bd.boost_init(-2)
    assert e.value.code == bd.EINVAL


@given(st.floats(min_value=1e-4, max_value=1.0, allow_nan=False))
@settings(max_examples=400, deadline=None)
def test_modulus_matches_oracle(alpha):
    assert bd.boost_modulus_from_alpha(alpha) == opl.modulus_from_alpha(alpha)


def test_modulus_paper_values():
    assert bd.boost_modulus_from_alpha(0.1) == 11
    assert bd.boost_modulus_from_alpha(350 / 3330) == 11


@given(st.integers(1, 300 * opl.PAGE), st.integers(2, 40),
       st.sampled_from([0, 1, 4096, 28672 * 128, 3 * 1024 * 1024,
                        7 * 1024 * 1024, opl.PAGE, 5 * opl.PAGE]))
@settings(max_examples=300, deadline=None)
def test_plan_mpp_matches_oracle(nbytes, M, footprint):
    got = bd.boost_plan_mpp(nbytes, M, footprint)
    exp = opl.mpp_tier_map(nbytes, M, footprint)
    assert np.array_equal(got, exp)
    assert bd.boost_superpage_pages(footprint) == opl.superpage_pages(footprint)


def test_plan_mpp_exhaustive_small():
    for n in range(1, 65):
        for M in range(2, 17):
            assert np.array_equal(bd.boost_plan_mpp(n * opl.PAGE, M),
                                  opl.mpp_tier_map(n * opl.PAGE, M))


@given(st.lists(st.integers(1, 200), min_size=1, max_size=10),
       st.floats(0.3, 1.05), st.integers(2, 300))
@settings(max_examples=200, deadline=None)
def test_budget_modulus_matches_oracle(pages, frac, M_alpha):
    sizes = [p * opl.PAGE - 123 for p in pages]
    budget = int(sum(pages) * frac) * opl.PAGE
    try:
        exp = opl.modulus_from_budget(sizes, budget, M_alpha)
    except MemoryError:
        with pytest.raises(bd.BoostError) as e:
            bd.boost_modulus_from_budget(sizes, budget, M_alpha)
        assert e.value.code == bd.ENOMEM
        return
    assert bd.boost_modulus_from_budget(sizes, budget, M_alpha) == exp


def test_budget_modulus_70b_chain():
    d, f, v = 8192, 28672, 128256
    per_layer = [(64 + 16) * 128 * d * 2, d * 64 * 128 * 2, 2 * f * d * 2, d * f * 2]
    sizes = per_layer * 80 + [v * d * 2] * 2
    assert bd.boost_modulus_from_budget(sizes, 120 * 10 ** 9, 10 ** 6) == 6


@given(st.integers(1, 300 * opl.PAGE), st.integers(2, 200), st.integers(0, 10 ** 6),
       st.integers(0, 2 ** 31))
@settings(max_examples=300, deadline=None)
def test_plan_contrast_matches_oracle(nbytes, M, phase, seed):
    import synth
    n = opl.n_pages(nbytes)
    u = synth.uniforms(seed, n)
    assert np.array_equal(bd.boost_plan_contrast(bd.PLACE_MPP, nbytes, M),
                          opl.mpp_tier_map(nbytes, M))
    assert np.array_equal(bd.boost_plan_contrast(bd.PLACE_MPP_GLOBAL, nbytes, M, phase),
                          opl.mpp_global_map(n, M, phase))
    assert np.array_equal(bd.boost_plan_contrast(bd.PLACE_LINEAR, nbytes, M),
                          opl.linear_map(n, M))
    assert np.array_equal(bd.boost_plan_contrast(bd.PLACE_RANDOM, nbytes, M, 0, u),
                          opl.bapp_r_from_uniforms(u, M))


def test_plan_contrast_random_boundary_draws():
    """Draws exactly at k / M decide the same way on both sides."""
    M = 12
    u = np.array([0.0, 1 / M, np.nextafter(1 / M, 0), np.nextafter(1 / M, 1), 0.5,
                  np.nextafter(1.0, 0)])
    got = bd.boost_plan_contrast(bd.PLACE_RANDOM, u.size * opl.PAGE, M, 0, u)
    assert np.array_equal(got, opl.bapp_r_from_uniforms(u, M))


def test_plan_contrast_bad_arguments():
    for args in ((9, opl.PAGE, 4), (bd.PLACE_MPP, 0, 4), (bd.PLACE_LINEAR, opl.PAGE, 1)):
        with pytest.raises(bd.BoostError) as e:
            bd.boost_plan_contrast(*args)
        assert e.value.code == bd.EINVAL
    with pytest.raises(bd.BoostError):
        bd.boost_plan_contrast(bd.PLACE_RANDOM, opl.PAGE, 4)
    with pytest.raises(ValueError):
        bd.boost_plan_contrast(bd.PLACE_RANDOM, 3 * opl.PAGE, 4, 0, np.zeros(2))
