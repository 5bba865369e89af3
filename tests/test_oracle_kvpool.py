"""Pins of the KV pool geometry (C4) and the DSR allocator (C5)."""
import itertools
import json
import os

import numpy as np
import pytest

from oracle import kvpool as kv

HERE = os.path.dirname(__file__)
GOLD = json.load(open(os.path.join(HERE, "golden", "paper_pins.json")))
WORKED = json.load(open(os.path.join(HERE, "golden", "dsr_worked_example.json")))


def test_shh_to_local_ratio_and_share():
    """§4.3: SHH and all-local blocks in the ratio H : (M - H) put 1/M of the
    KV bytes on host; with H = 4 and M = 12 that is 1 : 2 and 8.3%."""
    g = GOLD["dsr_qwen3_30b"]
    H, M = g["H"], g["M"]
    geom = kv.kv_geometry(512 * 3 * 5, H, 128, M)
    shh, loc = kv.block_lists(geom)
    a, b = g["shh_to_local"]
    assert len(shh) * b == len(loc) * a
    share = geom.host_heads.sum() / (H * geom.nb_pool)
    assert abs(share - 1.0 / M) < 1e-12 and abs(share - g["host_share"]) < 1e-9
    # worst case: a request made only of SHH blocks has 1/H of its KV on host
    assert geom.host_heads[shh].sum() / (H * len(shh)) == g["worst_case"]


@pytest.mark.parametrize("nb_req,H,D,M", [(9250, 8, 128, 111), (1, 8, 128, 2),
                                           (513, 4, 128, 12), (20000, 8, 64, 3),
                                           (3000, 2, 128, 40), (4096, 8, 128, 5)])
def test_geometry_closed_forms(nb_req, H, D, M):
    geom = kv.kv_geometry(nb_req, H, D, M)
    bpp = kv.PAGE // (16 * D * 2)
    assert geom.blocks_per_page == bpp
    assert geom.nb_pool % bpp == 0 and geom.nb_pool >= nb_req
    assert geom.nb_pool - nb_req < bpp
    assert geom.pages == H * geom.nb_pool // bpp
    assert geom.host_pages == geom.pages // M
    # host bytes are exactly the LPP tail pages (§4.2)
    assert geom.host_heads.sum() * geom.head_block_bytes == geom.host_pages * kv.PAGE
    # host heads per block take at most two adjacent values (§4.5)
    vals = set(geom.host_heads.tolist())
    assert len(vals) <= 2 and (len(vals) < 2 or max(vals) - min(vals) == 1)


def test_host_head_is_last_head_when_tail_fits_one_region():
    geom = kv.kv_geometry(9250, 8, 128, 111)
    shh, loc = kv.block_lists(geom)
    # tail = last host_pages pages of head 7's region: the last 512*h blocks
    assert shh == list(range(geom.nb_pool - 512 * geom.host_pages, geom.nb_pool))
    assert geom.host_pages == (8 * geom.nb_pool // 512) // 111


def test_more_heads_than_modulus_mixes_floor_and_ceil():
    """§4.5: with H > M, blocks carry floor(H/M) or ceil(H/M) host heads."""
    H, M = 8, 3
    geom = kv.kv_geometry(512 * 3, H, 128, M)
    vals = sorted(set(geom.host_heads.tolist()))
    assert vals == [H // M, -(-H // M)]
    assert abs(geom.host_heads.mean() - H / M) < 1e-12


def test_budget_split_extremes():
    """Capacity-budget split: a budget that holds the pool puts nothing on
    host (the all-HBM map); a zero budget puts every head of every block on
    host."""
    H, D, layers = 8, 128, 4
    full = kv.kv_geometry(3000, H, D, 2, hbm_pages=10 ** 9)
    assert full.host_pages == 0 and not full.host_heads.any()
    pages = full.pages
    assert kv.budget_hbm_pages(2 * layers * pages * kv.PAGE, layers) == pages
    assert kv.budget_hbm_pages(2 * layers * pages * kv.PAGE - 1, layers) == pages - 1
    none = kv.kv_geometry(3000, H, D, 2, hbm_pages=kv.budget_hbm_pages(0, layers))
    assert none.host_pages == pages and set(none.host_heads.tolist()) == {H}


def test_budget_split_high_throughput_shape():
    """The batch-256, 40e9-byte KV budget shape (8 KV heads, head_dim 128, 32
    layers, contexts uniform in [1024, 8192]): about three quarters of the KV
    bytes overflow to host, the tail covers whole heads H-1, H-2, ... and part
    of one more, so blocks carry c or c + 1 host heads (§4.5), with
    c = floor(h / pages_per_head) and the last (h mod pages_per_head) pages'
    blocks of the partly covered head one more."""
    rng = np.random.default_rng(0)
    lens = rng.integers(1024, 8192, 256, endpoint=True)
    nb_req = int(sum(-(-int(L) // 16) for L in lens))
    hbm = kv.budget_hbm_pages(40 * 10 ** 9, 32)
    g = kv.kv_geometry(nb_req, 8, 128, 2, hbm_pages=hbm)
    pph = g.nb_pool // g.blocks_per_page           # pages per head region
    assert g.host_pages == g.pages - hbm
    c, rem = divmod(g.host_pages, pph)
    expect = np.full(g.nb_pool, c)
    expect[g.nb_pool - rem * g.blocks_per_page:] += 1
    assert np.array_equal(g.host_heads, expect)
    assert g.host_heads.sum() * g.head_block_bytes == g.host_pages * kv.PAGE
    share = g.host_pages / g.pages
    assert 0.70 < share < 0.78


def _run(alloc, steps):
    out = []
    for st in steps:
        if st["op"] == "alloc":
            out.append(alloc.alloc(st["rid"], st["n"]))
        else:
            alloc.free_request(st["rid"])
            out.append(None)
    return out


def test_worked_example():
    a = kv.DSRAllocator(WORKED["shh"], WORKED["local"], WORKED["tau"])
    assert abs(a.tau - 2 / 8) < 1e-12
    for st, got in zip(WORKED["steps"], _run(a, WORKED["steps"])):
        if st["op"] != "alloc":
            continue
        exp = st["expect"]
        if exp == "EAGAIN":
            assert got == kv.EAGAIN, st
        else:
            assert got == exp, st


def _check_invariants(a, all_ids):
    free = a.free[kv.SHH] + a.free[kv.LOCAL]
    used = [b for bl in a.req_blocks.values() for b in bl]
    assert sorted(free + used) == sorted(all_ids)
    assert len(set(free)) == len(free) and len(set(used)) == len(used)
    for b in a.free[kv.SHH]:
        assert b in a.shh_set
    for b in a.free[kv.LOCAL]:
        assert b not in a.shh_set
    assert a.free[kv.SHH] == sorted(a.free[kv.SHH])
    assert a.free[kv.LOCAL] == sorted(a.free[kv.LOCAL])


@pytest.mark.parametrize("n_shh,n_loc", [(1, 3), (2, 2), (2, 6), (3, 5), (0, 4),
                                          (4, 0)])
def test_brute_force_event_orders(n_shh, n_loc):
    """Every sequence of up to 5 events over 3 requests (alloc of 1 or 2
    blocks, free) on tiny pools: conservation, typed lists, no EAGAIN while
    enough blocks are free, a type switch only when the preferred list is
    empty, and a new request's type follows the greedy rule."""
    shh = list(range(n_loc, n_loc + n_shh))
    loc = list(range(n_loc))
    all_ids = loc + shh
    events = [("a", r, n) for r in range(3) for n in (1, 2)] + \
             [("f", r, 0) for r in range(3)]
    for depth in range(1, 6):
        for seq in itertools.product(events, repeat=depth):
            a = kv.DSRAllocator(shh, loc)
            for op, r, n in seq:
                if op == "f":
                    if r in a.req_type:
                        a.free_request(r)
                    continue
                free_before = a.n_free()
                fs, fl = a.n_free(kv.SHH), a.n_free(kv.LOCAL)
                new = r not in a.req_type
                t0 = a.req_type.get(r)
                got = a.alloc(r, n)
                if free_before >= n:
                    assert got != kv.EAGAIN
                    if new:
                        greedy = (kv.SHH if (fs / (fs + fl) > a.tau and fs)
                                  else (kv.LOCAL if fl else kv.SHH))
                        t0 = greedy
                    # blocks come from t0's list until it empties
                    pref = [b for b in got if (b in a.shh_set) == (t0 == kv.SHH)]
                    avail = fs if t0 == kv.SHH else fl
                    assert len(pref) == min(n, avail)
                    assert got[:len(pref)] == pref
                    if len(pref) < n:
                        assert a.req_type[r] != t0      # sticky switch
                    else:
                        assert a.req_type[r] == t0
                else:
                    assert got == kv.EAGAIN
                    assert a.n_free() == free_before
                _check_invariants(a, all_ids)


def test_churn_keeps_host_share_near_target():
    """§5.11: under churn the realised host share of in-use KV stays within
    about 1% of the configured 1/M (four KV heads, modulus 12)."""
    H, M = 4, 12
    geom = kv.kv_geometry(512 * 3 * 4, H, 128, M)
    shh, loc = kv.block_lists(geom)
    a = kv.DSRAllocator(shh, loc)
    rng = np.random.default_rng(3)
    live = {}
    rid = 0
    shares = []
    for step in range(4000):
        # admit while there is room, else retire a random request
        n = int(rng.integers(8, 64))
        if a.n_free() >= n + 64 and len(live) < 64:
            got = a.alloc(rid, n)
            assert got != kv.EAGAIN
            live[rid] = n
            rid += 1
        else:
            victim = list(live)[int(rng.integers(0, len(live)))]
            a.free_request(victim)
            del live[victim]
        used = a.in_use_blocks()
        if step > 500 and used:
            shares.append(a.in_use_host_head_blocks(geom.host_heads) / (H * used))
    shares = np.array(shares)
    med = np.median(shares)
    assert abs(med - 1.0 / M) < 0.01
    # a rolling median over 50 steps never leaves a +-1.5% band
    roll = [np.median(shares[i:i + 50]) for i in range(0, len(shares) - 50, 10)]
    assert max(abs(r - 1.0 / M) for r in roll) < 0.015


POOL_TRACE = json.load(open(os.path.join(HERE, "golden", "dsr_pool_scale_example.json")))


def test_pool_scale_worked_example():
    g = POOL_TRACE["pool"]
    geom = kv.kv_geometry(g["n_blocks"], g["H"], g["D"], g["M"])
    shh, loc = kv.block_lists(geom)
    a = kv.DSRAllocator(shh, loc)
    assert a.tau == POOL_TRACE["tau"]
    for stp in POOL_TRACE["steps"]:
        op = stp["op"]
        if op == "alloc":
            got = a.alloc(stp["rid"], stp["n"])
            if stp.get("expect") == "EAGAIN":
                assert got == kv.EAGAIN
            elif "expect_range" in stp:
                assert got == list(range(*stp["expect_range"]))
            else:
                assert got == [b for r in stp["expect_ranges"] for b in range(*r)]
        elif op == "free":
            a.free_request(stp["rid"])
        elif op == "type":
            assert a.req_type[stp["rid"]] == stp["expect"]
        else:
            assert a.in_use_blocks() == stp["used_blocks"]
            assert a.in_use_host_head_blocks(geom.host_heads) == stp["used_host_head_blocks"]
