"""The wave-aware KV allocator under Poisson arrivals (the realized host
ratio study of §5.11, synthetic arrivals): the serving loop of bench.py
driving the C++ allocator (plan-only pool, through the C-ABI) must make the
same decisions, step for step, as a loop written here over the oracle
allocator; the realized host share stays near the pool's target."""
import numpy as np
import pytest

import bench
import synth
from oracle import kvpool as okv
from paper_2609_13592_amd import binding as bd


def oracle_serving(trace, steps, max_batch, nb_req, H, M):
    """The same serving loop, written independently, over the oracle pool:
    FIFO admission of whole prompts (stop at the first refusal), one token
    per running request per step with a new block when the last is full,
    preemption of the latest admitted request when the pool is empty,
    retirement after the output length."""
    g = okv.kv_geometry(nb_req, H, 128, M)
    shh, loc = okv.block_lists(g)
    a = okv.DSRAllocator(shh, loc)
    waiting, live = [], []
    ctx_len, out_len, owned = {}, {}, {}
    arrived, rows = 0, []
    refused = preempted = finished = 0
    for step in range(steps):
        while arrived < len(trace) and trace[arrived][0] <= step:
            waiting.append(arrived)
            arrived += 1
        while waiting and len(live) < max_batch:
            r = waiting[0]
            got = a.alloc(r, -(-trace[r][1] // 16))
            if got == okv.EAGAIN:
                refused += 1
                break
            waiting.pop(0)
            live.append(r)
            ctx_len[r], out_len[r], owned[r] = trace[r][1], 0, list(got)
        k = 0
        while k < len(live):
            r = live[k]
            if ctx_len[r] % 16 == 0:
                got = a.alloc(r, 1)
                while got == okv.EAGAIN:
                    v = live.pop()
                    a.free_request(v)
                    del ctx_len[v], out_len[v], owned[v]
                    waiting.insert(0, v)
                    preempted += 1
                    if v == r:
                        break
                    got = a.alloc(r, 1)
                if got == okv.EAGAIN:
                    continue
                owned[r].extend(got)
            ctx_len[r] += 1
            out_len[r] += 1
            k += 1
        stay = []
        for r in live:
            if out_len[r] >= trace[r][2]:
                a.free_request(r)
                finished += 1
                del ctx_len[r], out_len[r], owned[r]
            else:
                stay.append(r)
        live = stay
        shh_reqs = sum(1 for r in a.req_type if a.req_type[r] == okv.SHH)
        rows.append((a.in_use_blocks(), a.in_use_host_head_blocks(g.host_heads), len(live),
                     len(waiting), shh_reqs))
    return np.array(rows, dtype=np.int64), {"refused_admissions": refused,
                                            "preemptions": preempted,
                                            "finished": finished, "arrived": arrived}


def product_serving(trace, steps, max_batch, nb_req, H, M):
    ctx = bd.boost_init(-1)
    pool = bd.boost_kv_pool_create(ctx, 1, H, 128, nb_req, M, bd.KV_LPP, q_heads=4 * H)
    try:
        def alloc(rid, n):
            ids = bd.boost_kv_alloc(pool, rid, n)
            return None if ids == bd.EAGAIN else ids

        def stats():
            s = bd.boost_kv_stats(pool)
            return s["used_blocks"], s["used_host_head_blocks"], s["shh_requests"]
        return bench.run_churn(trace, steps, max_batch, alloc,
                               lambda rid: bd.boost_kv_free(pool, rid), stats)
    finally:
        bd.boost_kv_pool_destroy(pool)
        bd.boost_shutdown(ctx)


@pytest.mark.parametrize("rate,nb_req,H,M", [
    (0.2, 3000, 4, 12),      # saturated: refused admissions and preemptions
    (0.01, 3000, 8, 16),     # moderate load
    (0.05, 2000, 8, 127),    # this GPU's modulus, one host page per tensor
])
def test_serving_loop_matches_oracle(rate, nb_req, H, M):
    steps = 2500
    trace = synth.poisson_arrivals(5, steps, rate, 64, 1024, 64, 1024)
    rows_p, cnt_p = product_serving(trace, steps, 64, nb_req, H, M)
    rows_o, cnt_o = oracle_serving(trace, steps, 64, nb_req, H, M)
    assert cnt_p == cnt_o
    assert np.array_equal(rows_p, rows_o)
    if rate == 0.2:
        assert cnt_p["preemptions"] > 0 and cnt_p["refused_admissions"] > 0


def test_realized_host_share_near_target():
    """§5.11: under continuous arrivals the realized KV host share stays
    close to the target (the paper: rolling median 7.7-9.2 % against
    8.3 %).  4 KV heads, modulus 12; synthetic Poisson arrivals."""
    steps, warm = 8000, 1000
    trace = synth.poisson_arrivals(11, steps, 0.03, 256, 2048, 512, 4096)
    rows, cnt = oracle_serving(trace, steps, 256, 16000, 4, 12)
    used, host = rows[warm:, 0].astype(float), rows[warm:, 1].astype(float)
    share = host / np.maximum(4 * used, 1)
    assert cnt["preemptions"] == 0
    assert abs(share.mean() - 1 / 12) < 0.01
    rm = bench._rolling_median(share, 100)
    assert rm.min() > 1 / 12 - 0.02 and rm.max() < 1 / 12 + 0.02
