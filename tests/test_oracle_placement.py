"""Pins of the placement oracle (C1-C3) against the paper and brute force."""
import itertools
import json
import math
import os

import numpy as np
import pytest

from oracle import placement as pl
from oracle import waves

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                   "paper_pins.json")))
MiB = 1024 * 1024


def test_modulus_alpha_10pct():
    g = GOLD["alpha_10pct"]
    M = pl.modulus_from_alpha(g["alpha"])
    assert M == g["M"] and M - 1 == g["K"]
    # one host page in every M is exactly alpha / (1 + alpha) here
    assert abs(1.0 / M - g["host_share"]) < 1e-9
    assert abs(1.0 / M - g["alpha"] / (1 + g["alpha"])) < 1e-12


def test_modulus_gh200_measured():
    g = GOLD["gh200_measured"]
    M = pl.modulus_from_alpha(g["host_gib_s"] / g["hbm_gib_s"])
    assert M == g["M"]


def test_modulus_12_share():
    g = GOLD["modulus_12"]
    tiers = pl.mpp_tier_map(120 * pl.PAGE, g["M"])
    assert abs(tiers.mean() - g["host_share"]) < 1e-9


@pytest.mark.parametrize("alpha", np.linspace(0.004, 1.0, 400))
def test_ceil_rule_keeps_share_at_or_below_alpha(alpha):
    """§4.4: K = ceil(1/alpha) keeps the host share 1/(K+1) at or below the
    proportional share alpha/(1+alpha), and K is the smallest such integer."""
    M = pl.modulus_from_alpha(float(alpha))
    K = M - 1
    assert 1.0 / M <= alpha / (1 + alpha) + 1e-12
    if K > 1:
        assert 1.0 / K > alpha / (1 + alpha) - 1e-12


@pytest.mark.parametrize("bad", [0.0, -0.1, 1.5, float("nan")])
def test_modulus_rejects_bad_alpha(bad):
    with pytest.raises(ValueError):
        pl.modulus_from_alpha(bad)


def test_single_layer_map():
    g = GOLD["config_single_layer"]
    nbytes = g["rows"] * g["cols"] * 2
    t = pl.mpp_tier_map(nbytes, g["M"])
    assert len(t) == g["pages"]
    assert np.flatnonzero(t).tolist() == g["host_pages"]


def test_superpage_lcm_example():
    g = GOLD["superpage_down_proj"]
    S = pl.superpage_pages(int(g["footprint_mib"] * MiB))
    assert S == g["S"] and S * 2 == g["superpage_mib"]


def test_rows_per_page_example():
    g = GOLD["rows_per_page_28k"]
    assert pl.PAGE // g["row_bytes"] == g["whole_rows_per_page"]
    assert g["cta_columns"] * g["row_bytes"] / pl.PAGE == g["cta_pages"]


def test_superpages_stay_in_one_tier():
    S = pl.superpage_pages(int(3.5 * MiB))
    t = pl.mpp_tier_map(300 * pl.PAGE, 5, int(3.5 * MiB))
    for j in range(0, len(t), S):
        assert len(set(t[j:j + S].tolist())) == 1
    # superpage j on host iff j mod 5 == 4
    sp = t[::S]
    assert np.flatnonzero(sp).tolist() == [j for j in range(len(sp)) if j % 5 == 4]


@pytest.mark.parametrize("n,M,S", [(1, 2, 1), (15, 16, 1), (16, 16, 1),
                                    (17, 3, 2), (100, 7, 7), (501, 111, 1),
                                    (112, 111, 1), (110, 111, 1)])
def test_host_count_closed_form(n, M, S):
    """Host pages = size of the superpages j < ceil(n/S) with j mod M = M-1;
    a tensor with fewer than M superpages has none (per-tensor restart, §3.1)."""
    t = pl.mpp_tier_map(n * pl.PAGE, M, S * pl.PAGE if S > 1 else 0)
    nsp = -(-n // S)
    expect = sum(min(S, n - j * S) for j in range(M - 1, nsp, M))
    assert int(t.sum()) == expect
    if nsp < M:
        assert t.sum() == 0


def test_partial_last_page_counts():
    assert pl.n_pages(1) == 1
    assert pl.n_pages(pl.PAGE) == 1
    assert pl.n_pages(pl.PAGE + 1) == 2
    assert len(pl.mpp_tier_map(3 * pl.PAGE + 5, 2)) == 4


@pytest.mark.parametrize("M", range(2, 17))
def test_window_invariant_brute_force(M):
    """Insight-1 (§3.1): every window of P consecutive pages holds floor(P/M)
    or ceil(P/M) host pages, and exactly P/M when M divides P (no variance
    across waves).  Checked over every window of every size, n <= 64."""
    for n in range(1, 65):
        t = pl.mpp_tier_map(n * pl.PAGE, M)
        for P in range(1, n + 1):
            c = waves.window_host_counts(t, P)
            assert c.min() >= P // M
            assert c.max() <= -(-P // M)
            if P % M == 0 and n >= M * (n // M):
                full = [int(t[i:i + P].sum()) for i in range(0, n - P + 1)
                        if i + P <= M * (n // M)]
                assert all(v == P // M for v in full)


@pytest.mark.parametrize("M", range(2, 9))
def test_mpp_minimises_window_discrepancy_brute_force(M):
    """Optimality of the modulo rule (§3.1, Insight-1): among ALL tier maps
    of n <= 16 pages with the same number of host pages, none has a smaller
    largest window discrepancy max |host(window) - len(window) / M| than the
    modulo map, and the modulo map's is below one page."""
    for n in range(M, 17):
        t = pl.mpp_tier_map(n * pl.PAGE, M).astype(np.int64)
        h = int(t.sum())
        assert h == n // M

        def discrepancy(maps):  # maps [C, n] of 0/1 -> [C]
            ps = np.concatenate([np.zeros((maps.shape[0], 1), np.int64),
                                 np.cumsum(maps, axis=1)], axis=1)
            i, j = np.triu_indices(n + 1, k=1)
            cnt = ps[:, j] - ps[:, i]
            return np.abs(cnt - (j - i) / M).max(axis=1)

        d_mpp = discrepancy(t[None, :])[0]
        assert d_mpp < 1.0
        combos = np.array(list(itertools.combinations(range(n), h)), np.int64)
        maps = np.zeros((len(combos), n), np.int64)
        np.put_along_axis(maps, combos, 1, axis=1)
        assert discrepancy(maps).min() >= d_mpp - 1e-12


def test_random_placement_has_window_variance():
    """Contrast (§2.6): a random placement with the same share spreads far
    more than one page across windows, MPP never does."""
    n, M, P = 400, 11, 22
    mpp = waves.window_host_counts(pl.mpp_tier_map(n * pl.PAGE, M), P)
    assert mpp.max() - mpp.min() <= 1
    spreads = []
    for seed in range(20):
        r = waves.window_host_counts(pl.bapp_r_map(n, 1.0 / M, seed), P)
        spreads.append(r.max() - r.min())
    assert min(spreads) >= 2


def test_bapp_r_matches_binomial_spread():
    """§2.6 prints 10% +- 1.5% over a kernel and +- 3.6% within a wave; those
    are binomial spreads sqrt(p(1-p)/n) for n of about 400 and 69 pages."""
    g = GOLD["bapp_r_spread"]
    p = g["p"]
    n_kernel = round(p * (1 - p) / g["kernel_sd"] ** 2)
    n_wave = round(p * (1 - p) / g["wave_sd"] ** 2)
    assert 380 <= n_kernel <= 420 and 65 <= n_wave <= 72
    for n, sd in ((n_kernel, g["kernel_sd"]), (n_wave, g["wave_sd"])):
        fr = [pl.bapp_r_map(n, p, s).mean() for s in range(2000)]
        assert abs(np.mean(fr) - p) < 0.004
        assert abs(np.std(fr) - sd) < 0.15 * sd


def test_linear_map():
    t = pl.linear_map(25, 12)
    assert t.tolist() == [0] * 23 + [1] * 2


def test_budget_modulus_closed_form():
    """C3 against the closed form sum_t floor(n_t / M) host pages (S = 1)."""
    rng = np.random.default_rng(5)
    sizes = [int(s) * pl.PAGE for s in rng.integers(1, 400, size=12)]
    total = sum(s // pl.PAGE for s in sizes)
    for budget_pages in (total, total - 1, total - 30, int(total * 0.8),
                         int(total * 0.55)):
        M = pl.modulus_from_budget(sizes, budget_pages * pl.PAGE, 200)
        host = sum((s // pl.PAGE) // M for s in sizes)
        assert total - host <= budget_pages
        if M < 200:
            host_next = sum((s // pl.PAGE) // (M + 1) for s in sizes)
            assert total - host_next > budget_pages
    with pytest.raises(MemoryError):
        pl.modulus_from_budget(sizes, (total // 3) * pl.PAGE, 200)


def test_budget_modulus_70b_chain():
    """The 70B-shaped fused chain (80 layers, d 8192, FFN 28672, GQA 64/8,
    vocab 128256, embedding and lm_head included) under a 120e9-byte HBM
    weight budget.  Closed form with S = 1."""
    d, f, v = 8192, 28672, 128256
    per_layer = [(64 + 16) * 128 * d, d * 64 * 128, 2 * f * d, d * f]
    sizes = per_layer * 80 + [v * d, v * d]
    sizes = [s * 2 for s in sizes]
    pages = [s // pl.PAGE for s in sizes]
    assert pages[:4] == [80, 64, 448, 224] and pages[-1] == 1002
    M = pl.modulus_from_budget(sizes, 120 * 10 ** 9, 10 ** 6)
    host = sum(n // M for n in pages)
    assert M == 6 and host == 11054
    assert (sum(pages) - host) * pl.PAGE <= 120 * 10 ** 9
    assert (sum(pages) - sum(n // 7 for n in pages)) * pl.PAGE > 120 * 10 ** 9


# ------------------------------------------------------------ contrast maps
def test_global_modulo_at_phase_zero_is_mpp():
    """Special case: at phase 0 the pattern that runs across tensors is the
    per-tensor modulo map (§3.1) of that tensor."""
    for n in range(1, 70):
        for M in (2, 3, 11, 16, 127):
            assert np.array_equal(pl.mpp_global_map(n, M, 0),
                                  pl.mpp_tier_map(n * pl.PAGE, M))


def test_global_modulo_chain_is_one_big_tensor():
    """Without the per-tensor restart, the maps of consecutive tensors placed
    at cumulative phases are the modulo map of their concatenation."""
    rng = np.random.default_rng(3)
    for M in (5, 12, 127):
        sizes = [int(s) for s in rng.integers(1, 300, size=20)]
        phases = np.concatenate([[0], np.cumsum(sizes)[:-1]])
        cat = np.concatenate([pl.mpp_global_map(n, M, p) for n, p in zip(sizes, phases)])
        assert np.array_equal(cat, pl.mpp_tier_map(sum(sizes) * pl.PAGE, M))


@pytest.mark.parametrize("M", [2, 7, 12, 127])
def test_global_modulo_host_count_closed_form(M):
    for phase in range(0, 3 * M):
        for n in range(1, 3 * M):
            got = int(pl.mpp_global_map(n, M, phase).sum())
            assert got == (phase + n) // M - phase // M


def test_global_modulo_breaks_per_kernel_share():
    """§2.6: an interleave that ignores kernel boundaries can give a small
    tensor a host page, a host share far above 1/M for that kernel; modulo
    placement restarted per tensor (§3.1) never exceeds 1/M."""
    M, n = 127, 16        # a 16-page tensor at the measured modulus
    shares = [pl.mpp_global_map(n, M, p).mean() for p in range(M)]
    assert max(shares) == 1 / 16 and sum(s > 0 for s in shares) == n
    assert pl.mpp_tier_map(n * pl.PAGE, M).sum() == 0


def test_bapp_r_from_uniforms_grid():
    """Draws on the grid i / N put exactly ceil(N / M) pages on host: the
    first ones, where i * M < N."""
    for N in (10, 64, 127, 1000):
        for M in (2, 3, 11, 127):
            u = np.arange(N) / N
            t = pl.bapp_r_from_uniforms(u, M)
            assert t.sum() == -(-N // M)
            assert t[:-(-N // M)].all()


def test_bapp_r_from_uniforms_share():
    """Random draws: the host share is binomial around 1/M (§2.6)."""
    import synth
    M, n = 12, 400
    fr = np.array([pl.bapp_r_from_uniforms(synth.uniforms(s, n), M).mean()
                   for s in range(1000)])
    p = 1 / M
    assert abs(fr.mean() - p) < 0.003
    assert abs(fr.std() - math.sqrt(p * (1 - p) / n)) < 0.1 * math.sqrt(p * (1 - p) / n)
