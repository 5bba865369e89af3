"""Pins of the per-wave schedule model (C9)."""
import numpy as np

from oracle import placement as pl
from oracle import waves


def test_mpp_waves_have_zero_variance():
    """A wave that covers a multiple of M pages sees exactly 1/M host pages
    (§3.1 Insight-1); the final partial wave is excluded (§4.4)."""
    M, U = 11, 4                      # U work units per page
    tiers = pl.mpp_tier_map(500 * pl.PAGE, M)
    units = np.repeat(tiers, U)
    st = waves.wave_stats(units, 2 * M * U)
    assert st["waves"] == len(units) // (2 * M * U)
    assert abs(st["mean"] - 1.0 / M) < 1e-12 and st["var"] < 1e-30
    R = 2 * M * U
    counts = [int(units[w * R:(w + 1) * R].sum()) for w in range(st["waves"])]
    assert set(counts) == {2 * U}


def test_random_waves_vary():
    M, U = 11, 4
    t = pl.bapp_r_map(2000, 1.0 / M, 7)
    st = waves.wave_stats(np.repeat(t, U), M * U * 6)
    assert st["var"] > 0 and st["max_dev"] > 0.02


def test_partial_wave_excluded():
    f = waves.wave_host_fractions([1, 0, 0, 1, 1], 2)
    assert f.tolist() == [0.5, 0.5]
