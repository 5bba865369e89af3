"""C9: per-wave host share of a work-unit schedule (oracle, test-only).

§2.2 defines a wave as the set of threadblocks resident on the GPU at once;
§2.4 and §3 ("CAP") ask that every wave send its accesses to both tiers in
proportion to their bandwidths.  §4.4 notes that the final, partial wave of a
kernel leaves a residual variance, so it is excluded here.

Given the tier of every unit in dispatch order and a wave size R (units that
are resident together), the wave w covers units [w*R, (w+1)*R).
"""
from __future__ import annotations

import numpy as np


def wave_host_fractions(unit_tiers, R: int) -> np.ndarray:
    t = np.asarray(unit_tiers, dtype=np.float64)
    n_full = len(t) // R
    return np.array([t[w * R:(w + 1) * R].mean() for w in range(n_full)])


def window_host_counts(page_tiers, P: int) -> np.ndarray:
    """Host pages in every window of P consecutive pages (all offsets)."""
    t = np.asarray(page_tiers, dtype=np.int64)
    c = np.concatenate([[0], np.cumsum(t)])
    return c[P:] - c[:-P]


def wave_stats(unit_tiers, R: int):
    f = wave_host_fractions(unit_tiers, R)
    if len(f) == 0:
        return dict(waves=0, mean=0.0, max_dev=0.0, var=0.0)
    m = float(f.mean())
    return dict(waves=len(f), mean=m, max_dev=float(np.abs(f - m).max()),
                var=float(f.var()))
