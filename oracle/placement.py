"""C1-C3: modulus and page placement for static weights (oracle, test-only).

Paper passages followed:
  * §2.3: alpha is host (C2G) read bandwidth divided by HBM read bandwidth.
  * §3 "CAP": a fraction alpha/(1+alpha) of accesses should go to host.
  * §3.1 "Wave-aware Modulo Page Placement": for an HBM-to-host ratio K, the
    first K pages go to HBM and the (K+1)-th to host, repeating; every weight
    tensor is allocated on its own so the pattern restarts per tensor.
  * §3.2 and §4.4 "Superpages": group pages into superpages of
    lcm(CTA footprint, page) bytes, keep each superpage in one tier and apply
    the modulo rule over superpages.
  * §4.4: when 1/alpha is not an integer, K = ceil(1/alpha), keeping the host
    share below alpha.
  * §2.6 "Bandwidth-Aware Page Placement": BAPP-R, a random alpha share of pages
    on host (contrast only); Linux weighted interleaving stripes pages over
    the tiers without regard to kernel (tensor) boundaries (contrast only).
  * §5.7: proportional interleaving, i.e. a linear split, on weights
    (contrast only).
  * §4.2 "LPP": the first 1/(1+alpha) of pages in HBM, the rest on host.
"""
from __future__ import annotations

import math

import numpy as np

PAGE = 2 * 1024 * 1024          # 2 MiB GPU page (§1, §4.4)
HBM, HOST = 0, 1


def modulus_from_alpha(alpha: float) -> int:
    """M = K + 1 with K = ceil(1/alpha) (§3.1, §4.4).

    Reading: a 1e-9 guard keeps alpha = 0.1 from rounding up to K = 11 through
    floating-point error in 1/alpha.  alpha must lie in (0, 1].
    """
    if not (alpha > 0.0 and alpha <= 1.0):
        raise ValueError("alpha must be in (0, 1]")
    k = math.ceil(1.0 / alpha - 1e-9)
    return k + 1


def n_pages(nbytes: int, page: int = PAGE) -> int:
    """Pages a tensor occupies; a partial last page counts as a page."""
    return -(-int(nbytes) // page)


def superpage_pages(footprint: int, page: int = PAGE) -> int:
    """S = lcm(footprint, page) / page (§3.2, §4.4); 1 when footprint is 0."""
    if footprint <= 0:
        return 1
    return math.lcm(int(footprint), page) // page


def mpp_tier_map(nbytes: int, M: int, footprint: int = 0,
                 page: int = PAGE) -> np.ndarray:
    """Tier of every page of one tensor under modulo placement (C2).

    Superpage j covers pages [j*S, (j+1)*S).  Superpage j is on host exactly
    when j mod M == M - 1: M - 1 superpages in HBM, then one on host (§4.4).
    The phase restarts at 0 for every tensor (§3.1), so a tensor with fewer
    than M superpages keeps every page in HBM.
    """
    if M < 2:
        raise ValueError("M must be >= 2")
    n = n_pages(nbytes, page)
    S = superpage_pages(footprint, page)
    j = np.arange(n, dtype=np.int64) // S          # superpage of every page
    return (j % M == M - 1).astype(np.uint8)


def hbm_pages_under(sizes, M: int, footprints=None, page: int = PAGE) -> int:
    """Pages kept in HBM when every tensor is placed on its own by MPP."""
    total = 0
    seen = {}
    for t, nbytes in enumerate(sizes):
        f = 0 if footprints is None else footprints[t]
        key = (int(nbytes), int(f))
        if key not in seen:
            tiers = mpp_tier_map(nbytes, M, f, page)
            seen[key] = int(np.count_nonzero(tiers == HBM))
        total += seen[key]
    return total


def modulus_from_budget(sizes, hbm_budget: int, M_alpha: int,
                        footprints=None, page: int = PAGE) -> int:
    """Largest M in [2, M_alpha] whose HBM pages fit the budget (C3).

    Reading: the paper always places about an alpha share on host and never
    derives M from a capacity budget.  When the weights exceed an HBM budget we
    keep the modulo rule and lower M until the HBM-resident pages (counted as
    whole 2 MiB pages) fit.  Raises MemoryError when even M = 2 does not fit.
    """
    if M_alpha < 2:
        raise ValueError("M_alpha must be >= 2")
    # Past the largest superpage count every M gives the all-HBM map, so the
    # scan can start there.
    most = max(-(-n_pages(s, page) // superpage_pages(
        0 if footprints is None else footprints[t], page))
        for t, s in enumerate(sizes))
    for M in range(min(M_alpha, most + 1), 1, -1):
        if hbm_pages_under(sizes, M, footprints, page) * page <= hbm_budget:
            return M
    raise MemoryError("HBM budget below the M = 2 placement")


def bapp_r_map(n: int, share: float, seed: int) -> np.ndarray:
    """BAPP-R contrast (§2.6): each page independently on host with
    probability ``share`` (seeded)."""
    rng = np.random.default_rng(seed)
    return (rng.random(n) < share).astype(np.uint8)


def bapp_r_from_uniforms(u, M: int) -> np.ndarray:
    """BAPP-R (§2.6) with the random draws given: page i on host iff
    u[i] * M < 1, i.e. u[i] < 1/M written without the rounded reciprocal.
    The draws are inputs (uniform on [0, 1)), so any implementation fed the
    same draws makes the same decisions."""
    u = np.asarray(u, dtype=np.float64)
    return (u * float(M) < 1.0).astype(np.uint8)


def mpp_global_map(n: int, M: int, phase: int) -> np.ndarray:
    """Modulo placement that is NOT restarted per tensor (the contrast to
    §3.1's per-tensor allocation; an interleave blind to tensor boundaries,
    §2.6): a tensor whose first page has global index ``phase`` (pages of
    the tensors placed before it) puts page i on host iff
    (phase + i) mod M == M - 1."""
    if M < 2:
        raise ValueError("M must be >= 2")
    g = int(phase) + np.arange(int(n), dtype=np.int64)
    return (g % M == M - 1).astype(np.uint8)


def linear_map(n: int, M: int) -> np.ndarray:
    """Linear placement (§4.2 LPP) over n pages: the last floor(n/M) pages on
    host, the rest in HBM."""
    tiers = np.zeros(n, dtype=np.uint8)
    h = n // M
    if h:
        tiers[n - h:] = HOST
    return tiers
