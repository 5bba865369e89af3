"""C4-C5: KV pool geometry and the wave-aware block allocator (oracle, test-only).

Paper passages followed:
  * §4.2 "LPP": the KV virtual range is split linearly: the first 1/(1+alpha)
    of its pages in HBM, the last alpha/(1+alpha) on host, so the tier of a KV
    page is a fixed function of its address.
  * §4.5 "Tensor Layout Reordering": KV tensors are reshaped so KV heads are
    the outermost dimension; each head's data is contiguous and lines up with
    the LPP split, bounding the host share by 1/H.  With H > M, blocks carry
    floor(H/M) or ceil(H/M) host heads.
  * §4.3 "Block-level KV Head Chunk Partitioning": single-head-host (SHH) blocks
    hold one head on host, all-local blocks none; their ratio H : (M - H) puts
    1/M of the KV bytes on host.
  * §4.3 "Wave-aware Block Fulfillment": a new request gets the SHH type when
    the free-SHH fraction exceeds the target, else all-local; every block of a
    request has the request's type.  When the SHH list is empty the request
    falls back to all-local; when the all-local list is empty SHH blocks are
    appended to the all-local request and the request stays SHH (sticky); when
    blocks run out the call is handed back to the scheduler.
  * §4.5 "Virtual Memory Integration": two free lists, no per-page tracking.

Exact decision sequences depend on tie-breaks the paper leaves open; they are
fixed below and are "parity unpinned" against the paper (their invariants are
pinned by the tests).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

PAGE = 2 * 1024 * 1024
SHH, LOCAL = 1, 0          # block / request types
EAGAIN = -11


@dataclass(frozen=True)
class KVGeometry:
    """One KV tensor (one layer, K or V) laid out as [H][NB][T][D]."""
    heads: int
    head_dim: int
    block_tokens: int
    elem_bytes: int
    nb_pool: int            # blocks in the pool, a multiple of blocks_per_page
    blocks_per_page: int    # head-blocks per 2 MiB page
    pages: int              # pages of one K (or V) tensor
    host_pages: int         # LPP tail pages of one K (or V) tensor
    host_heads: np.ndarray = field(compare=False)   # per block, host heads

    @property
    def head_block_bytes(self) -> int:
        return self.block_tokens * self.head_dim * self.elem_bytes


def budget_hbm_pages(hbm_budget_bytes: int, layers: int, page: int = PAGE) -> int:
    """HBM pages of each K (or V) tensor when the whole pool (K and V of every
    layer) may hold hbm_budget_bytes in HBM: the budget split evenly over the
    2 * layers tensors, in whole pages (reading: the capacity budget of the
    high-throughput setting, §5.2, applied tensor by tensor)."""
    return hbm_budget_bytes // (2 * layers * page)


def kv_geometry(n_blocks_req: int, heads: int, head_dim: int, M: int,
                block_tokens: int = 16, elem_bytes: int = 2,
                page: int = PAGE, hbm_pages: int | None = None) -> KVGeometry:
    """C4.  Pool size, LPP tail and per-block host-head counts.

    * head-block = block_tokens * head_dim * elem_bytes bytes; it must divide a
      page so each page holds a whole number of head-blocks.
    * NB is rounded up to a multiple of blocks_per_page so that every head's
      region starts on a page boundary (§4.5).
    * pages p = H * NB / blocks_per_page; host pages h = floor(p / M) at the
      tail of the range (§4.2 LPP, with the floor that keeps the host share at
      or below 1/M as in §4.4).  With hbm_pages given (a capacity budget), M
      is not used and the tail is every page past the first hbm_pages.
    * head h of block b lies in page (h * NB + b) // blocks_per_page; the block
      has one host head per such page inside the tail.
    """
    if (hbm_pages is None and M < 2) or heads < 1 or head_dim < 1 or n_blocks_req < 1:
        raise ValueError("bad geometry")
    hbb = block_tokens * head_dim * elem_bytes
    if page % hbb:
        raise ValueError("head-block must divide the page")
    bpp = page // hbb
    nb = -(-n_blocks_req // bpp) * bpp
    p = heads * nb // bpp
    h = p // M if hbm_pages is None else max(0, p - hbm_pages)
    first_host_page = p - h
    host_heads = np.zeros(nb, dtype=np.int64)
    for head in range(heads):
        for b in range(nb):
            if (head * nb + b) // bpp >= first_host_page:
                host_heads[b] += 1
    return KVGeometry(heads, head_dim, block_tokens, elem_bytes, nb, bpp, p, h,
                      host_heads)


def block_lists(geom: KVGeometry):
    """Split block ids into the SHH list (the larger host-head count) and the
    all-local list (the smaller one).  For H <= M these are 1 and 0 host heads;
    for H > M they are ceil and floor of the tail's heads per block (§4.5).
    When every block has the same count all blocks are all-local."""
    hh = geom.host_heads
    lo, hi = int(hh.min()), int(hh.max())
    ids = np.arange(geom.nb_pool)
    if lo == hi:
        return [], ids.tolist()
    return ids[hh == hi].tolist(), ids[hh == lo].tolist()


class DSRAllocator:
    """C5, the wave-aware block fulfillment of §4.3 on two free lists.

    Readings (the paper is silent on these):
      1. tau, the SHH threshold, is the pool's own SHH fraction
         n_shh / NB (the paper's H/M realised by page-granular LPP).
      2. "exceeds" is strict (>).
      3. blocks are handed out lowest id first.
      4. a multi-block call is all-or-nothing: on shortfall it is rolled back
         and EAGAIN is returned (the scheduler decides, §4.3).
      5. the sticky switch works in both directions.
      6. a request's type is decided at its first allocation; afterwards only
         the empty-list fallback changes it.
    Decision sequences: parity unpinned (tie-breaks are ours).
    """

    def __init__(self, shh_ids, local_ids, tau=None):
        self.shh_set = set(int(b) for b in shh_ids)
        self.free = {SHH: sorted(int(b) for b in shh_ids),
                     LOCAL: sorted(int(b) for b in local_ids)}
        total = len(self.free[SHH]) + len(self.free[LOCAL])
        self.nb = total
        self.tau = (len(self.free[SHH]) / total) if tau is None else tau
        self.req_type = {}
        self.req_blocks = {}

    def n_free(self, t=None):
        if t is None:
            return len(self.free[SHH]) + len(self.free[LOCAL])
        return len(self.free[t])

    def _pop(self, t):
        # lowest id first (reading 3); lists are kept sorted
        return self.free[t].pop(0)

    def _push(self, b):
        t = SHH if b in self.shh_set else LOCAL
        lst = self.free[t]
        # insert keeping the list sorted
        lo, hi = 0, len(lst)
        while lo < hi:
            mid = (lo + hi) // 2
            if lst[mid] < b:
                lo = mid + 1
            else:
                hi = mid
        lst.insert(lo, b)

    def new_request_type(self):
        """Greedy type of a new request (§4.3)."""
        fs, fl = len(self.free[SHH]), len(self.free[LOCAL])
        if fs + fl == 0:
            return None
        f = fs / (fs + fl)
        if f > self.tau and fs > 0:
            return SHH
        if fl > 0:
            return LOCAL
        return SHH

    def alloc(self, rid, n):
        """Append n blocks to request rid; returns the new block ids or
        EAGAIN.  Raises ValueError for n < 1."""
        if n < 1:
            raise ValueError("n must be >= 1")
        if self.n_free() < n:
            return EAGAIN
        new = rid not in self.req_type
        t = self.new_request_type() if new else self.req_type[rid]
        if t is None:
            return EAGAIN
        out = []
        for _ in range(n):
            if not self.free[t]:
                t = LOCAL if t == SHH else SHH      # sticky fallback
            out.append(self._pop(t))
        self.req_type[rid] = t
        self.req_blocks.setdefault(rid, []).extend(out)
        return out

    def free_request(self, rid):
        if rid not in self.req_type:
            raise KeyError(rid)
        for b in self.req_blocks.pop(rid):
            self._push(b)
        del self.req_type[rid]

    def in_use_host_head_blocks(self, host_heads):
        return int(sum(int(host_heads[b]) for bl in self.req_blocks.values()
                       for b in bl))

    def in_use_blocks(self):
        return sum(len(bl) for bl in self.req_blocks.values())
