// KV pool geometry and the wave-aware block allocator (§4.2 LPP; §4.3 block
// types and greedy fulfillment with boundary conditions; §4.5 two free lists,
// heads-outermost layout, floor/ceil host heads when H > M).
#include "dsr.h"

#include <algorithm>

namespace bst {

int kv_geometry(uint32_t n_blocks, uint32_t H, uint32_t D, uint32_t T, uint32_t M,
                int mode, uint32_t layers, uint64_t hbm_budget_bytes, KvGeom& g) {
  if (n_blocks == 0 || H == 0 || D == 0 || T == 0)
    return fail(BOOST_EINVAL, "empty KV geometry");
  if (mode != BOOST_KV_LPP && mode != BOOST_KV_ALL_HBM && mode != BOOST_KV_ALL_HOST &&
      mode != BOOST_KV_BUDGET)
    return fail(BOOST_EINVAL, "tier_mode %d", mode);
  if (mode == BOOST_KV_BUDGET && layers == 0) return fail(BOOST_EINVAL, "0 layers");
  if (mode == BOOST_KV_LPP && M < 2) return fail(BOOST_EINVAL, "M=%u < 2", M);
  const uint64_t hbb = static_cast<uint64_t>(T) * D * 2;  // one head of one block
  if (kPage % hbb) return fail(BOOST_EINVAL, "head-block of %llu B does not divide a page",
                               (unsigned long long)hbb);
  g = KvGeom{};
  g.H = H;
  g.D = D;
  g.T = T;
  g.blocks_per_page = static_cast<uint32_t>(kPage / hbb);
  const uint64_t nb = (static_cast<uint64_t>(n_blocks) + g.blocks_per_page - 1) /
                      g.blocks_per_page * g.blocks_per_page;
  if (nb > 0x7fffffffull) return fail(BOOST_EINVAL, "pool too large");
  g.nb = static_cast<uint32_t>(nb);
  const uint64_t pages_per_head = nb / g.blocks_per_page;
  g.pages = H * pages_per_head;
  if (mode == BOOST_KV_LPP) {
    g.host_pages = g.pages / M;
  } else if (mode == BOOST_KV_BUDGET) {
    const uint64_t hbm = hbm_budget_bytes / (2ull * layers * kPage);  // per K or V tensor
    g.host_pages = g.pages > hbm ? g.pages - hbm : 0;
  } else {
    g.host_pages = mode == BOOST_KV_ALL_HOST ? g.pages : 0;
  }
  const uint64_t first_host = g.pages - g.host_pages;
  // head h of block b sits in page h * pages_per_head + b / blocks_per_page
  g.host_heads.assign(g.nb, 0);
  for (uint32_t h = 0; h < H; ++h) {
    const uint64_t head_first = h * pages_per_head;
    if (head_first + pages_per_head <= first_host) continue;  // head fully in HBM
    const uint64_t from_page = first_host > head_first ? first_host - head_first : 0;
    for (uint64_t b = from_page * g.blocks_per_page; b < g.nb; ++b) g.host_heads[b]++;
  }
  const auto mm = std::minmax_element(g.host_heads.begin(), g.host_heads.end());
  g.lo = *mm.first;
  g.hi = *mm.second;
  g.n_shh = 0;
  if (g.hi != g.lo)
    for (uint8_t c : g.host_heads) g.n_shh += c == g.hi;
  return BOOST_OK;
}

void Dsr::init(const KvGeom& g) {
  free_[0].clear();
  free_[1].clear();
  req_.clear();
  is_shh_.assign(g.nb, 0);
  host_heads_ = g.host_heads;
  for (uint32_t b = 0; b < g.nb; ++b) {
    const bool shh = g.hi != g.lo && g.host_heads[b] == g.hi;
    is_shh_[b] = shh;
    free_[shh ? BOOST_KV_SHH : BOOST_KV_LOCAL].insert(static_cast<int32_t>(b));
  }
  // reading: the greedy threshold is the pool's own SHH fraction (the paper's
  // H/M as realised by page-granular linear placement)
  tau_ = static_cast<double>(g.n_shh) / static_cast<double>(g.nb);
  used_ = used_hh_ = 0;
}

int Dsr::alloc(uint64_t rid, uint32_t n, int32_t* out) {
  if (n == 0 || !out) return fail(BOOST_EINVAL, "alloc of 0 blocks or null output");
  const uint64_t fs = free_[BOOST_KV_SHH].size(), fl = free_[BOOST_KV_LOCAL].size();
  // all-or-nothing: with the sticky fallback any n <= free blocks succeeds
  if (fs + fl < n) return fail(BOOST_EAGAIN, "pool has %llu free blocks, %u wanted",
                               (unsigned long long)(fs + fl), n);
  auto it = req_.find(rid);
  int type;
  if (it == req_.end()) {
    const double f = static_cast<double>(fs) / static_cast<double>(fs + fl);
    if (f > tau_ && fs > 0)
      type = BOOST_KV_SHH;
    else if (fl > 0)
      type = BOOST_KV_LOCAL;
    else
      type = BOOST_KV_SHH;
    it = req_.emplace(rid, Req{type, {}}).first;
  }
  Req& r = it->second;
  for (uint32_t i = 0; i < n; ++i) {
    if (free_[r.type].empty()) r.type ^= 1;  // sticky switch to the other list
    auto first = free_[r.type].begin();
    const int32_t b = *first;
    free_[r.type].erase(first);
    r.blocks.push_back(b);
    out[i] = b;
    used_ += 1;
    used_hh_ += host_heads_[b];
  }
  return BOOST_OK;
}

int Dsr::release(uint64_t rid) {
  auto it = req_.find(rid);
  if (it == req_.end())
    return fail(BOOST_EINVAL, "unknown request %llu", (unsigned long long)rid);
  for (int32_t b : it->second.blocks) {
    free_[is_shh_[b] ? BOOST_KV_SHH : BOOST_KV_LOCAL].insert(b);
    used_ -= 1;
    used_hh_ -= host_heads_[b];
  }
  req_.erase(it);
  return BOOST_OK;
}

int Dsr::type_of(uint64_t rid, int* type) const {
  auto it = req_.find(rid);
  if (it == req_.end() || !type)
    return fail(BOOST_EINVAL, "unknown request %llu", (unsigned long long)rid);
  *type = it->second.type;
  return BOOST_OK;
}

uint32_t Dsr::shh_requests() const {
  uint32_t n = 0;
  for (const auto& kv : req_) n += kv.second.type == BOOST_KV_SHH;
  return n;
}

}  // namespace bst
