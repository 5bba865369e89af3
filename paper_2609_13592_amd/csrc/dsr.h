// KV pool geometry (linear page placement with heads outermost) and the
// wave-aware block allocator.  CPU only.
#pragma once
#include <cstdint>
#include <set>
#include <unordered_map>
#include <vector>

#include "common.h"

namespace bst {

struct KvGeom {
  uint32_t H = 0, D = 0, T = 0;
  uint32_t blocks_per_page = 0;  // head-blocks of T*D bf16 per page
  uint32_t nb = 0;               // pool blocks, a multiple of blocks_per_page
  uint64_t pages = 0;            // pages of one K (or V) tensor: H * nb / bpp
  uint64_t host_pages = 0;       // tail pages on host
  std::vector<uint8_t> host_heads;  // per block
  uint8_t hi = 0, lo = 0;        // host-head counts of the SHH / local lists
  uint32_t n_shh = 0;
};

// Geometry of §4.2 / §4.5: every head's region is whole pages; the last
// `host_pages` pages of a tensor are on host (1/M of them for LPP; all pages
// past a per-tensor share of hbm_budget_bytes over `layers` layers of K and V
// for BOOST_KV_BUDGET).
int kv_geometry(uint32_t n_blocks, uint32_t H, uint32_t D, uint32_t T, uint32_t M,
                int mode, uint32_t layers, uint64_t hbm_budget_bytes, KvGeom& g);

// §4.3 wave-aware block fulfillment over two free lists.
class Dsr {
 public:
  void init(const KvGeom& g);
  int alloc(uint64_t rid, uint32_t n, int32_t* out);
  int release(uint64_t rid);
  int type_of(uint64_t rid, int* type) const;
  uint32_t free_shh() const { return static_cast<uint32_t>(free_[1].size()); }
  uint32_t free_local() const { return static_cast<uint32_t>(free_[0].size()); }
  uint64_t used_blocks() const { return used_; }
  uint64_t used_host_head_blocks() const { return used_hh_; }
  uint32_t requests() const { return static_cast<uint32_t>(req_.size()); }
  uint32_t shh_requests() const;
  double tau() const { return tau_; }

 private:
  struct Req {
    int type = 0;
    std::vector<int32_t> blocks;
  };
  std::set<int32_t> free_[2];  // [BOOST_KV_LOCAL], [BOOST_KV_SHH]
  std::vector<uint8_t> is_shh_, host_heads_;
  std::unordered_map<uint64_t, Req> req_;
  double tau_ = 0.0;
  uint64_t used_ = 0, used_hh_ = 0;
};

}  // namespace bst
