// Library-internal state shared by the HIP translation units.
#pragma once
#include <hip/hip_runtime.h>

#include "common.h"

#define BOOST_HIP(call)                                                     \
  do {                                                                      \
    hipError_t e_ = (call);                                                 \
    if (e_ != hipSuccess)                                                   \
      return bst::fail(BOOST_EHIP, "%s failed: %s (%s:%d)", #call,          \
                       hipGetErrorString(e_), __FILE__, __LINE__);          \
  } while (0)

struct boost_ctx {
  int device = -1;          // -1: plan-only
  int n_cu = 0;
  int host_coherent = 1;
  int host_numa = BOOST_NUMA_DEVICE;  // node that host-tier pages are bound to
  int gemv_schedule = BOOST_SCHED_CAP;
  int gemv_host_workers = 0;  // 0: default
  // split-K partials of the matrix-core GEMM (slices of K run by different
  // workgroups; a second kernel sums them in slice order)
  float* gemm_ws = nullptr;
  uint64_t gemm_ws_floats = 0;
};

namespace bst {

// One allocation that backs whole pages of one tier.
struct Slab {
  void* raw = nullptr;      // what hipMalloc / hipHostMalloc returned
  char* base = nullptr;     // device-visible, 2 MiB aligned
  char* host_base = nullptr;  // host-visible (host tier only)
  uint64_t pages = 0;
  bool host = false;
};

int slab_alloc(boost_ctx* ctx, uint64_t pages, bool host, Slab& s);
void slab_free(Slab& s);

// Device address of the attention's static scratch on `device` (the device
// current), looked up once per device; boost_init calls it.
int attn_scratch_setup(int device);

}  // namespace bst

struct boost_tensor {
  boost_ctx* ctx = nullptr;
  uint64_t bytes = 0;
  uint64_t n_pages = 0;
  std::vector<uint8_t> tiers;
  std::vector<char*> page_ptr;          // device-visible address per page
  std::vector<char*> copy_ptr;          // address for host-side copies
  std::vector<int32_t> hbm_pages, host_pages;
  bst::Slab hbm, host;
  // the map in closed form when it is modulo placement: page p on host iff
  // (p / lay_SP) % lay_M == lay_M - 1 (lay_M = 0: every page in HBM), each
  // tier's pages in page order in its slab; lay_M < 0: no closed form (the
  // kernels read the tables)
  int32_t lay_M = -1, lay_SP = 1;
  // device-side copies
  char** d_page_table = nullptr;        // [n_pages]
  uint8_t* d_tiers = nullptr;           // [n_pages] tier codes
  int32_t* d_hbm_pages = nullptr;       // HBM page ids, ascending
  int32_t* d_host_pages = nullptr;      // host page ids, ascending
  float* d_partial = nullptr;           // split-row partial sums
  // staged views (prefetch baseline): source host pages and their staging
  const boost_tensor* staged_from = nullptr;
  const char* stage_src = nullptr;      // host VA of the source's host pages
  char* stage_dst = nullptr;            // device staging area
  uint64_t stage_bytes = 0;
};

namespace bst {
constexpr int kMaxGemvBatch = 256;   // largest B of boost_decode_gemv
constexpr uint64_t kGemmWsFloats = 16ull << 20;  // split-K workspace per context (64 MiB)
}

#include "dsr.h"

struct boost_kv_pool {
  boost_ctx* ctx = nullptr;
  boost_kv_cfg cfg{};
  bst::KvGeom geom;
  bst::Dsr dsr;
  // device backing (absent on a plan-only context)
  bst::Slab hbm;
  std::vector<bst::Slab> host;    // per layer: K's host tail, then V's
  char** d_page_table = nullptr;  // [layers][2 (K, V)][pages]
  float* d_part_acc = nullptr;    // [max_batch][q_heads][max_parts][D]
  float* d_part_ml = nullptr;     // [max_batch][q_heads][max_parts][2] (max, sum)
  int max_parts = 0;
};
