// KV pool (§4.2 LPP, §4.5 heads-outermost layout and two free lists) and the
// KV write kernel.  Every layer has a K and a V tensor [H][NB][T][D] bf16;
// the LPP tail pages of each tensor live in pinned host memory, the rest in
// one HBM slab; the device page table maps (layer, K/V, page) to an address.
#include <algorithm>
#include <cstring>
#include <new>

#include "runtime.h"

namespace {

constexpr int kPartTokensMin = 64;  // smallest attention partition (4 blocks)

// One lane per 16 bytes of one (token, head) row of K and of V.
__global__ __launch_bounds__(256) void kv_write_kernel(
    const char* const* __restrict__ pt_k, const char* const* __restrict__ pt_v,
    const int32_t* __restrict__ slots, const uint4* __restrict__ k,
    const uint4* __restrict__ v, int n, int H, int D, int T, int nb) {
  const int chunks = D / 8;  // 16-byte chunks per head row
  const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t total = static_cast<int64_t>(n) * H * chunks;
  if (t >= total) return;
  const int c = static_cast<int>(t % chunks);
  const int64_t th = t / chunks;  // token * H + head
  const int h = static_cast<int>(th % H);
  const int64_t i = th / H;
  const int32_t slot = slots[i];
  if (slot < 0 || slot >= static_cast<int64_t>(nb) * T) return;
  const int32_t blk = slot / T, off = slot % T;
  const uint64_t byte = ((static_cast<uint64_t>(h) * nb + blk) * T + off) * D * 2 +
                        static_cast<uint64_t>(c) * 16;
  const uint64_t page = byte >> 21, in = byte & (bst::kPage - 1);
  *reinterpret_cast<uint4*>(const_cast<char*>(pt_k[page]) + in) = k[t];
  *reinterpret_cast<uint4*>(const_cast<char*>(pt_v[page]) + in) = v[t];
}

int destroy(boost_kv_pool* p) {
  if (!p) return BOOST_OK;
  if (p->ctx && p->ctx->device >= 0) (void)hipSetDevice(p->ctx->device);
  (void)hipFree(p->d_page_table);
  (void)hipFree(p->d_part_acc);
  (void)hipFree(p->d_part_ml);
  bst::slab_free(p->hbm);
  for (auto& h : p->host) bst::slab_free(h);
  delete p;
  return BOOST_OK;
}

}  // namespace

namespace bst {
int kv_parts_for(const boost_kv_pool* p, int max_blocks) {
  const int tokens = max_blocks * static_cast<int>(p->cfg.block_tokens);
  return std::max(1, (tokens + kPartTokensMin - 1) / kPartTokensMin);
}
}  // namespace bst

using namespace bst;

extern "C" {

int boost_kv_pool_create(boost_ctx* ctx, const boost_kv_cfg* cfg, boost_kv_pool** out) {
  if (!ctx || !cfg || !out) return fail(BOOST_EINVAL, "null argument");
  *out = nullptr;
  if (cfg->layers == 0) return fail(BOOST_EINVAL, "0 layers");
  if (cfg->block_tokens != 16) return fail(BOOST_EINVAL, "block_tokens must be 16");
  if (cfg->head_dim != 64 && cfg->head_dim != 128)
    return fail(BOOST_EINVAL, "head_dim must be 64 or 128");
  if (cfg->kv_heads == 0) return fail(BOOST_EINVAL, "0 kv_heads");
  if (cfg->q_heads == 0 || cfg->q_heads % cfg->kv_heads || cfg->q_heads / cfg->kv_heads > 16)
    return fail(BOOST_EINVAL, "q_heads %u must be a multiple of kv_heads %u (ratio <= 16)",
                cfg->q_heads, cfg->kv_heads);
  boost_kv_pool* p = nullptr;
  try {  // host-side allocator state: per-block host heads and the two free lists
    if (fault_host_alloc()) throw std::bad_alloc();
    p = new boost_kv_pool();
    p->ctx = ctx;
    p->cfg = *cfg;
    int rc = kv_geometry(cfg->n_blocks, cfg->kv_heads, cfg->head_dim, cfg->block_tokens,
                         cfg->M, cfg->tier_mode, cfg->layers, cfg->hbm_budget_bytes, p->geom);
    if (rc) {
      delete p;
      return rc;
    }
    p->dsr.init(p->geom);
  } catch (const std::bad_alloc&) {
    delete p;
    return fail(BOOST_ENOMEM, "KV pool: host memory for the allocator state");
  }
  int rc = BOOST_OK;
  if (ctx->device < 0) {  // plan-only: allocator bookkeeping only
    *out = p;
    return BOOST_OK;
  }
  if (cfg->max_batch == 0 || cfg->max_blocks_per_seq == 0) {
    delete p;
    return fail(BOOST_EINVAL, "max_batch and max_blocks_per_seq must be > 0");
  }
  if (hipSetDevice(ctx->device) != hipSuccess) {
    delete p;
    return fail(BOOST_EHIP, "hipSetDevice failed");
  }
  const uint64_t tensors = 2ull * cfg->layers;
  const uint64_t P = p->geom.pages, Hp = p->geom.host_pages;
  // one HBM slab for every tensor's HBM pages; the host tails in one pinned
  // slab per layer (K's tail then V's), which keeps each pinned allocation a
  // few GB even when most of a large pool lives on host
  rc = slab_alloc(ctx, tensors * (P - Hp), false, p->hbm);
  if (!rc && Hp) {
    p->host.resize(cfg->layers);
    for (uint32_t l = 0; l < cfg->layers && !rc; ++l)
      rc = slab_alloc(ctx, 2 * Hp, true, p->host[l]);
  }
  if (rc) {
    destroy(p);
    return rc;
  }
  std::vector<char*> table(tensors * P);
  for (uint64_t t = 0; t < tensors; ++t)
    for (uint64_t pg = 0; pg < P; ++pg)
      table[t * P + pg] = pg < P - Hp
                              ? p->hbm.base + (t * (P - Hp) + pg) * kPage
                              : p->host[t / 2].base + ((t % 2) * Hp + (pg - (P - Hp))) * kPage;
  p->max_parts = kv_parts_for(p, static_cast<int>(cfg->max_blocks_per_seq));
  const uint64_t rows = static_cast<uint64_t>(cfg->max_batch) * cfg->q_heads * p->max_parts;
  hipError_t e = hipMalloc(&p->d_page_table, table.size() * sizeof(char*));
  if (e == hipSuccess)
    e = hipMemcpy(p->d_page_table, table.data(), table.size() * sizeof(char*),
                  hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMalloc(&p->d_part_acc, rows * cfg->head_dim * sizeof(float));
  if (e == hipSuccess) e = hipMalloc(&p->d_part_ml, rows * 2 * sizeof(float));
  // zero the pool so unwritten slots hold defined values
  if (e == hipSuccess && p->hbm.pages) e = hipMemset(p->hbm.base, 0, p->hbm.pages * kPage);
  for (auto& h : p->host)
    if (e == hipSuccess) std::memset(h.host_base, 0, h.pages * kPage);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    destroy(p);
    return fail(e == hipErrorOutOfMemory ? BOOST_ENOMEM : BOOST_EHIP, "KV pool: %s",
                hipGetErrorString(e));
  }
  *out = p;
  return BOOST_OK;
}

int boost_kv_pool_info(const boost_kv_pool* p, boost_kv_info* info) {
  if (!p || !info) return fail(BOOST_EINVAL, "null argument");
  info->nb_pool = p->geom.nb;
  info->blocks_per_page = p->geom.blocks_per_page;
  info->pages_per_tensor = p->geom.pages;
  info->host_pages_per_tensor = p->geom.host_pages;
  info->n_shh = p->geom.n_shh;
  info->shh_host_heads = p->geom.hi;
  info->local_host_heads = p->geom.lo;
  info->tau = p->dsr.tau();
  return BOOST_OK;
}

int boost_kv_pool_destroy(boost_kv_pool* p) { return destroy(p); }

int boost_kv_block_host_heads(const boost_kv_pool* p, int32_t block, uint32_t* n) {
  if (!p || !n) return fail(BOOST_EINVAL, "null argument");
  if (block < 0 || static_cast<uint32_t>(block) >= p->geom.nb)
    return fail(BOOST_EINVAL, "block %d outside the pool", block);
  *n = p->geom.host_heads[block];
  return BOOST_OK;
}

int boost_kv_alloc(boost_kv_pool* p, uint64_t rid, uint32_t n, int32_t* out) {
  if (!p) return fail(BOOST_EINVAL, "null pool");
  return p->dsr.alloc(rid, n, out);
}

int boost_kv_free(boost_kv_pool* p, uint64_t rid) {
  if (!p) return fail(BOOST_EINVAL, "null pool");
  return p->dsr.release(rid);
}

int boost_kv_request_type(const boost_kv_pool* p, uint64_t rid, int* type) {
  if (!p) return fail(BOOST_EINVAL, "null pool");
  return p->dsr.type_of(rid, type);
}

int boost_kv_stats(const boost_kv_pool* p, boost_kv_usage* s) {
  if (!p || !s) return fail(BOOST_EINVAL, "null argument");
  s->free_shh = p->dsr.free_shh();
  s->free_local = p->dsr.free_local();
  s->used_blocks = p->dsr.used_blocks();
  s->used_host_head_blocks = p->dsr.used_host_head_blocks();
  s->requests = p->dsr.requests();
  s->shh_requests = p->dsr.shh_requests();
  return BOOST_OK;
}

int boost_kv_write(boost_ctx* ctx, const boost_kv_pool* p, int layer, const int32_t* slots,
                   const void* k, const void* v, int n, void* stream) {
  if (!ctx || !p || !slots || !k || !v) return fail(BOOST_EINVAL, "null argument");
  if (ctx->device < 0 || !p->d_page_table) return fail(BOOST_ENODEV, "plan-only pool");
  if (layer < 0 || static_cast<uint32_t>(layer) >= p->cfg.layers)
    return fail(BOOST_EINVAL, "layer %d", layer);
  if (n < 0) return fail(BOOST_EINVAL, "n=%d", n);
  if (n == 0) return BOOST_OK;
  if ((reinterpret_cast<uintptr_t>(k) | reinterpret_cast<uintptr_t>(v)) & 15)
    return fail(BOOST_EINVAL, "k and v must be 16-byte aligned");
  const uint64_t P = p->geom.pages;
  const char* const* pk = p->d_page_table + (2ull * layer) * P;
  const char* const* pv = p->d_page_table + (2ull * layer + 1) * P;
  const int64_t total = static_cast<int64_t>(n) * p->cfg.kv_heads * (p->cfg.head_dim / 8);
  hipLaunchKernelGGL(kv_write_kernel, dim3(static_cast<unsigned>((total + 255) / 256)),
                     dim3(256), 0, static_cast<hipStream_t>(stream), pk, pv, slots,
                     static_cast<const uint4*>(k), static_cast<const uint4*>(v), n,
                     static_cast<int>(p->cfg.kv_heads), static_cast<int>(p->cfg.head_dim),
                     static_cast<int>(p->cfg.block_tokens), static_cast<int>(p->geom.nb));
  BOOST_HIP(hipGetLastError());
  return BOOST_OK;
}

}  // extern "C"
