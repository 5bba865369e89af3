// Context, memory backend and weight placement (§4.2 PAM design, §4.4 PAM
// implementation).  HBM pages of a tensor share one device slab; host pages
// live in pinned, device-mapped host memory from hipHostMalloc (the MI355X
// counterpart of the paper's mmap + mbind + host registration per 2 MB page);
// a device page table gives every page's device-visible address.
#include <linux/mempolicy.h>
#include <sys/syscall.h>
#include <unistd.h>

#include <algorithm>
#include <cerrno>
#include <cstdio>
#include <cstring>

#include "runtime.h"

namespace bst {

namespace {

// Bits of the node masks passed to the memory-policy calls (the kernel asks
// get_mempolicy for at least its own node count).
constexpr int kMaskWords = 16;
constexpr unsigned long kMaskBits = 64ul * kMaskWords;

// Online host NUMA nodes: a list of ids and ranges ("0", "0-3", "0,2-3").
// Writes whether `node` is online; returns the count (1 when unreadable).
int online_nodes(int node, bool* is_online) {
  if (is_online) *is_online = node == 0;
  FILE* f = std::fopen("/sys/devices/system/node/online", "r");
  if (!f) return 1;
  char buf[256] = {0};
  const bool ok = std::fgets(buf, sizeof buf, f) != nullptr;
  std::fclose(f);
  if (!ok) return 1;
  int count = 0;
  if (is_online) *is_online = false;
  for (char* p = buf; *p && *p != '\n';) {
    char* end = nullptr;
    const long a = std::strtol(p, &end, 10);
    if (end == p) break;
    long b = a;
    p = end;
    if (*p == '-') {
      b = std::strtol(p + 1, &end, 10);
      p = end;
    }
    count += static_cast<int>(b - a + 1);
    if (is_online && node >= a && node <= b) *is_online = true;
    if (*p == ',') ++p;
  }
  return std::max(count, 1);
}

// NUMA node of the GPU's PCIe function (sysfs), -1 when the platform gives
// none.
int device_numa_node(int device) {
  char bus[64] = {0};
  if (device < 0 || hipDeviceGetPCIBusId(bus, sizeof bus, device) != hipSuccess) return -1;
  for (char* c = bus; *c; ++c)
    if (*c >= 'A' && *c <= 'F') *c = static_cast<char>(*c - 'A' + 'a');
  char path[160];
  std::snprintf(path, sizeof path, "/sys/bus/pci/devices/%s/numa_node", bus);
  FILE* f = std::fopen(path, "r");
  if (!f) return -1;
  int node = -1;
  if (std::fscanf(f, "%d", &node) != 1) node = -1;
  std::fclose(f);
  return node;
}

// The calling thread's memory policy, saved around a bound allocation.
struct ThreadPolicy {
  int mode = MPOL_DEFAULT;
  unsigned long mask[kMaskWords] = {};
  bool saved = false;
};

// Bind this thread's page allocations to `node` (§4.4 binds each 2 MiB
// region of the host tier to a chosen node); `old` keeps the policy to put
// back.
int bind_thread(int node, ThreadPolicy& old) {
  if (syscall(SYS_get_mempolicy, &old.mode, old.mask, kMaskBits, nullptr, 0) != 0)
    return fail(BOOST_EINVAL, "get_mempolicy failed (errno %d)", errno);
  old.saved = true;
  unsigned long mask[kMaskWords] = {};
  mask[node / 64] = 1ul << (node % 64);
  if (syscall(SYS_set_mempolicy, MPOL_BIND, mask, kMaskBits) != 0)
    return fail(BOOST_EINVAL, "set_mempolicy(node %d) failed (errno %d)", node, errno);
  return BOOST_OK;
}

void restore_thread(const ThreadPolicy& old) {
  if (!old.saved) return;
  const bool none = (old.mode & ~(MPOL_F_STATIC_NODES | MPOL_F_RELATIVE_NODES)) == MPOL_DEFAULT;
  (void)syscall(SYS_set_mempolicy, old.mode, none ? nullptr : old.mask, none ? 0 : kMaskBits);
}

}  // namespace

int slab_alloc(boost_ctx* ctx, uint64_t pages, bool host, Slab& s) {
  s = Slab{};
  s.pages = pages;
  s.host = host;
  if (pages == 0) return BOOST_OK;
  const size_t bytes = pages * kPage + kPage;  // room to align to 2 MiB
  if (host) {
    if (fault_host_alloc())
      return fail(BOOST_ENOMEM, "host allocation of %llu pages refused (BOOST_FAULT_HOST_ALLOC)",
                  (unsigned long long)pages);
    unsigned flags = hipHostMallocMapped |
                     (ctx->host_coherent ? hipHostMallocCoherent
                                         : hipHostMallocNonCoherent);
    // a chosen node: the pages follow this thread's policy while they are
    // pinned; by default HIP takes the node nearest the GPU
    ThreadPolicy old;
    if (ctx->host_numa >= 0) {
      flags |= hipHostMallocNumaUser;
      const int rc = bind_thread(ctx->host_numa, old);
      if (rc) {
        restore_thread(old);
        return rc;
      }
    }
    hipError_t e = hipHostMalloc(&s.raw, bytes, flags);
    restore_thread(old);
    if (e != hipSuccess || !s.raw)
      return fail(BOOST_ENOMEM, "hipHostMalloc(%zu) failed: %s", bytes,
                  hipGetErrorString(e));
    void* dev = nullptr;
    e = hipHostGetDevicePointer(&dev, s.raw, 0);
    if (e != hipSuccess) {
      (void)hipHostFree(s.raw);
      s.raw = nullptr;
      return fail(BOOST_EHIP, "hipHostGetDevicePointer failed: %s",
                  hipGetErrorString(e));
    }
    uint64_t pad = (kPage - (reinterpret_cast<uintptr_t>(dev) & (kPage - 1))) &
                   (kPage - 1);
    s.base = static_cast<char*>(dev) + pad;
    s.host_base = static_cast<char*>(s.raw) + pad;
  } else {
    hipError_t e = hipMalloc(&s.raw, bytes);
    if (e != hipSuccess || !s.raw)
      return fail(BOOST_ENOMEM, "hipMalloc(%zu) failed: %s", bytes,
                  hipGetErrorString(e));
    uint64_t pad = (kPage - (reinterpret_cast<uintptr_t>(s.raw) & (kPage - 1))) &
                   (kPage - 1);
    s.base = static_cast<char*>(s.raw) + pad;
  }
  return BOOST_OK;
}

void slab_free(Slab& s) {
  if (s.raw) {
    if (s.host)
      (void)hipHostFree(s.raw);
    else
      (void)hipFree(s.raw);
  }
  s = Slab{};
}

static int free_tensor(boost_tensor* t) {
  if (!t) return BOOST_OK;
  if (t->ctx && t->ctx->device >= 0) (void)hipSetDevice(t->ctx->device);
  (void)hipFree(t->d_page_table);
  (void)hipFree(t->d_tiers);
  (void)hipFree(t->d_hbm_pages);
  (void)hipFree(t->d_host_pages);
  (void)hipFree(t->d_partial);
  slab_free(t->hbm);
  slab_free(t->host);
  delete t;
  return BOOST_OK;
}

static int upload(void** dst, const void* src, size_t bytes) {
  if (bytes == 0) bytes = 16;  // keep a valid (unused) pointer
  BOOST_HIP(hipMalloc(dst, bytes));
  if (src) BOOST_HIP(hipMemcpy(*dst, src, bytes, hipMemcpyHostToDevice));
  return BOOST_OK;
}

// The closed form of a tier map that is modulo placement (§3.1): host iff
// (p / SP) % M == M - 1, with SP the first run of host pages and M - 1 the
// superpages before it; M = 0 when no page is on host; M = -1 when the map
// has no such form.
static void modulo_form(const std::vector<uint8_t>& tiers, int32_t& M, int32_t& SP) {
  M = -1;
  SP = 1;
  const uint64_t n = tiers.size();
  uint64_t first = 0;
  while (first < n && tiers[first] != BOOST_TIER_HOST) ++first;
  if (first == n) {
    M = 0;
    return;
  }
  uint64_t run = 0;
  while (first + run < n && tiers[first + run] == BOOST_TIER_HOST) ++run;
  if (first % run != 0 || first / run + 1 > INT32_MAX || run > INT32_MAX) return;
  const uint64_t m = first / run + 1;
  for (uint64_t i = 0; i < n; ++i)
    if ((tiers[i] == BOOST_TIER_HOST) != ((i / run) % m == m - 1)) return;
  M = static_cast<int32_t>(m);
  SP = static_cast<int32_t>(run);
}

static int place(boost_ctx* ctx, const void* src, uint64_t bytes,
                 const uint8_t* tiers, uint64_t n_pages, boost_tensor** out) {
  if (!ctx || !src || !out || !tiers) return fail(BOOST_EINVAL, "null argument");
  if (ctx->device < 0) return fail(BOOST_ENODEV, "plan-only context");
  if (bytes == 0) return fail(BOOST_EINVAL, "tensor of 0 bytes");
  if (n_pages != pages_of(bytes))
    return fail(BOOST_EINVAL, "tier map has %llu pages, tensor needs %llu",
                (unsigned long long)n_pages, (unsigned long long)pages_of(bytes));
  if (n_pages >= (1ull << 31)) return fail(BOOST_EINVAL, "tensor too large");
  BOOST_HIP(hipSetDevice(ctx->device));
  auto* t = new boost_tensor();
  t->ctx = ctx;
  t->bytes = bytes;
  t->n_pages = n_pages;
  t->tiers.assign(tiers, tiers + n_pages);
  for (uint64_t i = 0; i < n_pages; ++i) {
    if (tiers[i] == BOOST_TIER_HBM)
      t->hbm_pages.push_back(static_cast<int32_t>(i));
    else if (tiers[i] == BOOST_TIER_HOST)
      t->host_pages.push_back(static_cast<int32_t>(i));
    else {
      delete t;
      return fail(BOOST_EINVAL, "tier code %u at page %llu", tiers[i],
                  (unsigned long long)i);
    }
  }
  int rc = slab_alloc(ctx, t->hbm_pages.size(), false, t->hbm);
  if (!rc) rc = slab_alloc(ctx, t->host_pages.size(), true, t->host);
  if (rc) {
    free_tensor(t);
    return rc;
  }
  modulo_form(t->tiers, t->lay_M, t->lay_SP);
  t->page_ptr.resize(n_pages);
  t->copy_ptr.resize(n_pages);
  for (size_t i = 0; i < t->hbm_pages.size(); ++i)
    t->page_ptr[t->hbm_pages[i]] = t->copy_ptr[t->hbm_pages[i]] =
        t->hbm.base + i * kPage;
  for (size_t i = 0; i < t->host_pages.size(); ++i) {
    t->page_ptr[t->host_pages[i]] = t->host.base + i * kPage;
    t->copy_ptr[t->host_pages[i]] = t->host.host_base + i * kPage;
  }

  auto done = [&](int code) {
    if (code) free_tensor(t);
    return code;
  };
  // copy the bytes in, page by page; zero the tail of a partial last page
  for (uint64_t i = 0; i < n_pages; ++i) {
    const uint64_t off = i * kPage;
    const uint64_t len = std::min<uint64_t>(kPage, bytes - off);
    hipError_t e = hipMemcpy(t->copy_ptr[i], static_cast<const char*>(src) + off,
                             len, hipMemcpyDefault);
    if (e != hipSuccess)
      return done(fail(BOOST_EHIP, "copy of page %llu failed: %s",
                       (unsigned long long)i, hipGetErrorString(e)));
    if (len < kPage) {
      if (t->tiers[i] == BOOST_TIER_HOST)
        std::memset(t->copy_ptr[i] + len, 0, kPage - len);
      else
        e = hipMemset(t->page_ptr[i] + len, 0, kPage - len);
      if (e != hipSuccess)
        return done(fail(BOOST_EHIP, "hipMemset failed: %s", hipGetErrorString(e)));
    }
  }
  int r = upload(reinterpret_cast<void**>(&t->d_page_table), t->page_ptr.data(),
                 n_pages * sizeof(char*));
  if (!r) r = upload(reinterpret_cast<void**>(&t->d_tiers), t->tiers.data(), n_pages);
  if (!r) r = upload(reinterpret_cast<void**>(&t->d_hbm_pages), t->hbm_pages.data(),
                     t->hbm_pages.size() * sizeof(int32_t));
  if (!r) r = upload(reinterpret_cast<void**>(&t->d_host_pages), t->host_pages.data(),
                     t->host_pages.size() * sizeof(int32_t));
  // split-row scratch: one slot pair per page boundary, zeroed once here
  const size_t nb = n_pages + 1;
  if (!r) r = upload(reinterpret_cast<void**>(&t->d_partial), nullptr,
                     nb * 2 * kMaxGemvBatch * sizeof(float));
  if (r) return done(r);
  hipError_t e = hipMemset(t->d_partial, 0, nb * 2 * kMaxGemvBatch * sizeof(float));
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess)
    return done(fail(BOOST_EHIP, "placement sync failed: %s", hipGetErrorString(e)));
  *out = t;
  return BOOST_OK;
}

}  // namespace bst

using namespace bst;

extern "C" {

int boost_init(int device, boost_ctx** out) {
  if (!out) return fail(BOOST_EINVAL, "null out");
  *out = nullptr;
  auto* c = new boost_ctx();
  if (device >= 0) {
    int n = 0;
    hipError_t e = hipGetDeviceCount(&n);
    if (e != hipSuccess || device >= n) {
      delete c;
      return fail(e != hipSuccess ? BOOST_EHIP : BOOST_EINVAL,
                  "device %d unavailable (%d devices, %s)", device, n,
                  hipGetErrorString(e));
    }
    e = hipSetDevice(device);
    hipDeviceProp_t p;
    if (e == hipSuccess) e = hipGetDeviceProperties(&p, device);
    if (e != hipSuccess) {
      delete c;
      return fail(BOOST_EHIP, "device %d: %s", device, hipGetErrorString(e));
    }
    c->device = device;
    c->n_cu = p.multiProcessorCount;
    c->gemm_ws_floats = kGemmWsFloats;
    e = hipMalloc(&c->gemm_ws, c->gemm_ws_floats * sizeof(float));
    if (e != hipSuccess) {
      delete c;
      return fail(BOOST_ENOMEM, "GEMM workspace: %s", hipGetErrorString(e));
    }
    const int rc = attn_scratch_setup(device);
    if (rc) {
      (void)hipFree(c->gemm_ws);
      delete c;
      return rc;
    }
  } else if (device != -1) {
    delete c;
    return fail(BOOST_EINVAL, "device %d", device);
  }
  *out = c;
  return BOOST_OK;
}

int boost_shutdown(boost_ctx* ctx) {
  if (ctx && ctx->gemm_ws) {
    (void)hipSetDevice(ctx->device);
    (void)hipFree(ctx->gemm_ws);
  }
  delete ctx;
  return BOOST_OK;
}

int boost_ctx_info(const boost_ctx* ctx, int* device, int* n_cu) {
  if (!ctx) return fail(BOOST_EINVAL, "null ctx");
  if (device) *device = ctx->device;
  if (n_cu) *n_cu = ctx->n_cu;
  return BOOST_OK;
}

int boost_set_host_coherent(boost_ctx* ctx, int coherent) {
  if (!ctx) return fail(BOOST_EINVAL, "null ctx");
  ctx->host_coherent = coherent ? 1 : 0;
  return BOOST_OK;
}

int boost_set_host_numa(boost_ctx* ctx, int node) {
  if (!ctx) return fail(BOOST_EINVAL, "null ctx");
  if (node != BOOST_NUMA_DEVICE) {
    bool online = false;
    online_nodes(node, &online);
    if (node < 0 || node >= static_cast<int>(kMaskBits) - 1 || !online)
      return fail(BOOST_EINVAL, "NUMA node %d is not online", node);
  }
  ctx->host_numa = node;
  return BOOST_OK;
}

int boost_host_numa_info(const boost_ctx* ctx, int* device_node, int* n_nodes, int* node) {
  if (!ctx) return fail(BOOST_EINVAL, "null ctx");
  if (device_node) *device_node = device_numa_node(ctx->device);
  if (n_nodes) *n_nodes = online_nodes(-1, nullptr);
  if (node) *node = ctx->host_numa;
  return BOOST_OK;
}

int boost_place_weights(boost_ctx* ctx, const void* src, uint64_t bytes,
                        uint32_t M, uint64_t footprint_bytes, boost_tensor** out) {
  std::vector<uint8_t> tiers;
  int rc = mpp_tiers(bytes, M, footprint_bytes, tiers);
  if (rc) return rc;
  return place(ctx, src, bytes, tiers.data(), tiers.size(), out);
}

int boost_place_weights_map(boost_ctx* ctx, const void* src, uint64_t bytes,
                            const uint8_t* tiers, uint64_t n_pages,
                            boost_tensor** out) {
  return place(ctx, src, bytes, tiers, n_pages, out);
}

int boost_tensor_tiers(const boost_tensor* t, uint8_t* tier_out, uint64_t tier_cap,
                       uint64_t* n_pages) {
  if (!t || !n_pages) return fail(BOOST_EINVAL, "null argument");
  *n_pages = t->n_pages;
  if (tier_out)
    std::memcpy(tier_out, t->tiers.data(), std::min<uint64_t>(tier_cap, t->n_pages));
  return BOOST_OK;
}

int boost_tensor_layout(const boost_tensor* t, int32_t* M, int32_t* SP) {
  if (!t || !M || !SP) return fail(BOOST_EINVAL, "null argument");
  *M = t->lay_M;
  *SP = t->lay_SP;
  return BOOST_OK;
}

int boost_tensor_read(const boost_tensor* t, uint64_t offset, void* dst,
                      uint64_t bytes) {
  if (!t || !dst) return fail(BOOST_EINVAL, "null argument");
  if (offset > t->bytes || bytes > t->bytes - offset)
    return fail(BOOST_EINVAL, "range beyond tensor");
  BOOST_HIP(hipSetDevice(t->ctx->device));
  uint64_t done = 0;
  while (done < bytes) {
    const uint64_t off = offset + done;
    const uint64_t page = off / kPage, in = off % kPage;
    const uint64_t len = std::min(bytes - done, kPage - in);
    BOOST_HIP(hipMemcpy(static_cast<char*>(dst) + done, t->copy_ptr[page] + in, len,
                        hipMemcpyDefault));
    done += len;
  }
  return BOOST_OK;
}

int boost_tensor_free(boost_tensor* t) { return free_tensor(t); }

int boost_staged_view(boost_ctx* ctx, const boost_tensor* t, void* staging,
                      uint64_t staging_bytes, boost_tensor** view) {
  if (!ctx || !t || !view) return fail(BOOST_EINVAL, "null argument");
  if (ctx->device < 0) return fail(BOOST_ENODEV, "plan-only context");
  if (t->staged_from) return fail(BOOST_EINVAL, "cannot stage a staged view");
  const uint64_t need = t->host_pages.size() * kPage;
  if (need && (!staging || staging_bytes < need))
    return fail(BOOST_EINVAL, "staging needs %llu bytes", (unsigned long long)need);
  if (reinterpret_cast<uintptr_t>(staging) & 15)
    return fail(BOOST_EINVAL, "staging must be 16-byte aligned");
  BOOST_HIP(hipSetDevice(ctx->device));
  auto* v = new boost_tensor();
  v->ctx = ctx;
  v->bytes = t->bytes;
  v->n_pages = t->n_pages;
  v->tiers.assign(t->n_pages, BOOST_TIER_HBM);
  v->page_ptr = t->page_ptr;
  v->copy_ptr = t->copy_ptr;
  for (size_t i = 0; i < t->host_pages.size(); ++i) {
    v->page_ptr[t->host_pages[i]] = static_cast<char*>(staging) + i * kPage;
    v->copy_ptr[t->host_pages[i]] = v->page_ptr[t->host_pages[i]];
  }
  for (uint64_t i = 0; i < t->n_pages; ++i) v->hbm_pages.push_back(static_cast<int32_t>(i));
  v->staged_from = t;
  v->stage_src = t->host.host_base;
  v->stage_dst = static_cast<char*>(staging);
  v->stage_bytes = need;
  const size_t nb = t->n_pages + 1;
  int r = upload(reinterpret_cast<void**>(&v->d_page_table), v->page_ptr.data(),
                 v->n_pages * sizeof(char*));
  if (!r) r = upload(reinterpret_cast<void**>(&v->d_tiers), v->tiers.data(), v->n_pages);
  if (!r) r = upload(reinterpret_cast<void**>(&v->d_hbm_pages), v->hbm_pages.data(),
                     v->hbm_pages.size() * sizeof(int32_t));
  if (!r) r = upload(reinterpret_cast<void**>(&v->d_host_pages), nullptr, 0);
  if (!r) r = upload(reinterpret_cast<void**>(&v->d_partial), nullptr,
                     nb * 2 * kMaxGemvBatch * sizeof(float));
  if (r) {
    free_tensor(v);
    return r;
  }
  *view = v;
  return BOOST_OK;
}

int boost_prefetch(boost_ctx* ctx, const boost_tensor* view, void* stream) {
  if (!ctx || !view) return fail(BOOST_EINVAL, "null argument");
  if (!view->staged_from) return fail(BOOST_EINVAL, "not a staged view");
  if (view->stage_bytes == 0) return BOOST_OK;
  BOOST_HIP(hipMemcpyAsync(view->stage_dst, view->stage_src, view->stage_bytes,
                           hipMemcpyHostToDevice, static_cast<hipStream_t>(stream)));
  return BOOST_OK;
}

}  // extern "C"
