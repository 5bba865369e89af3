// Placement engine (CPU only): modulus from the bandwidth ratio, modulo page
// placement over superpages with per-tensor restart, modulus under an HBM
// budget.  Follows §3.1 (modulo placement, per-tensor allocation), §3.2 and
// §4.4 (superpages of lcm(CTA footprint, page); ceil rule).  Contrast
// placements for the comparisons of §2.6 and §5.7: modulo placement without
// the per-tensor restart, a linear split, and random (BAPP-R) placement.
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <numeric>
#include <unordered_map>

#include "common.h"

namespace bst {

static thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

void clear_error() { g_err.clear(); }

uint64_t pages_of(uint64_t bytes) { return (bytes + kPage - 1) / kPage; }

bool fault_host_alloc() {
  const char* e = std::getenv("BOOST_FAULT_HOST_ALLOC");
  return e && std::strtol(e, nullptr, 10) != 0;
}

static uint64_t superpage(uint64_t footprint) {
  if (footprint == 0) return 1;
  // lcm(footprint, page) / page = footprint / gcd(footprint, page)
  uint64_t g = std::gcd(footprint, kPage);
  return footprint / g;
}

int mpp_tiers(uint64_t bytes, uint32_t M, uint64_t footprint,
              std::vector<uint8_t>& tiers) {
  if (bytes == 0) return fail(BOOST_EINVAL, "tensor of 0 bytes");
  if (M < 2) return fail(BOOST_EINVAL, "modulus M=%u < 2", M);
  const uint64_t n = pages_of(bytes);
  const uint64_t S = superpage(footprint);
  tiers.assign(n, BOOST_TIER_HBM);
  // superpage j is host-resident iff j mod M == M-1; the pattern restarts at
  // page 0 of every tensor
  for (uint64_t j = M - 1; j * S < n; j += M)
    for (uint64_t i = j * S; i < n && i < (j + 1) * S; ++i)
      tiers[i] = BOOST_TIER_HOST;
  return BOOST_OK;
}

}  // namespace bst

using namespace bst;

extern "C" {

const char* boost_last_error(void) { return g_err.c_str(); }

int boost_version(void) { return 100; }

int boost_modulus_from_alpha(double alpha, uint32_t* M) {
  if (!M) return fail(BOOST_EINVAL, "null M");
  if (!(alpha > 0.0 && alpha <= 1.0))
    return fail(BOOST_EINVAL, "alpha=%g outside (0, 1]", alpha);
  // K = ceil(1/alpha); the guard keeps 1/0.1 from landing just above 10
  const double k = std::ceil(1.0 / alpha - 1e-9);
  if (k > 4.0e9) return fail(BOOST_EINVAL, "alpha=%g too small", alpha);
  *M = static_cast<uint32_t>(k) + 1u;
  return BOOST_OK;
}

int boost_superpage_pages(uint64_t footprint_bytes, uint32_t* S) {
  if (!S) return fail(BOOST_EINVAL, "null S");
  uint64_t s = superpage(footprint_bytes);
  if (s > 0xffffffffull) return fail(BOOST_EINVAL, "superpage too large");
  *S = static_cast<uint32_t>(s);
  return BOOST_OK;
}

int boost_plan_mpp(uint64_t bytes, uint32_t M, uint64_t footprint_bytes,
                   uint8_t* tier_out, uint64_t tier_cap, uint64_t* n_pages) {
  if (!n_pages) return fail(BOOST_EINVAL, "null n_pages");
  std::vector<uint8_t> t;
  int rc = mpp_tiers(bytes, M, footprint_bytes, t);
  if (rc) return rc;
  *n_pages = t.size();
  if (tier_out) std::memcpy(tier_out, t.data(), std::min<uint64_t>(tier_cap, t.size()));
  return BOOST_OK;
}

int boost_plan_contrast(int kind, uint64_t bytes, uint32_t M, uint64_t phase,
                        const double* uniforms, uint8_t* tier_out, uint64_t tier_cap,
                        uint64_t* n_pages) {
  if (!n_pages) return fail(BOOST_EINVAL, "null n_pages");
  if (bytes == 0) return fail(BOOST_EINVAL, "tensor of 0 bytes");
  if (M < 2) return fail(BOOST_EINVAL, "modulus M=%u < 2", M);
  const uint64_t n = pages_of(bytes);
  std::vector<uint8_t> t(n, BOOST_TIER_HBM);
  switch (kind) {
    case BOOST_PLACE_MPP: {
      int rc = mpp_tiers(bytes, M, 0, t);
      if (rc) return rc;
      break;
    }
    case BOOST_PLACE_MPP_GLOBAL:
      // the modulo pattern runs on over the pages of earlier tensors: the
      // page with global index phase + i is on host iff that index is the
      // last of its group of M
      for (uint64_t i = 0; i < n; ++i)
        if ((phase + i) % M == M - 1) t[i] = BOOST_TIER_HOST;
      break;
    case BOOST_PLACE_LINEAR:
      // the first pages in HBM, the last floor(n / M) on host
      for (uint64_t i = n - n / M; i < n; ++i) t[i] = BOOST_TIER_HOST;
      break;
    case BOOST_PLACE_RANDOM:
      if (!uniforms) return fail(BOOST_EINVAL, "random placement needs n uniforms");
      // each page on host with probability 1/M, decided by the caller's draw
      for (uint64_t i = 0; i < n; ++i)
        if (uniforms[i] * M < 1.0) t[i] = BOOST_TIER_HOST;
      break;
    default:
      return fail(BOOST_EINVAL, "placement kind %d", kind);
  }
  *n_pages = n;
  if (tier_out) std::memcpy(tier_out, t.data(), std::min<uint64_t>(tier_cap, n));
  return BOOST_OK;
}

int boost_modulus_from_budget(const uint64_t* tensor_bytes,
                              const uint64_t* footprints, size_t n_tensors,
                              uint64_t hbm_budget_bytes, uint32_t M_alpha,
                              uint32_t* M) {
  if (!tensor_bytes || !M || n_tensors == 0)
    return fail(BOOST_EINVAL, "null or empty tensor list");
  if (M_alpha < 2) return fail(BOOST_EINVAL, "M_alpha=%u < 2", M_alpha);
  // HBM pages of a tensor under modulus M: n - (pages of host superpages).
  // Distinct (bytes, footprint) pairs are few, so count per pair.
  struct Key {
    uint64_t b, f;
    bool operator==(const Key& o) const { return b == o.b && f == o.f; }
  };
  struct H {
    size_t operator()(const Key& k) const { return k.b * 1315423911u ^ k.f; }
  };
  std::unordered_map<Key, uint64_t, H> mult;
  uint64_t most_sp = 0;
  for (size_t t = 0; t < n_tensors; ++t) {
    if (tensor_bytes[t] == 0) return fail(BOOST_EINVAL, "tensor %zu has 0 bytes", t);
    Key k{tensor_bytes[t], footprints ? footprints[t] : 0};
    mult[k] += 1;
    uint64_t S = superpage(k.f);
    most_sp = std::max(most_sp, (pages_of(k.b) + S - 1) / S);
  }
  // beyond the largest superpage count every M gives the all-HBM map
  uint64_t start = std::min<uint64_t>(M_alpha, most_sp + 1);
  for (uint64_t m = start; m >= 2; --m) {
    uint64_t hbm_pages = 0;
    for (auto& kv : mult) {
      const uint64_t n = pages_of(kv.first.b);
      const uint64_t S = superpage(kv.first.f);
      uint64_t host = 0;
      for (uint64_t j = m - 1; j * S < n; j += m) host += std::min(S, n - j * S);
      hbm_pages += (n - host) * kv.second;
    }
    if (hbm_pages * kPage <= hbm_budget_bytes) {
      *M = static_cast<uint32_t>(m);
      return BOOST_OK;
    }
  }
  return fail(BOOST_ENOMEM, "HBM budget %llu B is below the M=2 placement",
              (unsigned long long)hbm_budget_bytes);
}

}  // extern "C"
