// a4: decode GEMV over tiered pages, y[b, n] = sum_k W[n, k] x[b, k].
//
// W is an [N, K] row-major bf16 matrix placed page by page on HBM or host
// (§3.1 modulo placement).  The work unit of a workgroup is a group of rows
// restricted to ONE page, so a workgroup reads one tier for its whole life
// (§3.2 CTA-level confinement: a workgroup never mixes tiers).  A row that
// straddles a page boundary is split-K across the two workgroups of those
// pages; each writes its partial sum and the second to arrive adds them in a
// fixed order (part of the earlier page first), so results are bitwise
// reproducible and independent of the placement.
//
// Schedules (which workgroup takes which unit):
//   address order -- workgroup i takes unit i, blind to tiers (the
//     transparent kernel of §3.1; CAP then depends on where host pages fall);
//   CAP -- the first `host_workers` workgroups (dispatched first, spread over
//     the XCDs) stream all host-page units in a persistent loop while every
//     other workgroup takes one HBM-page unit, so the host link and HBM are
//     busy together in every wave (§3 CAP; §3.2 CTA specialisation).
//
// Inside a unit each wavefront owns RW rows and walks K with 16-byte loads:
// lane l reads columns [8l + 512i, 8l + 512i + 8) of every row, so one load
// instruction of a wavefront covers 1 KiB of one row contiguously.  The x
// chunk is loaded once per column step and reused for the RW rows.  Partial
// sums are reduced across the 64 lanes by a fixed xor butterfly.
#include <algorithm>

#include "runtime.h"

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int64_t kPageElems = static_cast<int64_t>(bst::kPage / 2);

struct GemvParams {
  const char* const* page_table;
  const int32_t* hbm_pages;
  const int32_t* host_pages;
  int n_hbm_pages;
  int n_host_pages;
  int units_per_page;
  int host_workers;
  int address_order;
  int N;
  int K;
  const uint16_t* x;
  void* y;
  int y_bf16;
  float* partial;  // [(n_pages + 1) boundaries][2 sides][kMaxGemvBatch]
  int* flags;      // [(n_pages + 1) boundaries]
};

__device__ __forceinline__ float lo_bf16(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t v) {
  return __uint_as_float(v & 0xffff0000u);
}

__device__ __forceinline__ float dot8(const uint4& w, const uint4& x, float acc) {
  acc = fmaf(lo_bf16(w.x), lo_bf16(x.x), acc);
  acc = fmaf(hi_bf16(w.x), hi_bf16(x.x), acc);
  acc = fmaf(lo_bf16(w.y), lo_bf16(x.y), acc);
  acc = fmaf(hi_bf16(w.y), hi_bf16(x.y), acc);
  acc = fmaf(lo_bf16(w.z), lo_bf16(x.z), acc);
  acc = fmaf(hi_bf16(w.z), hi_bf16(x.z), acc);
  acc = fmaf(lo_bf16(w.w), lo_bf16(x.w), acc);
  acc = fmaf(hi_bf16(w.w), hi_bf16(x.w), acc);
  return acc;
}

// Round-to-nearest-even float -> bf16 bits (finite inputs; NaN kept quiet).
__device__ __forceinline__ uint16_t to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return 0x7fc0;
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}

__device__ __forceinline__ void store_y(const GemvParams& P, int b, int64_t row, float v) {
  const int64_t i = static_cast<int64_t>(b) * P.N + row;
  if (P.y_bf16)
    static_cast<uint16_t*>(P.y)[i] = to_bf16(v);
  else
    static_cast<float*>(P.y)[i] = v;
}

// Combine the two halves of a row split at page boundary `bnd` (between pages
// bnd-1 and bnd).  side 0 = the part in the earlier page.
template <int B>
__device__ void finish_split(const GemvParams& P, int64_t row, int bnd, int side,
                             const float* v) {
  float* slot = P.partial + (static_cast<int64_t>(bnd) * 2 + side) * bst::kMaxGemvBatch;
#pragma unroll
  for (int b = 0; b < B; ++b)
    __hip_atomic_store(slot + b, v[b], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const int prev = __hip_atomic_fetch_add(P.flags + bnd, 1, __ATOMIC_ACQ_REL,
                                          __HIP_MEMORY_SCOPE_AGENT);
  if (prev == 1) {
    const float* s0 = P.partial + static_cast<int64_t>(bnd) * 2 * bst::kMaxGemvBatch;
    const float* s1 = s0 + bst::kMaxGemvBatch;
#pragma unroll
    for (int b = 0; b < B; ++b) {
      const float a0 = __hip_atomic_load(s0 + b, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const float a1 = __hip_atomic_load(s1 + b, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      store_y(P, b, row, a0 + a1);
    }
    __hip_atomic_store(P.flags + bnd, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// One unit: rows [r_first + j*RW*kWaves, ...) of page `page`, restricted to
// the page's bytes.
template <int B, int RW, int UN>
__device__ void gemv_unit(const GemvParams& P, int page, int j) {
  const int64_t K = P.K;
  const int64_t total = static_cast<int64_t>(P.N) * K;
  const int64_t pe0 = static_cast<int64_t>(page) * kPageElems;
  const int64_t pe1 = min(pe0 + kPageElems, total);
  const int64_t r_lo = pe0 / K;
  const int64_t r_hi = (pe1 - 1) / K;  // inclusive
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int64_t r0 = r_lo + static_cast<int64_t>(j) * (RW * kWaves) + wave * RW;
  if (r0 > r_hi) return;

  const char* page_base = P.page_table[page];  // element pe0
  int64_t c0[RW], c1[RW];
  const char* rp[RW];  // address of column 0 of the row (may lie outside the page)
  bool whole = true;
#pragma unroll
  for (int i = 0; i < RW; ++i) {
    const int64_t r = r0 + i;
    const int64_t e0 = r * K;
    if (r <= r_hi) {
      c0[i] = max(static_cast<int64_t>(0), pe0 - e0);
      c1[i] = min(K, pe1 - e0);
    } else {
      c0[i] = 0;
      c1[i] = 0;
    }
    whole = whole && c0[i] == 0 && c1[i] == K;
    rp[i] = page_base + (e0 - pe0) * 2;
  }

  float acc[RW][B];
#pragma unroll
  for (int i = 0; i < RW; ++i)
#pragma unroll
    for (int b = 0; b < B; ++b) acc[i][b] = 0.f;

  const uint4 zero = make_uint4(0, 0, 0, 0);
  const int64_t step = 64 * 8;
  if (whole) {
    // every row of this wavefront lies wholly inside the page
    for (int64_t kb = 0; kb < K; kb += step * UN) {
      uint4 wv[UN][RW], xv[UN][B];
#pragma unroll
      for (int u = 0; u < UN; ++u) {
        const int64_t kc = kb + u * step + lane * 8;
        const bool in = kc < K;
#pragma unroll
        for (int i = 0; i < RW; ++i)
          wv[u][i] = in ? *reinterpret_cast<const uint4*>(rp[i] + kc * 2) : zero;
#pragma unroll
        for (int b = 0; b < B; ++b)
          xv[u][b] = in ? *reinterpret_cast<const uint4*>(P.x + b * K + kc) : zero;
      }
#pragma unroll
      for (int u = 0; u < UN; ++u)
#pragma unroll
        for (int i = 0; i < RW; ++i)
#pragma unroll
          for (int b = 0; b < B; ++b) acc[i][b] = dot8(wv[u][i], xv[u][b], acc[i][b]);
    }
  } else {
    // some row is cut by a page boundary: read only this page's columns;
    // out-of-page lanes load a safe in-page address and contribute zero
    for (int64_t kb = 0; kb < K; kb += step * UN) {
      uint4 wv[UN][RW], xv[UN][B];
#pragma unroll
      for (int u = 0; u < UN; ++u) {
        const int64_t kc = kb + u * step + lane * 8;
        const bool in = kc < K;
#pragma unroll
        for (int i = 0; i < RW; ++i) {
          const bool ok = in && kc >= c0[i] && kc < c1[i];
          wv[u][i] = ok ? *reinterpret_cast<const uint4*>(rp[i] + kc * 2) : zero;
        }
#pragma unroll
        for (int b = 0; b < B; ++b)
          xv[u][b] = in ? *reinterpret_cast<const uint4*>(P.x + b * K + kc) : zero;
      }
#pragma unroll
      for (int u = 0; u < UN; ++u)
#pragma unroll
        for (int i = 0; i < RW; ++i)
#pragma unroll
          for (int b = 0; b < B; ++b) acc[i][b] = dot8(wv[u][i], xv[u][b], acc[i][b]);
    }
  }

#pragma unroll
  for (int i = 0; i < RW; ++i) {
    float v[B];
#pragma unroll
    for (int b = 0; b < B; ++b) v[b] = wave_sum(acc[i][b]);
    const int64_t r = r0 + i;
    if (r > r_hi || lane != 0) continue;
    if (c0[i] == 0 && c1[i] == K) {
#pragma unroll
      for (int b = 0; b < B; ++b) store_y(P, b, r, v[b]);
    } else if (c0[i] > 0) {
      finish_split<B>(P, r, page, 1, v);  // tail of a row begun on page-1
    } else {
      finish_split<B>(P, r, page + 1, 0, v);  // head of a row ending on page+1
    }
  }
}

template <int B, int RW, int UN>
__global__ __launch_bounds__(kThreads) void gemv_kernel(GemvParams P) {
  const int bid = blockIdx.x;
  const int U = P.units_per_page;
  if (P.address_order) {
    gemv_unit<B, RW, UN>(P, bid / U, bid % U);
  } else if (bid < P.host_workers) {
    const int n_host_units = P.n_host_pages * U;
    for (int v = bid; v < n_host_units; v += P.host_workers)
      gemv_unit<B, RW, UN>(P, P.host_pages[v / U], v % U);
  } else {
    const int u = bid - P.host_workers;
    gemv_unit<B, RW, UN>(P, P.hbm_pages[u / U], u % U);
  }
}

template <int B>
struct Shape {
  static constexpr int RW = B <= 2 ? 2 : (B <= 4 ? 2 : 1);
  static constexpr int UN = B <= 2 ? 4 : (B <= 4 ? 2 : 2);
};

template <int B>
int launch(GemvParams& P, int n_pages, const boost_ctx* ctx, hipStream_t s) {
  constexpr int RW = Shape<B>::RW, UN = Shape<B>::UN;
  const int rows_wg = RW * kWaves;
  // units per page: enough for the page that meets the most rows
  const int64_t K = P.K, total = static_cast<int64_t>(P.N) * K;
  int64_t most = 0;
  for (int p = 0; p < n_pages; ++p) {
    const int64_t pe0 = static_cast<int64_t>(p) * kPageElems;
    const int64_t pe1 = std::min(pe0 + kPageElems, total);
    most = std::max(most, (pe1 - 1) / K - pe0 / K + 1);
  }
  P.units_per_page = static_cast<int>((most + rows_wg - 1) / rows_wg);
  int64_t grid;
  if (P.address_order || P.n_host_pages == 0) {
    P.address_order = 1;
    P.host_workers = 0;
    grid = static_cast<int64_t>(n_pages) * P.units_per_page;
  } else {
    const int64_t host_units = static_cast<int64_t>(P.n_host_pages) * P.units_per_page;
    int h = ctx->gemv_host_workers > 0 ? ctx->gemv_host_workers
                                       : std::max(1, ctx->n_cu / 16);
    P.host_workers = static_cast<int>(std::min<int64_t>(h, host_units));
    grid = P.host_workers + static_cast<int64_t>(P.n_hbm_pages) * P.units_per_page;
  }
  if (grid > 0x7fffffff) return bst::fail(BOOST_EINVAL, "grid too large");
  hipLaunchKernelGGL((gemv_kernel<B, RW, UN>), dim3(static_cast<unsigned>(grid)),
                     dim3(kThreads), 0, s, P);
  BOOST_HIP(hipGetLastError());
  return BOOST_OK;
}

}  // namespace

using namespace bst;

extern "C" {

int boost_gemv_set_schedule(boost_ctx* ctx, int schedule, int host_workers) {
  if (!ctx) return fail(BOOST_EINVAL, "null ctx");
  if (schedule != BOOST_SCHED_ADDRESS && schedule != BOOST_SCHED_CAP)
    return fail(BOOST_EINVAL, "schedule %d", schedule);
  if (host_workers < 0) return fail(BOOST_EINVAL, "host_workers %d", host_workers);
  ctx->gemv_schedule = schedule;
  ctx->gemv_host_workers = host_workers;
  return BOOST_OK;
}

int boost_decode_gemv(boost_ctx* ctx, const boost_tensor* W, int N, int K, const void* x,
                      int B, void* y, int y_dtype, void* stream) {
  if (!ctx || !W || !x || !y) return fail(BOOST_EINVAL, "null argument");
  if (ctx->device < 0) return fail(BOOST_ENODEV, "plan-only context");
  if (N < 1 || K < 8 || K % 8) return fail(BOOST_EINVAL, "N=%d K=%d (K %% 8 == 0)", N, K);
  if (static_cast<uint64_t>(K) * 2 > kPage)
    return fail(BOOST_EINVAL, "row of %d elements exceeds a page", K);
  if (B < 1 || B > kMaxGemvBatch) return fail(BOOST_EINVAL, "B=%d outside [1, 8]", B);
  if (y_dtype != BOOST_DTYPE_F32 && y_dtype != BOOST_DTYPE_BF16)
    return fail(BOOST_EINVAL, "y_dtype %d", y_dtype);
  if (static_cast<uint64_t>(N) * K * 2 != W->bytes)
    return fail(BOOST_EINVAL, "N*K*2=%llu but tensor holds %llu bytes",
                (unsigned long long)(static_cast<uint64_t>(N) * K * 2),
                (unsigned long long)W->bytes);
  if ((reinterpret_cast<uintptr_t>(x) & 15) || (reinterpret_cast<uintptr_t>(y) & 3))
    return fail(BOOST_EINVAL, "x must be 16-byte and y 4-byte aligned");
  GemvParams P{};
  P.page_table = W->d_page_table;
  P.hbm_pages = W->d_hbm_pages;
  P.host_pages = W->d_host_pages;
  P.n_hbm_pages = static_cast<int>(W->hbm_pages.size());
  P.n_host_pages = static_cast<int>(W->host_pages.size());
  P.address_order = ctx->gemv_schedule == BOOST_SCHED_ADDRESS;
  P.N = N;
  P.K = K;
  P.x = static_cast<const uint16_t*>(x);
  P.y = y;
  P.y_bf16 = y_dtype == BOOST_DTYPE_BF16;
  P.partial = W->d_partial;
  P.flags = W->d_flags;
  auto s = static_cast<hipStream_t>(stream);
  const int n = static_cast<int>(W->n_pages);
  switch (B) {
    case 1: return launch<1>(P, n, ctx, s);
    case 2: return launch<2>(P, n, ctx, s);
    case 3: return launch<3>(P, n, ctx, s);
    case 4: return launch<4>(P, n, ctx, s);
    case 5: return launch<5>(P, n, ctx, s);
    case 6: return launch<6>(P, n, ctx, s);
    case 7: return launch<7>(P, n, ctx, s);
    default: return launch<8>(P, n, ctx, s);
  }
}

}  // extern "C"
