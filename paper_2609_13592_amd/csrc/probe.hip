// a0: per-tier streaming read probe and calibration of alpha (§2.3 defines
// alpha as host read bandwidth over HBM read bandwidth; §5.1 measures each
// tier's peak on its own).  One kernel streams a buffer with 16-byte loads;
// pointed at device memory it measures HBM, pointed at pinned device-mapped
// host memory it measures the PCIe host link.
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <vector>

#include "runtime.h"

namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 8;

// Stream one contiguous slice (part of `parts`) of n_vec 16-byte vectors:
// lanes stride by 256 vectors so a wavefront's 64 lanes cover 1 KiB
// contiguous per load.  Loads are raw buffer loads with the non-temporal
// policy, exactly as the decode kernels stream their operands, so alpha is
// the ratio the kernels can actually reach.  A slice is at most 2 GiB (the
// 32-bit buffer offset; checked on the host).  Returns the XOR of every word,
// which the callers store only when it equals a magic value: that keeps the
// loads alive without a data-dependent store in practice.
__device__ __forceinline__ uint32_t stream_slice(const char* src, uint64_t n_vec, int part,
                                                 int parts) {
  const uint64_t per = (n_vec + parts - 1) / parts;
  const uint64_t beg = static_cast<uint64_t>(part) * per;
  const uint64_t end = beg + per < n_vec ? beg + per : n_vec;
  uint32_t acc = 0;
  if (beg >= end) return acc;
  const uint64_t span = (end - beg) * 16;  // < 2^31, checked on the host
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<char*>(src) + beg * 16, 0, static_cast<int>(span), 0x00020000);
  const uint32_t n = static_cast<uint32_t>(end - beg);
  uint32_t i = threadIdx.x;
  for (; i + (kUnroll - 1) * kThreads < n; i += kUnroll * kThreads) {
    uint4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      auto t = __builtin_amdgcn_raw_buffer_load_b128(r, (i + u * kThreads) * 16, 0, 2);
      v[u] = *reinterpret_cast<uint4*>(&t);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < n; i += kThreads) {
    auto t = __builtin_amdgcn_raw_buffer_load_b128(r, i * 16, 0, 2);
    uint4 v = *reinterpret_cast<uint4*>(&t);
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  return acc;
}

__global__ __launch_bounds__(kThreads) void stream_read(const char* __restrict__ src,
                                                        uint64_t n_vec,
                                                        uint32_t* __restrict__ sink) {
  const uint32_t acc = stream_slice(src, n_vec, blockIdx.x, gridDim.x);
  if (acc == 0x9e3779b9u) sink[blockIdx.x] = acc;
}

// Concurrent two-tier stream (the streaming probe behind the CAP bound of §3:
// a fixed set of workgroups reads the host tier while the others read HBM).
// The host workgroups are the first host_wgs multiples of host_stride
// (stride 1: the first host_wgs workgroups; stride 8: workgroups 0, 8, 16,
// ..., which the dispatcher places on one XCD when it deals workgroups to
// the 8 XCDs in turn); they split the host buffer into contiguous slices and
// the others split the HBM buffer; both walk their slice exactly as
// stream_read does.  Thread 0 of every workgroup stores the constant-rate
// clock at its start and after its last load returned, so the host can tell
// when each tier's workgroups finished inside the one launch.
__global__ __launch_bounds__(kThreads) void cap_stream(const char* __restrict__ hbm,
                                                       uint64_t hbm_vec,
                                                       const char* __restrict__ host,
                                                       uint64_t host_vec, int host_wgs,
                                                       int host_stride,
                                                       uint64_t* __restrict__ clocks,
                                                       uint32_t* __restrict__ sink) {
  const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
  const int bid = blockIdx.x;
  // HBM workgroups are numbered in order around the host ones: bid minus
  // the host workgroups before it
  const bool is_host = bid % host_stride == 0 && bid / host_stride < host_wgs;
  const int hosts_before = min(host_wgs, (bid + host_stride - 1) / host_stride);
  const uint32_t acc = is_host
                           ? stream_slice(host, host_vec, bid / host_stride, host_wgs)
                           : stream_slice(hbm, hbm_vec, bid - hosts_before,
                                          static_cast<int>(gridDim.x) - host_wgs);
  __syncthreads();  // every wavefront's loads returned (their values were used)
  if (threadIdx.x == 0) {
    clocks[2 * bid] = t0;
    clocks[2 * bid + 1] = __builtin_amdgcn_s_memrealtime();
  }
  if (acc == 0x9e3779b9u) sink[bid] = acc;
}

int measure(const void* src, uint64_t bytes, int grid, int iters, uint32_t* sink,
            double* gbps) {
  hipEvent_t a, b;
  BOOST_HIP(hipEventCreate(&a));
  BOOST_HIP(hipEventCreate(&b));
  const uint64_t n_vec = bytes / 16;
  if ((n_vec + grid - 1) / grid * 16 >= (1ull << 31))
    return bst::fail(BOOST_EINVAL, "slice per workgroup exceeds 2 GiB; raise the grid");
  hipLaunchKernelGGL(stream_read, dim3(grid), dim3(kThreads), 0, 0,
                     static_cast<const char*>(src), n_vec, sink);
  BOOST_HIP(hipGetLastError());
  BOOST_HIP(hipEventRecord(a, 0));
  for (int it = 0; it < iters; ++it)
    hipLaunchKernelGGL(stream_read, dim3(grid), dim3(kThreads), 0, 0,
                       static_cast<const char*>(src), n_vec, sink);
  BOOST_HIP(hipGetLastError());
  BOOST_HIP(hipEventRecord(b, 0));
  BOOST_HIP(hipEventSynchronize(b));
  float ms = 0;
  BOOST_HIP(hipEventElapsedTime(&ms, a, b));
  (void)hipEventDestroy(a);
  (void)hipEventDestroy(b);
  *gbps = static_cast<double>(bytes) * iters / (ms * 1e-3) / 1e9;
  return BOOST_OK;
}

// Clock rate of s_memrealtime (the constant 100 MHz reference clock).
constexpr double kRealtimeHz = 100e6;

}  // namespace

using namespace bst;

extern "C" {

int boost_stream_read_gbps(boost_ctx* ctx, const void* src, uint64_t bytes, int grid,
                           int iters, double* gbps) {
  if (!ctx || !src || !gbps) return fail(BOOST_EINVAL, "null argument");
  if (ctx->device < 0) return fail(BOOST_ENODEV, "plan-only context");
  if (bytes == 0 || bytes % 4096 || grid < 1 || iters < 1)
    return fail(BOOST_EINVAL, "bytes=%llu grid=%d iters=%d",
                (unsigned long long)bytes, grid, iters);
  BOOST_HIP(hipSetDevice(ctx->device));
  uint32_t* sink = nullptr;
  BOOST_HIP(hipMalloc(&sink, static_cast<size_t>(grid) * sizeof(uint32_t)));
  int rc = measure(src, bytes, grid, iters, sink, gbps);
  (void)hipFree(sink);
  return rc;
}

int boost_cap_sweep(boost_ctx* ctx, uint64_t hbm_bytes, uint64_t host_bytes, int n_points,
                    const uint64_t* hbm_use, const int* hbm_wgs, const uint64_t* host_use,
                    const int* host_wgs, const int* host_stride, int iters,
                    double* results) {
  if (!ctx || !hbm_use || !hbm_wgs || !host_use || !host_wgs || !results)
    return fail(BOOST_EINVAL, "null argument");
  if (ctx->device < 0) return fail(BOOST_ENODEV, "plan-only context");
  if (n_points < 1 || iters < 1) return fail(BOOST_EINVAL, "n_points=%d iters=%d", n_points, iters);
  hbm_bytes &= ~4095ull;
  host_bytes &= ~4095ull;
  int max_grid = 1;
  auto stride = [&](int i) { return host_stride ? host_stride[i] : 1; };
  for (int i = 0; i < n_points; ++i) {
    if (stride(i) < 1 || stride(i) > 64 ||
        (host_wgs[i] > 0 && static_cast<int64_t>(host_wgs[i] - 1) * stride(i) >=
                                static_cast<int64_t>(host_wgs[i]) + hbm_wgs[i]))
      return fail(BOOST_EINVAL, "point %d: host stride %d does not fit the grid", i,
                  stride(i));
    if (hbm_use[i] > hbm_bytes || host_use[i] > host_bytes || (hbm_use[i] | host_use[i]) % 16 ||
        hbm_wgs[i] < 0 || host_wgs[i] < 0 || hbm_wgs[i] + host_wgs[i] < 1 ||
        (hbm_use[i] && !hbm_wgs[i]) || (host_use[i] && !host_wgs[i]) ||
        hbm_wgs[i] > (1 << 20) || host_wgs[i] > (1 << 20))
      return fail(BOOST_EINVAL, "point %d: bytes %llu / %llu on %d / %d workgroups", i,
                  (unsigned long long)hbm_use[i], (unsigned long long)host_use[i], hbm_wgs[i],
                  host_wgs[i]);
    if (hbm_wgs[i] && (hbm_use[i] / 16 + hbm_wgs[i] - 1) / hbm_wgs[i] * 16 >= (1ull << 31))
      return fail(BOOST_EINVAL, "point %d: HBM slice exceeds 2 GiB", i);
    if (host_wgs[i] && (host_use[i] / 16 + host_wgs[i] - 1) / host_wgs[i] * 16 >= (1ull << 31))
      return fail(BOOST_EINVAL, "point %d: host slice exceeds 2 GiB", i);
    max_grid = std::max(max_grid, hbm_wgs[i] + host_wgs[i]);
  }
  BOOST_HIP(hipSetDevice(ctx->device));
  Slab dev, host;
  int rc = slab_alloc(ctx, std::max<uint64_t>(1, (hbm_bytes + kPage - 1) / kPage), false, dev);
  if (!rc) rc = slab_alloc(ctx, std::max<uint64_t>(1, (host_bytes + kPage - 1) / kPage), true, host);
  uint32_t* sink = nullptr;
  uint64_t* clocks = nullptr;
  hipEvent_t ea = nullptr, eb = nullptr;
  if (!rc && (hipMalloc(&sink, static_cast<size_t>(max_grid) * 4) != hipSuccess ||
              hipMalloc(&clocks, static_cast<size_t>(max_grid) * 16) != hipSuccess))
    rc = fail(BOOST_ENOMEM, "probe scratch allocation failed");
  if (!rc && hbm_bytes && hipMemset(dev.base, 0x5a, hbm_bytes) != hipSuccess)
    rc = fail(BOOST_EHIP, "memset failed");
  if (!rc && host_bytes) std::memset(host.host_base, 0x5a, host_bytes);
  if (!rc && (hipEventCreate(&ea) != hipSuccess || hipEventCreate(&eb) != hipSuccess))
    rc = fail(BOOST_EHIP, "event creation failed");
  std::vector<uint64_t> clk;
  for (int i = 0; i < n_points && !rc; ++i) {
    const int grid = hbm_wgs[i] + host_wgs[i];
    auto launch = [&]() {
      hipLaunchKernelGGL(cap_stream, dim3(grid), dim3(kThreads), 0, 0,
                         static_cast<const char*>(dev.base), hbm_use[i] / 16,
                         static_cast<const char*>(host.base), host_use[i] / 16, host_wgs[i],
                         stride(i), clocks, sink);
    };
    launch();  // warm-up
    hipError_t e = hipEventRecord(ea, 0);
    for (int it = 0; it < iters && e == hipSuccess; ++it) launch();
    if (e == hipSuccess) e = hipGetLastError();
    if (e == hipSuccess) e = hipEventRecord(eb, 0);
    if (e == hipSuccess) e = hipEventSynchronize(eb);
    float ms = 0;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, ea, eb);
    clk.assign(2 * static_cast<size_t>(grid), 0);
    if (e == hipSuccess)
      e = hipMemcpy(clk.data(), clocks, clk.size() * sizeof(uint64_t), hipMemcpyDeviceToHost);
    if (e != hipSuccess) {
      rc = fail(BOOST_EHIP, "probe point %d: %s", i, hipGetErrorString(e));
      break;
    }
    // clocks of the last pass: each tier's span from the launch's first start
    uint64_t t0 = UINT64_MAX, end_host = 0, end_hbm = 0;
    for (int b = 0; b < grid; ++b) t0 = std::min(t0, clk[2 * b]);
    for (int b = 0; b < grid; ++b) {
      const bool is_host = b % stride(i) == 0 && b / stride(i) < host_wgs[i];
      uint64_t& end = is_host ? end_host : end_hbm;
      end = std::max(end, clk[2 * b + 1]);
    }
    const double total = static_cast<double>(hbm_use[i] + host_use[i]);
    double* r = results + 5 * static_cast<size_t>(i);
    r[0] = total * iters / (ms * 1e-3) / 1e9;  // GB/s of both tiers, launches back to back
    r[1] = static_cast<double>(ms) * 1e3 / iters;  // us per launch
    r[2] = hbm_use[i] && end_hbm > t0 ? hbm_use[i] / ((end_hbm - t0) / kRealtimeHz) / 1e9 : 0.0;
    r[3] = host_use[i] && end_host > t0 ? host_use[i] / ((end_host - t0) / kRealtimeHz) / 1e9
                                        : 0.0;
    r[4] = (std::max(end_hbm, end_host) - t0) / kRealtimeHz * 1e6;  // us, first start to last end
  }
  if (ea) (void)hipEventDestroy(ea);
  if (eb) (void)hipEventDestroy(eb);
  (void)hipFree(sink);
  (void)hipFree(clocks);
  slab_free(dev);
  slab_free(host);
  return rc;
}

int boost_calibrate(boost_ctx* ctx, uint64_t hbm_bytes, uint64_t host_bytes, int iters,
                    double* hbm_gbps, double* host_gbps, double* alpha) {
  if (!ctx) return fail(BOOST_EINVAL, "null ctx");
  if (ctx->device < 0) return fail(BOOST_ENODEV, "plan-only context");
  const uint64_t min_bytes = 64ull << 20;
  if (hbm_bytes < min_bytes || host_bytes < min_bytes || iters < 1)
    return fail(BOOST_EINVAL, "calibration needs >= 64 MiB per tier and iters >= 1");
  hbm_bytes &= ~4095ull;
  host_bytes &= ~4095ull;
  BOOST_HIP(hipSetDevice(ctx->device));
  Slab dev, host;
  int rc = slab_alloc(ctx, (hbm_bytes + kPage - 1) / kPage, false, dev);
  if (!rc) rc = slab_alloc(ctx, (host_bytes + kPage - 1) / kPage, true, host);
  double best_d = 0, best_h = 0;
  uint32_t* sink = nullptr;
  if (!rc && hipMalloc(&sink, 1 << 20) != hipSuccess)
    rc = fail(BOOST_ENOMEM, "sink allocation failed");
  if (!rc && hipMemset(dev.base, 0x5a, hbm_bytes) != hipSuccess)
    rc = fail(BOOST_EHIP, "memset failed");
  if (!rc) std::memset(host.host_base, 0x5a, host_bytes);
  // HBM: grids of 4 to 32 workgroups per CU
  for (int mult : {4, 8, 16, 32}) {
    if (rc) break;
    double g = 0;
    rc = measure(dev.base, hbm_bytes, ctx->n_cu * mult, iters, sink, &g);
    best_d = std::max(best_d, g);
  }
  // host link: from a handful of workgroups up to one per CU and beyond
  for (int grid : {16, 64, 256, 1024}) {
    if (rc) break;
    double g = 0;
    rc = measure(host.base, host_bytes, grid, iters, sink, &g);
    best_h = std::max(best_h, g);
  }
  (void)hipFree(sink);
  slab_free(dev);
  slab_free(host);
  if (rc) return rc;
  if (hbm_gbps) *hbm_gbps = best_d;
  if (host_gbps) *host_gbps = best_h;
  if (alpha) *alpha = best_d > 0 ? best_h / best_d : 0.0;
  return BOOST_OK;
}

}  // extern "C"
