// a6: the element-wise glue of a full decode step of a pre-norm Llama-style
// model (the paper runs whole decode steps, §5.1; the operators themselves
// are not its subject): embedding gather, RMSNorm, RoPE with the q/k/v split
// of the fused qkv output, KV append, SiLU(gate) * up, residual add and
// argmax.  The residual stream is fp32; operands of the matrix products and
// of attention are bf16 (round to nearest even).
#include <cmath>

#include "runtime.h"

namespace {

__device__ __forceinline__ float lo_bf16(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t v) {
  return __uint_as_float(v & 0xffff0000u);
}
__device__ __forceinline__ uint16_t to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return 0x7fc0;
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// A split-K GEMV output handed over as its S partial slices: [S][B][N]
// fp32, then, for the rows that cross a 2 MiB page of the [N, K] matrix, the
// two parts of each such row ([page of the row's end][part][S][B]).  S == 1
// is the unsplit output itself.
struct Slices {
  const float* p;
  int S, B;
  int64_t N, K;
};

constexpr int64_t kPageElems = static_cast<int64_t>(bst::kPage / 2);

// Whether row r of the [N, K] bf16 matrix crosses a page boundary (K = 0:
// never, the caller having found that K divides a page).
__device__ __forceinline__ bool cut_row(int64_t r, int64_t K) {
  return (r * K) / kPageElems != (r * K + K - 1) / kPageElems;
}

// Element (b, r) of the output: the slices summed in slice order from zero,
// and a cut row's earlier part then its later part, the additions the
// GEMV's own reduction kernel makes, so a consumer that takes the slices
// sees the same bits as one that takes the reduced output.  All loads go out
// before the sums (a loop over a run-time S would wait for each in turn).
__device__ __forceinline__ float slice_value(const Slices& sl, int b, int64_t r) {
  const int64_t i = static_cast<int64_t>(b) * sl.N + r;
  if (sl.S == 1) return sl.p[i];
  const int64_t stride = static_cast<int64_t>(sl.B) * sl.N;
  if (!cut_row(r, sl.K)) {
    float part[BOOST_MAX_GEMV_SLICES];
#pragma unroll
    for (int s = 0; s < BOOST_MAX_GEMV_SLICES; ++s)
      part[s] = s < sl.S ? sl.p[s * stride + i] : 0.f;
    float v = 0.f;
#pragma unroll
    for (int s = 0; s < BOOST_MAX_GEMV_SLICES; ++s)
      if (s < sl.S) v += part[s];
    return v;
  }
  const int64_t p1 = (r * sl.K + sl.K - 1) / kPageElems;
  const float* cut = sl.p + sl.S * stride;
  float part0[BOOST_MAX_GEMV_SLICES], part1[BOOST_MAX_GEMV_SLICES];
#pragma unroll
  for (int s = 0; s < BOOST_MAX_GEMV_SLICES; ++s) {
    part0[s] = s < sl.S ? cut[((p1 * 2 + 0) * sl.S + s) * sl.B + b] : 0.f;
    part1[s] = s < sl.S ? cut[((p1 * 2 + 1) * sl.S + s) * sl.B + b] : 0.f;
  }
  float v = 0.f, v1 = 0.f;
#pragma unroll
  for (int s = 0; s < BOOST_MAX_GEMV_SLICES; ++s)
    if (s < sl.S) {
      v += part0[s];
      v1 += part1[s];
    }
  return v + v1;
}

// One lane per 8 elements of one row; the row of token t is read through the
// embedding tensor's page table.
__global__ __launch_bounds__(256) void embed_gather_kernel(const char* const* __restrict__ pt,
                                                           const int32_t* __restrict__ tok,
                                                           int B, int V, int d,
                                                           float* __restrict__ out) {
  const int chunks = d / 8;
  const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= static_cast<int64_t>(B) * chunks) return;
  const int b = static_cast<int>(t / chunks), c = static_cast<int>(t % chunks);
  const int32_t id = tok[b];
  float4* o = reinterpret_cast<float4*>(out + static_cast<int64_t>(b) * d + c * 8);
  if (id < 0 || id >= V) {
    o[0] = make_float4(0.f, 0.f, 0.f, 0.f);
    o[1] = o[0];
    return;
  }
  const uint64_t byte = (static_cast<uint64_t>(id) * d + c * 8) * 2;
  const uint4 u = *reinterpret_cast<const uint4*>(pt[byte >> 21] + (byte & (bst::kPage - 1)));
  o[0] = make_float4(lo_bf16(u.x), hi_bf16(u.x), lo_bf16(u.y), hi_bf16(u.y));
  o[1] = make_float4(lo_bf16(u.z), hi_bf16(u.z), lo_bf16(u.w), hi_bf16(u.w));
}

// One workgroup per row: sum of squares in a fixed order, then
// y = bf16(x * (1 / sqrt(mean + eps)) * w).  With ADD the row first takes
// the residual r (x += r in fp32, stored back), the same additions the
// separate residual add makes, so the fused call gives the same bits; the
// residual may come as split-K slices (see slice_value; rs.p is r).
template <bool ADD>
__global__ __launch_bounds__(256) void rmsnorm_kernel(float* __restrict__ x, Slices rs,
                                                      const uint16_t* __restrict__ w, int d,
                                                      float eps, uint16_t* __restrict__ y) {
  __shared__ float part[4];
  float* row = x + static_cast<int64_t>(blockIdx.x) * d;
  float s = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) {
    float v = row[i];
    if constexpr (ADD) {
      v += slice_value(rs, blockIdx.x, i);
      row[i] = v;  // read back below by this same lane
    }
    s = fmaf(v, v, s);
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) s += __shfl_xor(s, m, 64);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = s;
  __syncthreads();
  const float tot = ((part[0] + part[1]) + part[2]) + part[3];
  const float scale = 1.0f / sqrtf(tot / static_cast<float>(d) + eps);
  uint16_t* out = y + static_cast<int64_t>(blockIdx.x) * d;
  for (int i = threadIdx.x; i < d; i += 256)
    out[i] = to_bf16(row[i] * scale * __uint_as_float(static_cast<uint32_t>(w[i]) << 16));
}

// The same for rows of d <= 8192 floats with d % 4 == 0 and 16-byte aligned
// rows: each of the workgroup's 1024 lanes loads its (at most NV = 2) float4s
// of the row at once and keeps them in registers for the second pass (the
// plain loop above is a chain of dependent round trips: 20 us for a batch of
// 8 rows of 8192); sixteen wavefronts per row keep its slice loads in flight.
constexpr int kNormThreads = 1024;
constexpr int kNormVec = 2;
// Pages of the producing [d, K] matrix (at most d, since K <= 2^20 elements
// and d <= 8192 here): a workgroup of the vector norm sums each cut row once
// into LDS, indexed by the page of the row's last column.
constexpr int kMaxCutPages = 4 * kNormThreads * kNormVec;
template <bool ADD, int NV>
__global__ __launch_bounds__(kNormThreads) void rmsnorm_vec_kernel(
    float* __restrict__ x, Slices rs, const uint16_t* __restrict__ w, int d, float eps,
    uint16_t* __restrict__ y) {
  constexpr int NT = kNormThreads;
  __shared__ float part[NT / 64];
  const int n4 = d / 4;
  float4* row = reinterpret_cast<float4*>(x + static_cast<int64_t>(blockIdx.x) * d);
  float4 v[NV];
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    const int i = threadIdx.x + u * NT;
    v[u] = i < n4 ? row[i] : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  if constexpr (ADD) {
    // the residual, or the slice-order sum of its S slices (see
    // slice_value), taken in groups of four slices whose loads of the whole
    // row go out before the group's additions (uniform guards, no waits
    // between).  A row of the producing matrix that crosses a page takes
    // its value from its two parts instead: one lane per page boundary sums
    // them into LDS while the first group's loads are in flight.
    __shared__ float cutv[kMaxCutPages];
    const int S = rs.S;
    const int64_t stride = static_cast<int64_t>(rs.B) * d;
    float4 a[NV];
    const float* r0 = rs.p + static_cast<int64_t>(blockIdx.x) * d;
    if (S == 1) {
#pragma unroll
      for (int u = 0; u < NV; ++u) {
        const int i = threadIdx.x + u * NT;
        a[u] = i < n4 ? reinterpret_cast<const float4*>(r0)[i] : make_float4(0.f, 0.f, 0.f, 0.f);
      }
    } else {
      const int nu = (n4 + NT - 1) / NT;
      const int64_t pages = (static_cast<int64_t>(d) * rs.K + kPageElems - 1) / kPageElems;
#pragma unroll
      for (int u = 0; u < NV; ++u) a[u] = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int s0 = 0; s0 < S; s0 += 4) {
        float4 t[NV][4];
#pragma unroll
        for (int u = 0; u < NV; ++u)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int i = threadIdx.x + u * NT;
            t[u][j] = u < nu && s0 + j < S && i < n4
                          ? reinterpret_cast<const float4*>(r0 + (s0 + j) * stride)[i]
                          : make_float4(0.f, 0.f, 0.f, 0.f);
          }
        if (s0 == 0)
          for (int q = threadIdx.x + 1; q < pages; q += NT) {
            const int64_t e = static_cast<int64_t>(q) * kPageElems;
            if (e % rs.K != 0) cutv[q] = slice_value(rs, blockIdx.x, e / rs.K);
          }
#pragma unroll
        for (int u = 0; u < NV; ++u)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (s0 + j < S) {
              a[u].x += t[u][j].x;
              a[u].y += t[u][j].y;
              a[u].z += t[u][j].z;
              a[u].w += t[u][j].w;
            }
      }
      __syncthreads();  // cutv
      auto cut_value = [&](int64_t e) { return cutv[(e * rs.K + rs.K - 1) / kPageElems]; };
#pragma unroll
      for (int u = 0; u < NV; ++u) {
        const int i = threadIdx.x + u * NT;
        if (u < nu && i < n4) {
          const int64_t e = 4 * static_cast<int64_t>(i);
          if (cut_row(e, rs.K)) a[u].x = cut_value(e);
          if (cut_row(e + 1, rs.K)) a[u].y = cut_value(e + 1);
          if (cut_row(e + 2, rs.K)) a[u].z = cut_value(e + 2);
          if (cut_row(e + 3, rs.K)) a[u].w = cut_value(e + 3);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      const int i = threadIdx.x + u * NT;
      if (i < n4) {
        v[u].x += a[u].x;
        v[u].y += a[u].y;
        v[u].z += a[u].z;
        v[u].w += a[u].w;
        row[i] = v[u];
      }
    }
  }
  float s = 0.f;
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    s = fmaf(v[u].x, v[u].x, s);
    s = fmaf(v[u].y, v[u].y, s);
    s = fmaf(v[u].z, v[u].z, s);
    s = fmaf(v[u].w, v[u].w, s);
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) s += __shfl_xor(s, m, 64);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = s;
  __syncthreads();
  float tot = part[0];  // the wavefronts' sums in wavefront order
#pragma unroll
  for (int i = 1; i < NT / 64; ++i) tot += part[i];
  const float scale = 1.0f / sqrtf(tot / static_cast<float>(d) + eps);
  const uint2* w4 = reinterpret_cast<const uint2*>(w);
  uint2* out = reinterpret_cast<uint2*>(y + static_cast<int64_t>(blockIdx.x) * d);
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    const int i = threadIdx.x + u * NT;
    if (i >= n4) break;
    const uint2 ww = w4[i];
    const float w0 = __uint_as_float(ww.x << 16), w1 = __uint_as_float(ww.x & 0xffff0000u);
    const float w2 = __uint_as_float(ww.y << 16), w3 = __uint_as_float(ww.y & 0xffff0000u);
    uint2 o;
    o.x = to_bf16(v[u].x * scale * w0) | (static_cast<uint32_t>(to_bf16(v[u].y * scale * w1)) << 16);
    o.y = to_bf16(v[u].z * scale * w2) | (static_cast<uint32_t>(to_bf16(v[u].w * scale * w3)) << 16);
    out[i] = o;
  }
}

// Where the key and value heads of the new token go when they are written
// straight into the pool (the fused RoPE + KV append): the layer's K and V
// page tables, the block tables and the pool geometry.
struct PoolSlot {
  const char* const* pt_k;
  const char* const* pt_v;
  const int32_t* tables;
  int max_blocks, T, nb;
};

// One wavefront per (request, head of the fused qkv output), four to a
// workgroup, one lane per rotation pair.  Query and key heads are rotated (half-split pairs, angle in
// double precision); value heads are converted.  With POOL the key and value
// heads go to the token's slot of the pool (the same bits the KV append
// copies there), skipped like the append skips a position or block outside
// the table or the pool.  qkv may come as split-K slices (see slice_value).
constexpr int kRopeWaves = 4;
template <bool POOL>
__global__ __launch_bounds__(64 * kRopeWaves) void rope_qkv_kernel(
    Slices qkv, const int32_t* __restrict__ pos, int Hq, int H, int D, double log2_theta,
    uint16_t* __restrict__ q, uint16_t* __restrict__ k, uint16_t* __restrict__ v, PoolSlot ps) {
  const int heads = Hq + 2 * H;
  const int item = blockIdx.x * kRopeWaves + static_cast<int>(threadIdx.x >> 6);
  if (item >= qkv.B * heads) return;  // uniform over the wavefront; no barrier follows
  const int b = item / heads, h = item % heads;
  const int lane = threadIdx.x & 63;
  const int half = D / 2;
  const int64_t col0 = static_cast<int64_t>(h) * D;  // this head's first column
  uint16_t* dst;
  if (h < Hq) {
    dst = q + (static_cast<int64_t>(b) * Hq + h) * D;
  } else if constexpr (POOL) {
    const int p = pos[b];  // uniform over the wavefront
    if (p < 0 || p >= ps.max_blocks * ps.T) return;
    const int32_t blk = ps.tables[static_cast<int64_t>(b) * ps.max_blocks + p / ps.T];
    if (blk < 0 || blk >= ps.nb) return;
    const int g = h < Hq + H ? h - Hq : h - Hq - H;
    // a head row (D * 2 bytes, dividing the page) never crosses a page
    const uint64_t byte = ((static_cast<uint64_t>(g) * ps.nb + blk) * ps.T + p % ps.T) * D * 2;
    const char* const* pt = h < Hq + H ? ps.pt_k : ps.pt_v;
    dst = reinterpret_cast<uint16_t*>(const_cast<char*>(pt[byte >> 21]) +
                                      (byte & (bst::kPage - 1)));
  } else if (h < Hq + H) {
    dst = k + (static_cast<int64_t>(b) * H + (h - Hq)) * D;
  } else {
    dst = v + (static_cast<int64_t>(b) * H + (h - Hq - H)) * D;
  }
  for (int i = lane; i < half; i += 64) {
    const float a = slice_value(qkv, b, col0 + i), c = slice_value(qkv, b, col0 + i + half);
    if (h >= Hq + H) {
      dst[i] = to_bf16(a);
      dst[i + half] = to_bf16(c);
      continue;
    }
    const double inv = exp2(-(2.0 * i / D) * log2_theta);
    const double ang = static_cast<double>(pos[b]) * inv;
    double sn, cs;
    sincos(ang, &sn, &cs);
    dst[i] = to_bf16(static_cast<float>(a * cs - c * sn));
    dst[i + half] = to_bf16(static_cast<float>(a * sn + c * cs));
  }
}

// The new token of request b (position pos[b]) goes to slot
// table[b][pos / T] * T + pos % T of the layer's K and V tensors.
__global__ __launch_bounds__(256) void kv_append_kernel(
    const char* const* __restrict__ pt_k, const char* const* __restrict__ pt_v,
    const int32_t* __restrict__ tables, int max_blocks, const int32_t* __restrict__ pos,
    const uint4* __restrict__ k, const uint4* __restrict__ v, int B, int H, int D, int T,
    int nb) {
  const int chunks = D / 8;
  const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= static_cast<int64_t>(B) * H * chunks) return;
  const int c = static_cast<int>(t % chunks);
  const int h = static_cast<int>((t / chunks) % H);
  const int b = static_cast<int>(t / (static_cast<int64_t>(chunks) * H));
  const int p = pos[b];
  if (p < 0 || p >= max_blocks * T) return;
  const int32_t blk = tables[static_cast<int64_t>(b) * max_blocks + p / T];
  if (blk < 0 || blk >= nb) return;
  const uint64_t byte = ((static_cast<uint64_t>(h) * nb + blk) * T + p % T) * D * 2 +
                        static_cast<uint64_t>(c) * 16;
  const uint64_t page = byte >> 21, in = byte & (bst::kPage - 1);
  *reinterpret_cast<uint4*>(const_cast<char*>(pt_k[page]) + in) = k[t];
  *reinterpret_cast<uint4*>(const_cast<char*>(pt_v[page]) + in) = v[t];
}

__global__ __launch_bounds__(256) void silu_mul_kernel(const float* __restrict__ gu, int B,
                                                       int F, uint16_t* __restrict__ out) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= static_cast<int64_t>(B) * F) return;
  const int64_t b = t / F, j = t % F;
  const float g = gu[b * 2 * F + j], u = gu[b * 2 * F + F + j];
  out[t] = to_bf16(g / (1.0f + expf(-g)) * u);
}

__global__ __launch_bounds__(256) void residual_add_kernel(float* __restrict__ x,
                                                           const float* __restrict__ y,
                                                           int64_t n) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t < n) x[t] += y[t];
}

__device__ __forceinline__ void better(float& bv, int& bi, float v, int i) {
  // larger value wins; equal values keep the lower index
  if (v > bv || (v == bv && i < bi)) {
    bv = v;
    bi = i;
  }
}

// One 1024-lane workgroup per row; ties go to the lowest index (the rule is
// order-free, so the traversal order does not matter).  Rows of V % 4 == 0
// at 16-byte alignment are read as float4, four loads in flight per lane.
constexpr int kArgThreads = 1024;
__global__ __launch_bounds__(kArgThreads) void argmax_kernel(const float* __restrict__ logits,
                                                             int V, int vec,
                                                             int32_t* __restrict__ ids) {
  __shared__ float sv[kArgThreads / 64];
  __shared__ int si[kArgThreads / 64];
  const float* row = logits + static_cast<int64_t>(blockIdx.x) * V;
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  if (vec) {
    const float4* r4 = reinterpret_cast<const float4*>(row);
    const int n4 = V / 4;
    for (int i0 = threadIdx.x; i0 < n4; i0 += 4 * kArgThreads) {
      float4 q[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = i0 + u * kArgThreads;
        q[u] = i < n4 ? r4[i] : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = 4 * (i0 + u * kArgThreads);
        better(bv, bi, q[u].x, i);
        better(bv, bi, q[u].y, i + 1);
        better(bv, bi, q[u].z, i + 2);
        better(bv, bi, q[u].w, i + 3);
      }
    }
  } else {
    for (int i = threadIdx.x; i < V; i += kArgThreads) better(bv, bi, row[i], i);
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const float ov = __shfl_xor(bv, m, 64);
    const int oi = __shfl_xor(bi, m, 64);
    better(bv, bi, ov, oi);
  }
  if ((threadIdx.x & 63) == 0) {
    sv[threadIdx.x >> 6] = bv;
    si[threadIdx.x >> 6] = bi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < kArgThreads / 64; ++w) better(bv, bi, sv[w], si[w]);
    ids[blockIdx.x] = bi == 0x7fffffff ? 0 : bi;
  }
}

inline unsigned blocks_for(int64_t n, int per) { return static_cast<unsigned>((n + per - 1) / per); }

}  // namespace

using namespace bst;

extern "C" {

int boost_embed_gather(boost_ctx* ctx, const boost_tensor* E, int V, int d,
                       const int32_t* tokens, int B, float* out, void* stream) {
  if (!ctx || !E || !tokens || !out) return fail(BOOST_EINVAL, "null argument");
  if (ctx->device < 0) return fail(BOOST_ENODEV, "plan-only context");
  if (V < 1 || d < 8 || d % 8 || B < 1) return fail(BOOST_EINVAL, "V=%d d=%d B=%d", V, d, B);
  if (static_cast<uint64_t>(V) * d * 2 != E->bytes)
    return fail(BOOST_EINVAL, "V*d*2 does not match the tensor");
  const int64_t n = static_cast<int64_t>(B) * (d / 8);
  hipLaunchKernelGGL(embed_gather_kernel, dim3(blocks_for(n, 256)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), E->d_page_table, tokens, B, V, d, out);
  BOOST_HIP(hipGetLastError());
  return BOOST_OK;
}

}  // extern "C"

namespace {
// x (+= r when r is given), then the norm; the row layout decides the
// kernel, never r, so the fused and the separate calls take the same one
int launch_rmsnorm(boost_ctx* ctx, float* x, const float* r, int S, int K, const void* w,
                   int B, int d, float eps, void* out, void* stream) {
  if (!ctx || !x || !w || !out) return fail(BOOST_EINVAL, "null argument");
  if (ctx->device < 0) return fail(BOOST_ENODEV, "plan-only context");
  if (B < 1 || d < 1 || !(eps >= 0.f)) return fail(BOOST_EINVAL, "B=%d d=%d eps=%g", B, d, eps);
  const bool vec = d % 4 == 0 && d <= 4 * kNormThreads * kNormVec &&
                   (reinterpret_cast<uintptr_t>(x) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(r) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(w) & 7) == 0 &&
                   (reinterpret_cast<uintptr_t>(out) & 7) == 0;
  auto s = static_cast<hipStream_t>(stream);
  auto wp = static_cast<const uint16_t*>(w);
  auto op = static_cast<uint16_t*>(out);
  // K = 0: no row of the producing matrix crosses a page
  const Slices rs{r, S, B, d, kPageElems % K ? K : 0};
  const bool nv1 = d <= 4 * kNormThreads;  // one float4 per lane covers the row
  const dim3 g(B), t(kNormThreads);
  if (vec && r && nv1)
    hipLaunchKernelGGL((rmsnorm_vec_kernel<true, 1>), g, t, 0, s, x, rs, wp, d, eps, op);
  else if (vec && r)
    hipLaunchKernelGGL((rmsnorm_vec_kernel<true, kNormVec>), g, t, 0, s, x, rs, wp, d, eps, op);
  else if (vec && nv1)
    hipLaunchKernelGGL((rmsnorm_vec_kernel<false, 1>), g, t, 0, s, x, rs, wp, d, eps, op);
  else if (vec)
    hipLaunchKernelGGL((rmsnorm_vec_kernel<false, kNormVec>), g, t, 0, s, x, rs, wp, d, eps, op);
  else if (r)
    hipLaunchKernelGGL(rmsnorm_kernel<true>, dim3(B), dim3(256), 0, s, x, rs, wp, d, eps, op);
  else
    hipLaunchKernelGGL(rmsnorm_kernel<false>, dim3(B), dim3(256), 0, s, x, rs, wp, d, eps, op);
  BOOST_HIP(hipGetLastError());
  return BOOST_OK;
}
}  // namespace

extern "C" {

int boost_rmsnorm(boost_ctx* ctx, const float* x, const void* w, int B, int d, float eps,
                  void* out, void* stream) {
  // the kernel without the residual never writes x
  return launch_rmsnorm(ctx, const_cast<float*>(x), nullptr, 1, 1, w, B, d, eps, out, stream);
}

int boost_add_rmsnorm(boost_ctx* ctx, float* x, const float* r, const void* w, int B, int d,
                      float eps, void* out, void* stream) {
  if (!r) return fail(BOOST_EINVAL, "null argument");
  if (reinterpret_cast<uintptr_t>(r) & 15) return fail(BOOST_EINVAL, "r must be 16-byte aligned");
  return launch_rmsnorm(ctx, x, r, 1, 1, w, B, d, eps, out, stream);
}

int boost_add_rmsnorm_slices(boost_ctx* ctx, float* x, const float* r, int S, int K,
                             const void* w, int B, int d, float eps, void* out, void* stream) {
  if (!r) return fail(BOOST_EINVAL, "null argument");
  if (reinterpret_cast<uintptr_t>(r) & 15) return fail(BOOST_EINVAL, "r must be 16-byte aligned");
  if (S < 1 || S > BOOST_MAX_GEMV_SLICES || K < 1 || K > kPageElems)
    return fail(BOOST_EINVAL, "S=%d (1..%d) K=%d (1..2^20)", S, BOOST_MAX_GEMV_SLICES, K);
  return launch_rmsnorm(ctx, x, r, S, K, w, B, d, eps, out, stream);
}

int boost_rope_qkv(boost_ctx* ctx, const float* qkv, const int32_t* positions, int B, int Hq,
                   int H, int D, double theta, void* q, void* k, void* v, void* stream) {
  if (!ctx || !qkv || !positions || !q || !k || !v) return fail(BOOST_EINVAL, "null argument");
  if (ctx->device < 0) return fail(BOOST_ENODEV, "plan-only context");
  if (B < 1 || Hq < 1 || H < 1 || D < 2 || D % 2 || !(theta > 1.0))
    return fail(BOOST_EINVAL, "B=%d Hq=%d H=%d D=%d theta=%g", B, Hq, H, D, theta);
  const Slices sl{qkv, 1, B, static_cast<int64_t>(Hq + 2 * H) * D, 1};
  hipLaunchKernelGGL(rope_qkv_kernel<false>,
                     dim3((B * (Hq + 2 * H) + kRopeWaves - 1) / kRopeWaves),
                     dim3(64 * kRopeWaves), 0,
                     static_cast<hipStream_t>(stream), sl, positions, Hq, H, D, std::log2(theta),
                     static_cast<uint16_t*>(q), static_cast<uint16_t*>(k),
                     static_cast<uint16_t*>(v), PoolSlot{});
  BOOST_HIP(hipGetLastError());
  return BOOST_OK;
}

int boost_rope_kv_append(boost_ctx* ctx, const boost_kv_pool* p, int layer, const float* qkv,
                         const int32_t* positions, int B, int Hq, double theta,
                         const int32_t* block_tables, int max_blocks, void* q, void* stream) {
  return boost_rope_kv_append_slices(ctx, p, layer, qkv, 1, 1, positions, B, Hq, theta,
                                     block_tables, max_blocks, q, stream);
}

int boost_rope_kv_append_slices(boost_ctx* ctx, const boost_kv_pool* p, int layer,
                                const float* qkv, int S, int K, const int32_t* positions,
                                int B, int Hq, double theta, const int32_t* block_tables,
                                int max_blocks, void* q, void* stream) {
  if (!ctx || !p || !qkv || !positions || !block_tables || !q)
    return fail(BOOST_EINVAL, "null argument");
  if (ctx->device < 0 || !p->d_page_table) return fail(BOOST_ENODEV, "plan-only pool");
  if (layer < 0 || static_cast<uint32_t>(layer) >= p->cfg.layers)
    return fail(BOOST_EINVAL, "layer %d", layer);
  const int H = static_cast<int>(p->cfg.kv_heads), D = static_cast<int>(p->cfg.head_dim);
  if (B < 1 || max_blocks < 1 || Hq < 1 || !(theta > 1.0) || kPage % (2ull * D) != 0)
    return fail(BOOST_EINVAL, "B=%d max_blocks=%d Hq=%d theta=%g D=%d", B, max_blocks, Hq,
                theta, D);
  if (S < 1 || S > BOOST_MAX_GEMV_SLICES || K < 1 || K > kPageElems)
    return fail(BOOST_EINVAL, "S=%d (1..%d) K=%d (1..2^20)", S, BOOST_MAX_GEMV_SLICES, K);
  const uint64_t P = p->geom.pages;
  const PoolSlot ps{p->d_page_table + 2ull * layer * P, p->d_page_table + (2ull * layer + 1) * P,
                    block_tables, max_blocks, static_cast<int>(p->cfg.block_tokens),
                    static_cast<int>(p->geom.nb)};
  // K = 0: no row of the producing matrix crosses a page
  const Slices sl{qkv, S, B, static_cast<int64_t>(Hq + 2 * H) * D, kPageElems % K ? K : 0};
  hipLaunchKernelGGL(rope_qkv_kernel<true>,
                     dim3((B * (Hq + 2 * H) + kRopeWaves - 1) / kRopeWaves),
                     dim3(64 * kRopeWaves), 0,
                     static_cast<hipStream_t>(stream), sl, positions, Hq, H, D, std::log2(theta),
                     static_cast<uint16_t*>(q), nullptr, nullptr, ps);
  BOOST_HIP(hipGetLastError());
  return BOOST_OK;
}

int boost_kv_append(boost_ctx* ctx, const boost_kv_pool* p, int layer,
                    const int32_t* block_tables, int max_blocks, const int32_t* positions,
                    const void* k, const void* v, int B, void* stream) {
  if (!ctx || !p || !block_tables || !positions || !k || !v)
    return fail(BOOST_EINVAL, "null argument");
  if (ctx->device < 0 || !p->d_page_table) return fail(BOOST_ENODEV, "plan-only pool");
  if (layer < 0 || static_cast<uint32_t>(layer) >= p->cfg.layers)
    return fail(BOOST_EINVAL, "layer %d", layer);
  if (B < 1 || max_blocks < 1) return fail(BOOST_EINVAL, "B=%d max_blocks=%d", B, max_blocks);
  if ((reinterpret_cast<uintptr_t>(k) | reinterpret_cast<uintptr_t>(v)) & 15)
    return fail(BOOST_EINVAL, "k and v must be 16-byte aligned");
  const uint64_t P = p->geom.pages;
  const int H = static_cast<int>(p->cfg.kv_heads), D = static_cast<int>(p->cfg.head_dim);
  const int64_t n = static_cast<int64_t>(B) * H * (D / 8);
  hipLaunchKernelGGL(kv_append_kernel, dim3(blocks_for(n, 256)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), p->d_page_table + 2ull * layer * P,
                     p->d_page_table + (2ull * layer + 1) * P, block_tables, max_blocks,
                     positions, static_cast<const uint4*>(k), static_cast<const uint4*>(v), B,
                     H, D, static_cast<int>(p->cfg.block_tokens), static_cast<int>(p->geom.nb));
  BOOST_HIP(hipGetLastError());
  return BOOST_OK;
}

int boost_silu_mul(boost_ctx* ctx, const float* gu, int B, int F, void* out, void* stream) {
  if (!ctx || !gu || !out) return fail(BOOST_EINVAL, "null argument");
  if (ctx->device < 0) return fail(BOOST_ENODEV, "plan-only context");
  if (B < 1 || F < 1) return fail(BOOST_EINVAL, "B=%d F=%d", B, F);
  const int64_t n = static_cast<int64_t>(B) * F;
  hipLaunchKernelGGL(silu_mul_kernel, dim3(blocks_for(n, 256)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), gu, B, F, static_cast<uint16_t*>(out));
  BOOST_HIP(hipGetLastError());
  return BOOST_OK;
}

int boost_residual_add(boost_ctx* ctx, float* x, const float* y, int64_t n, void* stream) {
  if (!ctx || !x || !y) return fail(BOOST_EINVAL, "null argument");
  if (ctx->device < 0) return fail(BOOST_ENODEV, "plan-only context");
  if (n < 1) return fail(BOOST_EINVAL, "n=%lld", (long long)n);
  hipLaunchKernelGGL(residual_add_kernel, dim3(blocks_for(n, 256)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), x, y, n);
  BOOST_HIP(hipGetLastError());
  return BOOST_OK;
}

int boost_argmax(boost_ctx* ctx, const float* logits, int B, int V, int32_t* ids,
                 void* stream) {
  if (!ctx || !logits || !ids) return fail(BOOST_EINVAL, "null argument");
  if (ctx->device < 0) return fail(BOOST_ENODEV, "plan-only context");
  if (B < 1 || V < 1) return fail(BOOST_EINVAL, "B=%d V=%d", B, V);
  const int vec = V % 4 == 0 && (reinterpret_cast<uintptr_t>(logits) & 15) == 0;
  hipLaunchKernelGGL(argmax_kernel, dim3(B), dim3(kArgThreads), 0,
                     static_cast<hipStream_t>(stream), logits, V, vec, ids);
  BOOST_HIP(hipGetLastError());
  return BOOST_OK;
}

}  // extern "C"
