// a5: GQA paged-attention decode over a tiered KV pool.
//
// Work item = (KV head g, request b, context partition): the workgroup is the
// paper's "KV head chunk" threadblock (§3.3).  Its G = Hq/H query heads share
// every K/V load.  A block's K (or V) rows of one head are 16 x 128 bf16 =
// 4 KiB contiguous (heads outermost, §4.5), so one 16-byte load per lane of
// the 256-lane workgroup reads a whole head-block: lane = 16 * token + chunk,
// chunk = 8 dimensions.  The block's address comes from the device page table
// of the pool, so the same code reads HBM and host pages; a request of the
// SHH type keeps head H-1 on host for all its blocks, so those work items
// read only host memory for their whole life (§3.2 confinement).  Items of
// the heads that can hold host pages (the highest heads, where the linear
// tail lies) are dispatched first so their slow reads overlap the HBM items.
//
// Each of the 16 token slots of the workgroup keeps its own running max, sum
// and weighted V (online softmax); slots are merged at the end of the
// partition (xor shuffles inside a wavefront, LDS across wavefronts, fixed
// order), partitions by a second kernel that applies log-sum-exp weights in
// partition order.  The arithmetic is independent of the placement.
#include <algorithm>
#include <cmath>

#include "runtime.h"

namespace bst {
int kv_parts_for(const boost_kv_pool* p, int max_blocks);
}

namespace {

constexpr int kThreads = 256;
constexpr int kD = 128;          // head dimension of this kernel
constexpr int kT = 16;           // tokens per block
constexpr int kLanesTok = kD / 8;  // lanes per token row (16)
constexpr int kUnroll = 4;       // blocks in flight per workgroup

struct AttnParams {
  const char* const* pk;  // page table of this layer's K tensor
  const char* const* pv;  // ... and V tensor
  const uint16_t* q;      // [B, Hq, D]
  const int32_t* tables;  // [B, max_blocks]
  const int32_t* lens;    // [B]
  int B, H, Hq, nb, max_blocks;
  int part_blocks, n_parts;  // partition size in blocks, partitions per request
  int max_parts;             // stride of the partial buffers
  float scale;
  float* part_acc;  // [B * Hq * max_parts][D] unnormalised sums of p * v
  float* part_ml;   // [B * Hq * max_parts][2] running max, sum of p
  void* out;
  int out_bf16;
};

__device__ __forceinline__ float lo_bf16(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t v) {
  return __uint_as_float(v & 0xffff0000u);
}

__device__ __forceinline__ void unpack8(const uint4& u, float* f) {
  f[0] = lo_bf16(u.x); f[1] = hi_bf16(u.x);
  f[2] = lo_bf16(u.y); f[3] = hi_bf16(u.y);
  f[4] = lo_bf16(u.z); f[5] = hi_bf16(u.z);
  f[6] = lo_bf16(u.w); f[7] = hi_bf16(u.w);
}

__device__ __forceinline__ uint16_t to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return 0x7fc0;
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

__device__ __forceinline__ uint4 load_block(const char* base, bool ok, uint32_t off) {
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<char*>(base), 0, ok ? kT * kD * 2 : 0, 0x00020000);
  auto v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 2);
  return *reinterpret_cast<uint4*>(&v);
}

// merge running state (m, l, acc) with another one; symmetric in its operands
template <int G>
__device__ __forceinline__ void merge_state(float* m, float* l, float (*acc)[8],
                                            const float* m2, const float* l2,
                                            const float (*acc2)[8]) {
#pragma unroll
  for (int j = 0; j < G; ++j) {
    const float M = fmaxf(m[j], m2[j]);
    if (M == -INFINITY) continue;  // both empty
    const float c1 = m[j] == -INFINITY ? 0.f : __expf(m[j] - M);
    const float c2 = m2[j] == -INFINITY ? 0.f : __expf(m2[j] - M);
    l[j] = l[j] * c1 + l2[j] * c2;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[j][e] = acc[j][e] * c1 + acc2[j][e] * c2;
    m[j] = M;
  }
}

template <int G>
__global__ __launch_bounds__(kThreads) void attn_partition(AttnParams P) {
  __shared__ float s_ml[4][G][2];
  __shared__ float s_acc[4][G][kD];
  const int tid = threadIdx.x;
  const int ts = tid / kLanesTok;  // token slot 0..15
  const int dc = tid % kLanesTok;  // 8-dim chunk
  const int part = blockIdx.x % P.n_parts;
  const int rest = blockIdx.x / P.n_parts;
  const int b = rest % P.B;
  const int g = P.H - 1 - rest / P.B;  // highest heads first
  const int L = P.lens[b];
  const int n_blk = min((L + kT - 1) / kT, P.max_blocks);
  const int blk_beg = part * P.part_blocks;
  if (L <= 0 || blk_beg >= n_blk) return;  // uniform: empty partition
  const int blk_end = min(n_blk, blk_beg + P.part_blocks);

  float qf[G][8];
#pragma unroll
  for (int j = 0; j < G; ++j) {
    const uint4 u = *reinterpret_cast<const uint4*>(
        P.q + (static_cast<int64_t>(b) * P.Hq + g * G + j) * kD + dc * 8);
    unpack8(u, qf[j]);
#pragma unroll
    for (int e = 0; e < 8; ++e) qf[j][e] *= P.scale;
  }
  float m[G], l[G], acc[G][8];
#pragma unroll
  for (int j = 0; j < G; ++j) {
    m[j] = -INFINITY;
    l[j] = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[j][e] = 0.f;
  }

  const int32_t* row = P.tables + static_cast<int64_t>(b) * P.max_blocks;
  const uint32_t lane_off = static_cast<uint32_t>(tid) * 16;
  for (int i = blk_beg; i < blk_end; i += kUnroll) {
    uint4 kv[kUnroll], vv[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int bi = i + u;
      const int32_t blk = bi < blk_end ? row[bi] : -1;
      const bool ok = blk >= 0 && blk < P.nb;
      const uint64_t byte = ok ? (static_cast<uint64_t>(g) * P.nb + blk) * (kT * kD * 2) : 0;
      const uint64_t page = byte >> 21, in = byte & (bst::kPage - 1);
      kv[u] = load_block(P.pk[page] + in, ok, lane_off);
      vv[u] = load_block(P.pv[page] + in, ok, lane_off);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int t = (i + u) * kT + ts;  // token of this lane's slot
      float kf[8], vf[8];
      unpack8(kv[u], kf);
      unpack8(vv[u], vf);
      float s[G];
#pragma unroll
      for (int j = 0; j < G; ++j) {
        float d = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) d = fmaf(qf[j][e], kf[e], d);
        // sum over the 16 lanes of this token row (fixed butterfly)
        d += __shfl_xor(d, 8, 64);
        d += __shfl_xor(d, 4, 64);
        d += __shfl_xor(d, 2, 64);
        d += __shfl_xor(d, 1, 64);
        s[j] = d;
      }
      if (i + u < blk_end && t < L) {  // uniform over the 16 lanes of the slot
#pragma unroll
        for (int j = 0; j < G; ++j) {
          const float mn = fmaxf(m[j], s[j]);
          const float c = m[j] == -INFINITY ? 0.f : __expf(m[j] - mn);
          const float p = __expf(s[j] - mn);
          l[j] = l[j] * c + p;
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[j][e] = fmaf(p, vf[e], acc[j][e] * c);
          m[j] = mn;
        }
      }
    }
  }

  // merge the 4 slots of a wavefront (lanes 16 and 32 apart hold the same dims)
#pragma unroll
  for (int off = 16; off <= 32; off <<= 1) {
    float m2[G], l2[G], a2[G][8];
#pragma unroll
    for (int j = 0; j < G; ++j) {
      m2[j] = __shfl_xor(m[j], off, 64);
      l2[j] = __shfl_xor(l[j], off, 64);
#pragma unroll
      for (int e = 0; e < 8; ++e) a2[j][e] = __shfl_xor(acc[j][e], off, 64);
    }
    merge_state<G>(m, l, acc, m2, l2, a2);
  }
  const int wave = tid >> 6, lane = tid & 63;
  if (lane < kLanesTok) {
#pragma unroll
    for (int j = 0; j < G; ++j) {
      if (lane == 0) {
        s_ml[wave][j][0] = m[j];
        s_ml[wave][j][1] = l[j];
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) s_acc[wave][j][dc * 8 + e] = acc[j][e];
    }
  }
  __syncthreads();
  if (wave != 0 || lane >= kLanesTok) return;
  // wavefront 0 folds in wavefronts 1..3 in order
  for (int w = 1; w < 4; ++w) {
    float m2[G], l2[G], a2[G][8];
#pragma unroll
    for (int j = 0; j < G; ++j) {
      m2[j] = s_ml[w][j][0];
      l2[j] = s_ml[w][j][1];
#pragma unroll
      for (int e = 0; e < 8; ++e) a2[j][e] = s_acc[w][j][dc * 8 + e];
    }
    merge_state<G>(m, l, acc, m2, l2, a2);
  }
#pragma unroll
  for (int j = 0; j < G; ++j) {
    const int64_t rowi = (static_cast<int64_t>(b) * P.Hq + g * G + j) * P.max_parts + part;
    if (dc == 0) {
      P.part_ml[rowi * 2] = m[j];
      P.part_ml[rowi * 2 + 1] = l[j];
    }
    float4* dst = reinterpret_cast<float4*>(P.part_acc + rowi * kD + dc * 8);
    dst[0] = make_float4(acc[j][0], acc[j][1], acc[j][2], acc[j][3]);
    dst[1] = make_float4(acc[j][4], acc[j][5], acc[j][6], acc[j][7]);
  }
}

// One wavefront per (request, query head): o = sum_p acc_p e^(m_p - M) /
// sum_p l_p e^(m_p - M) over the request's partitions, in partition order.
__global__ __launch_bounds__(64) void attn_merge(AttnParams P) {
  const int bh = blockIdx.x;  // b * Hq + h
  const int b = bh / P.Hq;
  const int lane = threadIdx.x;
  const int L = P.lens[b];
  const int n_blk = min((L + kT - 1) / kT, P.max_blocks);
  const int np = L <= 0 ? 0 : (n_blk + P.part_blocks - 1) / P.part_blocks;
  const int64_t base = static_cast<int64_t>(bh) * P.max_parts;
  float M = -INFINITY;
  for (int p = 0; p < np; ++p) M = fmaxf(M, P.part_ml[(base + p) * 2]);
  float den = 0.f, o0 = 0.f, o1 = 0.f;
  for (int p = 0; p < np; ++p) {
    const float mp = P.part_ml[(base + p) * 2];
    if (mp == -INFINITY) continue;
    const float w = __expf(mp - M);
    den = fmaf(P.part_ml[(base + p) * 2 + 1], w, den);
    const float2 a = *reinterpret_cast<const float2*>(P.part_acc + (base + p) * kD + lane * 2);
    o0 = fmaf(a.x, w, o0);
    o1 = fmaf(a.y, w, o1);
  }
  const float inv = den > 0.f ? 1.f / den : 0.f;
  const int64_t oi = static_cast<int64_t>(bh) * kD + lane * 2;
  if (P.out_bf16) {
    uint16_t* o = static_cast<uint16_t*>(P.out) + oi;
    o[0] = to_bf16(o0 * inv);
    o[1] = to_bf16(o1 * inv);
  } else {
    *reinterpret_cast<float2*>(static_cast<float*>(P.out) + oi) = make_float2(o0 * inv, o1 * inv);
  }
}

template <int G>
int launch(AttnParams& P, hipStream_t s) {
  const int64_t grid = static_cast<int64_t>(P.H) * P.B * P.n_parts;
  if (grid > 0x7fffffff) return bst::fail(BOOST_EINVAL, "grid too large");
  hipLaunchKernelGGL(attn_partition<G>, dim3(static_cast<unsigned>(grid)), dim3(kThreads),
                     0, s, P);
  BOOST_HIP(hipGetLastError());
  hipLaunchKernelGGL(attn_merge, dim3(static_cast<unsigned>(P.B * P.Hq)), dim3(64), 0, s, P);
  BOOST_HIP(hipGetLastError());
  return BOOST_OK;
}

}  // namespace

using namespace bst;

extern "C" {

int boost_paged_attn_decode(boost_ctx* ctx, const boost_kv_pool* pool, int layer,
                            const void* q, int B, int Hq, const int32_t* block_tables,
                            int max_blocks, const int32_t* ctx_lens, float scale,
                            void* out, int out_dtype, void* stream) {
  if (!ctx || !pool || !q || !block_tables || !ctx_lens || !out)
    return fail(BOOST_EINVAL, "null argument");
  if (ctx->device < 0 || !pool->d_page_table) return fail(BOOST_ENODEV, "plan-only pool");
  const boost_kv_cfg& c = pool->cfg;
  if (layer < 0 || static_cast<uint32_t>(layer) >= c.layers)
    return fail(BOOST_EINVAL, "layer %d", layer);
  if (c.head_dim != kD) return fail(BOOST_EINVAL, "attention supports head_dim 128");
  if (B < 1 || static_cast<uint32_t>(B) > c.max_batch)
    return fail(BOOST_EINVAL, "B=%d outside [1, %u]", B, c.max_batch);
  if (Hq < 1 || static_cast<uint32_t>(Hq) != c.q_heads)
    return fail(BOOST_EINVAL, "Hq=%d but the pool was sized for %u", Hq, c.q_heads);
  if (max_blocks < 1 || static_cast<uint32_t>(max_blocks) > c.max_blocks_per_seq)
    return fail(BOOST_EINVAL, "max_blocks=%d outside [1, %u]", max_blocks,
                c.max_blocks_per_seq);
  if (out_dtype != BOOST_DTYPE_F32 && out_dtype != BOOST_DTYPE_BF16)
    return fail(BOOST_EINVAL, "out_dtype %d", out_dtype);
  if (reinterpret_cast<uintptr_t>(q) & 15) return fail(BOOST_EINVAL, "q must be 16-byte aligned");
  const int H = static_cast<int>(c.kv_heads);
  const int G = Hq / H;
  AttnParams P{};
  const uint64_t pages = pool->geom.pages;
  P.pk = pool->d_page_table + (2ull * layer) * pages;
  P.pv = pool->d_page_table + (2ull * layer + 1) * pages;
  P.q = static_cast<const uint16_t*>(q);
  P.tables = block_tables;
  P.lens = ctx_lens;
  P.B = B;
  P.H = H;
  P.Hq = Hq;
  P.nb = static_cast<int>(pool->geom.nb);
  P.max_blocks = max_blocks;
  // about 2048 work items when the context allows it; at least 4 blocks each
  const int want_parts = std::max(1, (2048 + B * H - 1) / (B * H));
  P.part_blocks = std::max(4, (max_blocks + want_parts - 1) / want_parts);
  P.n_parts = (max_blocks + P.part_blocks - 1) / P.part_blocks;
  P.max_parts = pool->max_parts;
  if (P.n_parts > P.max_parts) return fail(BOOST_EINVAL, "partition scratch too small");
  P.scale = scale > 0.f ? scale : 1.0f / std::sqrt(static_cast<float>(kD));
  P.part_acc = pool->d_part_acc;
  P.part_ml = pool->d_part_ml;
  P.out = out;
  P.out_bf16 = out_dtype == BOOST_DTYPE_BF16;
  auto s = static_cast<hipStream_t>(stream);
  switch (G) {
    case 1: return launch<1>(P, s);
    case 2: return launch<2>(P, s);
    case 4: return launch<4>(P, s);
    case 8: return launch<8>(P, s);
    default: return fail(BOOST_EINVAL, "Hq/H=%d not in {1, 2, 4, 8}", G);
  }
}

}  // extern "C"
