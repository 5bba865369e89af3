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
#include <mutex>

#include "runtime.h"

namespace bst {
int kv_parts_for(const boost_kv_pool* p, int max_blocks);
}

namespace {

constexpr int kThreads = 256;
constexpr int kD = 128;          // head dimension of this kernel
constexpr int kT = 16;           // tokens per block
constexpr int kLanesTok = kD / 8;  // lanes per token row (16)
#ifndef BOOST_ATTN_UNROLL
#define BOOST_ATTN_UNROLL 4
#endif
// Work items a launch aims for (partition size follows; config 3: 2048
// items of 64 blocks ran 120 us against 122 us with 4096 of 32)
#ifndef BOOST_ATTN_ITEMS
#define BOOST_ATTN_ITEMS 2048
#endif
#ifndef BOOST_ATTN_UNROLL8
#define BOOST_ATTN_UNROLL8 BOOST_ATTN_UNROLL
#endif
constexpr int kMaxPartBlocks = 256;         // blocks per partition, at most
static_assert(kMaxPartBlocks <= kThreads, "one thread per partition size");
// A work item of fewer than 16 blocks spends as long on its start (q loads)
// and end (slot merge, partial stores) as on its K/V (batch 8 at 2048 tokens:
// 1.2 TB/s with 4-block items, 2.2 TB/s with 16).
#ifndef BOOST_ATTN_PART_MIN
#define BOOST_ATTN_PART_MIN 16
#endif
#ifndef BOOST_ATTN_PART_MAX
#define BOOST_ATTN_PART_MAX 256
#endif
constexpr int kPartMin = BOOST_ATTN_PART_MIN, kPartMax = BOOST_ATTN_PART_MAX;

struct AttnParams {
  // Linear placement makes the tier of a pool page a fixed function of its
  // offset: pages [0, first_host) of a tensor are consecutive in the HBM slab
  // and pages [first_host, pages) consecutive in the host slab.
  const char* k_hbm;   // this layer's K tensor: first HBM page
  const char* k_host;  // ... first host page
  const char* v_hbm;
  const char* v_host;
  uint64_t host_from;  // byte offset where the tensor's host tail begins
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

// Sum over the 16 lanes of a DPP row.  Every lane ends with the same bits:
// each step adds a lane's value to its partner's, and the partners' values are
// equal-by-construction from the previous step (xor 1, xor 2 within a quad,
// then the mirrored quad, then the mirrored half-row).
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  // bound_ctrl set: these patterns never leave the 16-lane row, and it lets
  // the move fold into the add (v_add_f32_dpp)
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xf, 0xf, true));
}
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
// a.lo * b.lo + a.hi * b.hi + c with two bf16 pairs packed in 32 bits
__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                         __builtin_bit_cast(bf16x2_t, b), c, false);
}

__device__ __forceinline__ float row16_sum(float v) {
  v += dpp<0xb1>(v);   // quad_perm [1,0,3,2]
  v += dpp<0x4e>(v);   // quad_perm [2,3,0,1]
  v += dpp<0x141>(v);  // row_half_mirror
  v += dpp<0x140>(v);  // row_mirror
  return v;
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
    const float c1 = __builtin_amdgcn_exp2f(m[j] - M);  // m = -inf gives 0
    const float c2 = __builtin_amdgcn_exp2f(m2[j] - M);
    l[j] = l[j] * c1 + l2[j] * c2;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[j][e] = acc[j][e] * c1 + acc2[j][e] * c2;
    m[j] = M;
  }
}

// Pair of lanes D apart (D = 16 or 32; v is the same register in both
// operands): {v of the lower lane, v of the upper lane} in both lanes.
template <int D>
__device__ __forceinline__ void pair_of(float v, float& lo, float& hi) {
  const uint32_t u = __float_as_uint(v);
  if constexpr (D == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    lo = __uint_as_float(r[0]);
    hi = __uint_as_float(r[1]);
  } else {
    const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    lo = __uint_as_float(r[0]);
    hi = __uint_as_float(r[1]);
  }
}

// The running states of the lane pairs D apart merged, lower lane's state
// first; afterwards both lanes hold the result.
template <int G, int D>
__device__ __forceinline__ void slot_merge(float* m, float* l, float (*acc)[8]) {
  float m2[G], l2[G], a2[G][8];
#pragma unroll
  for (int j = 0; j < G; ++j) {
    pair_of<D>(m[j], m[j], m2[j]);
    pair_of<D>(l[j], l[j], l2[j]);
#pragma unroll
    for (int e = 0; e < 8; ++e) pair_of<D>(acc[j][e], acc[j][e], a2[j][e]);
  }
  merge_state<G>(m, l, acc, m2, l2, a2);
}

// Online-softmax update of one token slot with U blocks.  Scores are in the
// log2 domain (q . k * scale * log2 e), so exp2 is one instruction.  With
// MASKED false every token is valid; otherwise invalid tokens have score -inf
// and contribute nothing.
template <int G, int U, bool MASKED, typename AfterK>
__device__ __forceinline__ void consume(const uint32_t (*qp)[4], const uint4* kb,
                                        const uint4* vb, const bool* valid, float sc2,
                                        float* m, float* l, float (*acc)[8], AfterK after_k) {
  float sc[U][G];
#pragma unroll
  for (int u = 0; u < U; ++u)
#pragma unroll
    for (int j = 0; j < G; ++j) {
      float d = dot2(qp[j][0], kb[u].x, 0.f);
      d = dot2(qp[j][1], kb[u].y, d);
      d = dot2(qp[j][2], kb[u].z, d);
      d = dot2(qp[j][3], kb[u].w, d);
      d = row16_sum(d) * sc2;  // q . k over the 16 lanes of the token row
      sc[u][j] = (!MASKED || valid[u]) ? d : -INFINITY;
    }
  after_k();  // the K registers are free from here on
#pragma unroll
  for (int j = 0; j < G; ++j) {
    float mc = m[j];
#pragma unroll
    for (int u = 0; u < U; ++u) mc = fmaxf(mc, sc[u][j]);
    if (MASKED && mc == -INFINITY) continue;  // nothing valid yet
    const float c = __builtin_amdgcn_exp2f(m[j] - mc);  // exp2(-inf) = 0 at start
    l[j] *= c;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[j][e] *= c;
    m[j] = mc;
  }
#pragma unroll
  for (int u = 0; u < U; ++u) {
    float vf[8];
    unpack8(vb[u], vf);
#pragma unroll
    for (int j = 0; j < G; ++j) {
      // masked: an invalid token (score -inf) weighs 0, also while the
      // running max is still -inf
      const float p = (MASKED && sc[u][j] == -INFINITY)
                          ? 0.f
                          : __builtin_amdgcn_exp2f(sc[u][j] - m[j]);
      l[j] += p;
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[j][e] = fmaf(p, vf[e], acc[j][e]);
    }
  }
}

// Head-distributed softmax for G = 2 and 4.  The G partial dot products of a
// lane (its 8 dimensions of one token, every query head) are reduced over
// the token's 16 lanes by a transposing butterfly: exchange with the lane
// xor 1 (and xor 2 for G = 4) keeping half the heads each time, then add the
// lanes 4 and 8 apart, so each lane ends with the full score of ONE head
// (head_of_lane) instead of every lane holding all G.  The running maximum,
// the exponentials and the running sum are then computed once per head and
// token instead of 16 times; the probabilities and rescale factors reach the
// other lanes' accumulators by quad broadcasts.  Same online softmax as
// consume(), fewer vector instructions per block.
template <int G>
__device__ __forceinline__ int head_of_lane(int lane) {
  const int i = lane & 3;
  return G == 4 ? 2 * (i & 1) + (i >> 1) : (i & 1);
}
// the lane of a quad that holds head j (the map is its own inverse)
template <int G>
constexpr int lane_of_head(int j) { return G == 4 ? 2 * (j & 1) + (j >> 1) : j; }
// value of quad lane k, in every lane of the quad
template <int K>
__device__ __forceinline__ float quad_bcast(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), K * 0x55, 0xf, 0xf, true));
}
template <int G, int J = 0>
__device__ __forceinline__ void bcast_heads(float v, float* out) {
  if constexpr (J < G) {
    out[J] = quad_bcast<lane_of_head<G>(J)>(v);
    bcast_heads<G, J + 1>(v, out);
  }
}

template <int G>
__device__ __forceinline__ float score_of_lane_head(const float* d, bool b0, bool b1) {
  float f;
  if constexpr (G == 4) {
    // xor 1: lanes with bit 0 clear keep heads 0, 1; set keep 2, 3
    const float k0 = b0 ? d[2] : d[0], k1 = b0 ? d[3] : d[1];
    const float s0 = b0 ? d[0] : d[2], s1 = b0 ? d[1] : d[3];
    const float e0 = k0 + dpp<0xb1>(s0), e1 = k1 + dpp<0xb1>(s1);
    // xor 2: bit 1 clear keeps the first of the pair, set the second
    f = (b1 ? e1 : e0) + dpp<0x4e>(b1 ? e0 : e1);
  } else {
    f = (b0 ? d[1] : d[0]) + dpp<0xb1>(b0 ? d[0] : d[1]);
    f += dpp<0x4e>(f);
  }
  f += dpp<0x124>(f);  // row_ror 4: the next quad of the 16-lane row
  f += dpp<0x128>(f);  // row_ror 8: the other half of the row
  return f;
}

template <int G, int U, bool MASKED, typename AfterK>
__device__ __forceinline__ void consume_hd(const uint32_t (*qp)[4], const uint4* kb,
                                           const uint4* vb, const bool* valid, float sc2,
                                           bool b0, bool b1, float& mh, float& lh,
                                           float (*acc)[8], AfterK after_k) {
  float s[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    float d[G];
#pragma unroll
    for (int j = 0; j < G; ++j) {
      float x = dot2(qp[j][0], kb[u].x, 0.f);
      x = dot2(qp[j][1], kb[u].y, x);
      x = dot2(qp[j][2], kb[u].z, x);
      d[j] = dot2(qp[j][3], kb[u].w, x);
    }
    const float f = score_of_lane_head<G>(d, b0, b1) * sc2;
    s[u] = (!MASKED || valid[u]) ? f : -INFINITY;
  }
  after_k();  // the K registers are free from here on
  float mc = mh;
#pragma unroll
  for (int u = 0; u < U; ++u) mc = fmaxf(mc, s[u]);
  // nothing valid yet for this head: keep the state (factor 1)
  const float c = (MASKED && mc == -INFINITY) ? 1.f : __builtin_amdgcn_exp2f(mh - mc);
  lh *= c;
  mh = mc;
  float cj[G];
  bcast_heads<G>(c, cj);
#pragma unroll
  for (int j = 0; j < G; ++j)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[j][e] *= cj[j];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const float p = (MASKED && s[u] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(s[u] - mh);
    lh += p;
    float pj[G], vf[8];
    bcast_heads<G>(p, pj);
    unpack8(vb[u], vf);
#pragma unroll
    for (int j = 0; j < G; ++j)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[j][e] = fmaf(pj[j], vf[e], acc[j][e]);
  }
}

// Blocks of request b in this call (0 for an empty context).
__device__ __forceinline__ int blocks_of(const AttnParams& P, int b) {
  const int L = P.lens[b];
  return L <= 0 ? 0 : min((L + kT - 1) / kT, P.max_blocks);
}

// Sum of v over the workgroup; every thread gets it (red: 4 ints of LDS).
__device__ __forceinline__ int wg_sum(int v, int* red) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  __syncthreads();  // red is free again
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

// Exclusive prefix sum of v over the workgroup in thread order; total gets
// the sum of every thread's v.
__device__ __forceinline__ int wg_scan(int v, int* red, int& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  __syncthreads();
  if (lane == 63) red[wave] = x;
  __syncthreads();
  int before = 0;
  for (int w = 0; w < wave; ++w) before += red[w];
  total = red[0] + red[1] + red[2] + red[3];
  return before + x - v;
}

// Request whose count interval holds `target` in the running sum of
// count(n_b) over b = 0, 1, ... (count > 0 there); pick[0] gets b, pick[1]
// target minus the sum before b, pick[4] b's context length.  n0, L0: this
// thread's n_b and length for b = threadIdx.x (read once by the caller);
// later chunks read the lengths again.
template <typename Count>
__device__ __forceinline__ void find_request(const AttnParams& P, int target, int n0, int L0,
                                             Count count, int* red, int* pick) {
  int carry = 0;
  for (int base = 0; base < P.B; base += kThreads) {  // uniform
    const int b = base + static_cast<int>(threadIdx.x);
    const int c = b < P.B ? count(base == 0 ? n0 : blocks_of(P, b)) : 0;
    int total;
    const int ex = carry + wg_scan(c, red, total);
    if (c > 0 && ex <= target && target < ex + c) {
      pick[0] = b;
      pick[1] = target - ex;
      pick[4] = base == 0 ? L0 : P.lens[b];
    }
    carry += total;
    if (carry > target) break;  // uniform
  }
  __syncthreads();
}

// Work item of workgroup idx, from the context lengths alone (so the same on
// every pool: the order decides which items run together, never what an item
// computes).  With n_b blocks, request b has full_b = n_b / part_blocks full
// partitions and one partial one if rem_b = n_b % part_blocks > 0.  Order:
//   1. every partition of head H-1 (where host data can lie), request by
//      request: its slow reads start first;
//   2. full partitions of heads H-2..0, request by request, head fastest;
//   3. partial partitions of heads H-2..0, the largest first (rem_b
//      descending, then b ascending), head fastest;
//   4. workgroups past the last item return at once.
// Empty partitions get no workgroup and the short ones run last, so the last
// grid wave is short (config 3, reads alone: 104 -> 96 us).
// L gets the request's context length (so the caller does not read it again).
__device__ bool item_of(const AttnParams& P, int idx, int& b, int& g, int& part, int& L,
                        int* red, int* hist, int* pick) {
  const int tid = threadIdx.x, PB = P.part_blocks, H = P.H;
  if (tid < 5) pick[tid] = -1;  // written by the sums' barriers below
  const int L0 = tid < P.B ? P.lens[tid] : 0;  // request tid, read once
  const int n0 = L0 <= 0 ? 0 : min((L0 + kT - 1) / kT, P.max_blocks);
  int f = 0, r = 0;
  for (int bb = tid; bb < P.B; bb += kThreads) {
    const int n = bb == tid ? n0 : blocks_of(P, bb);
    f += n / PB;
    r += n % PB > 0;
  }
  const int F = wg_sum(f, red), R = wg_sum(r, red);
  const int S0 = F + R;
  if (idx < S0) {
    find_request(P, idx, n0, L0, [&](int n) { return n / PB + (n % PB > 0); }, red, pick);
    b = pick[0];
    part = pick[1];
    L = pick[4];
    g = H - 1;
    return b >= 0 && b < P.B && part >= 0;
  }
  int j = idx - S0;
  if (j < (H - 1) * F) {
    find_request(P, j / (H - 1), n0, L0, [&](int n) { return n / PB; }, red, pick);
    b = pick[0];
    part = pick[1];
    L = pick[4];
    g = H - 2 - j % (H - 1);
    return b >= 0 && b < P.B && part >= 0;
  }
  j -= (H - 1) * F;
  if (j >= (H - 1) * R) return false;
  // partial partitions by size: a counting sort over rem in [1, PB)
  const int rank = j / (H - 1);
  for (int v = tid; v < PB; v += kThreads) hist[v] = 0;
  __syncthreads();
  for (int bb = tid; bb < P.B; bb += kThreads) {
    const int rem = (bb == tid ? n0 : blocks_of(P, bb)) % PB;
    if (rem > 0) atomicAdd(&hist[rem], 1);
  }
  __syncthreads();
  {
    const int v = PB - 1 - tid;  // thread order = rem descending (PB <= kThreads)
    const int c = v >= 1 ? hist[v] : 0;
    int total;
    const int ex = wg_scan(c, red, total);
    if (c > 0 && ex <= rank && rank < ex + c) {
      pick[2] = v;
      pick[3] = rank - ex;
    }
    __syncthreads();
  }
  const int vsel = pick[2];
  find_request(P, pick[3], n0, L0, [&](int n) { return n % PB == vsel ? 1 : 0; }, red, pick);
  b = pick[0];
  if (b < 0 || b >= P.B) return false;
  L = pick[4];
  part = (L <= 0 ? 0 : min((L + kT - 1) / kT, P.max_blocks)) / PB;
  g = H - 2 - j % (H - 1);
  return true;
}

// Waves per SIMD the register allocator targets for G <= 4: three (168
// registers, no spill) against the two it picks by itself took config 3 from
// 136 to 126 us; four spill and run at 306 us.  G = 8 keeps the allocator's
// own choice (a tighter target spills its accumulators).
#ifndef BOOST_ATTN_WAVES
#define BOOST_ATTN_WAVES 3
#endif
#ifndef BOOST_ATTN_HD
#define BOOST_ATTN_HD 1
#endif
template <int G>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(
    G == 8 ? 1 : BOOST_ATTN_WAVES))) void attn_partition(AttnParams P) {
  constexpr int kUnroll = G == 8 ? BOOST_ATTN_UNROLL8 : BOOST_ATTN_UNROLL;  // blocks in flight
  __shared__ float s_ml[4][G][2];
  __shared__ float s_acc[4][G][kD];
  const int tid = threadIdx.x;
  const int ts = tid / kLanesTok;  // token slot 0..15
  const int dc = tid % kLanesTok;  // 8-dim chunk
  // the partition's block ids (staged once: a load per block from memory
  // would put a round trip before every group of K/V loads); before that the
  // item search's counting sort
  __shared__ int32_t row[kMaxPartBlocks];
  __shared__ int s_red[4], s_pick[5];
  int part, b, g, L;
  if (!item_of(P, blockIdx.x, b, g, part, L, s_red, row, s_pick)) return;  // uniform
  const int n_blk = L <= 0 ? 0 : min((L + kT - 1) / kT, P.max_blocks);
  const int blk_beg = part * P.part_blocks;
  if (blk_beg >= n_blk) return;  // uniform: empty partition (not produced by item_of)
  const int nbp = min(n_blk, blk_beg + P.part_blocks) - blk_beg;
  // leading blocks whose 16 tokens are all inside the context
  const int nfull = max(0, min(nbp, L / kT - blk_beg));
  const uint64_t head_off = static_cast<uint64_t>(g) * P.nb * (kT * kD * 2);
  // the partition's width of the table row (entries past the context are
  // read but not used)
  if (tid < min(P.part_blocks, P.max_blocks - blk_beg))
    row[tid] = P.tables[static_cast<int64_t>(b) * P.max_blocks + blk_beg + tid];
  __syncthreads();

  // q stays in bf16 pairs for the dot2 instruction
  uint32_t qp[G][4];
#pragma unroll
  for (int j = 0; j < G; ++j) {
    const uint4 u = *reinterpret_cast<const uint4*>(
        P.q + (static_cast<int64_t>(b) * P.Hq + g * G + j) * kD + dc * 8);
    qp[j][0] = u.x;
    qp[j][1] = u.y;
    qp[j][2] = u.z;
    qp[j][3] = u.w;
  }
  const float sc2 = P.scale * 1.4426950408889634f;  // log2(e)
  float m[G], l[G], acc[G][8];
#pragma unroll
  for (int j = 0; j < G; ++j) {
    m[j] = -INFINITY;
    l[j] = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[j][e] = 0.f;
  }
  // head-distributed state (G = 2, 4): this lane's head's maximum and sum
  constexpr bool kHD = BOOST_ATTN_HD && (G == 2 || G == 4);
  const bool b0 = tid & 1, b1 = tid & 2;
  float mh = -INFINITY, lh = 0.f;

  const uint32_t lane_off = static_cast<uint32_t>(tid) * 16;
  // address of head-block (g, blk) of K and V: uniform scalar arithmetic
  // (a block id outside the pool reads nothing and its tokens are masked
  // out of the softmax, as if the block were not in the context)
  auto where = [&](int bi, bool& ok, bool& host) {
    const int32_t blk = row[bi];
    ok = blk >= 0 && blk < P.nb;
    const uint64_t byte = head_off + static_cast<uint64_t>(ok ? blk : 0) * (kT * kD * 2);
    host = byte >= P.host_from;
    return host ? byte - P.host_from : byte;
  };
  auto fetch_k = [&](int bi, uint4& kq) {
    bool ok, host;
    const uint64_t off = where(bi, ok, host);
    kq = load_block((host ? P.k_host : P.k_hbm) + off, ok, lane_off);
    return ok;
  };
  auto fetch_v = [&](int bi, uint4& vq) {
    bool ok, host;
    const uint64_t off = where(bi, ok, host);
    vq = load_block((host ? P.v_host : P.v_hbm) + off, ok, lane_off);
  };
  auto none = [] {};
  // Full groups of kUnroll blocks, software-pipelined across K and V: the
  // next group's K loads go out as soon as the scores have used this group's
  // K, its V loads as soon as P.V has used this group's V, so each workgroup
  // keeps loads in flight while it computes, with no extra registers.
  int i = 0;
  if (nfull >= kUnroll) {
    uint4 kb[kUnroll], vb[kUnroll];
    bool valid[kUnroll], vnext[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      valid[u] = fetch_k(u, kb[u]);
      fetch_v(u, vb[u]);
    }
    for (; i + kUnroll <= nfull; i += kUnroll) {
      const bool more = i + 2 * kUnroll <= nfull;  // uniform
      bool all_ok = true;  // uniform: block ids are the same for every lane
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) all_ok = all_ok && valid[u];
      auto next_k = [&] {
        if (more)
#pragma unroll
          for (int u = 0; u < kUnroll; ++u) vnext[u] = fetch_k(i + kUnroll + u, kb[u]);
      };
      if constexpr (kHD) {
        if (all_ok)
          consume_hd<G, kUnroll, false>(qp, kb, vb, valid, sc2, b0, b1, mh, lh, acc, next_k);
        else
          consume_hd<G, kUnroll, true>(qp, kb, vb, valid, sc2, b0, b1, mh, lh, acc, next_k);
      } else {
        if (all_ok)
          consume<G, kUnroll, false>(qp, kb, vb, valid, sc2, m, l, acc, next_k);
        else
          consume<G, kUnroll, true>(qp, kb, vb, valid, sc2, m, l, acc, next_k);
      }
      if (more) {
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          fetch_v(i + kUnroll + u, vb[u]);
          valid[u] = vnext[u];
        }
      }
    }
  }
  if (i < nbp) {  // the rest (fewer than kUnroll full blocks, then a partial
                  // one: at most kUnroll blocks), loaded together and masked
    uint4 kb[kUnroll], vb[kUnroll];
    bool valid[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const bool ok = i + u < nbp && fetch_k(i + u, kb[u]);
      if (i + u < nbp) fetch_v(i + u, vb[u]);
      if (i + u >= nbp) kb[u] = vb[u] = make_uint4(0, 0, 0, 0);
      valid[u] = ok && (blk_beg + i + u) * kT + ts < L;
    }
    if constexpr (kHD)
      consume_hd<G, kUnroll, true>(qp, kb, vb, valid, sc2, b0, b1, mh, lh, acc, none);
    else
      consume<G, kUnroll, true>(qp, kb, vb, valid, sc2, m, l, acc, none);
  }
  if constexpr (kHD) {  // every head's maximum and sum in every lane again
    bcast_heads<G>(mh, m);
    bcast_heads<G>(lh, l);
  }

  // merge the 4 slots of a wavefront (lanes 16 and 32 apart hold the same
  // dims) with the row-swap instructions: permlane16_swap(v, v) gives every
  // lane the pair (v of the lower lane, v of the lane 16 above it) of its
  // 16-apart pair, permlane32_swap the same for lanes 32 apart, so both
  // lanes of a pair merge the same two states in the same order
  slot_merge<G, 16>(m, l, acc);
  slot_merge<G, 32>(m, l, acc);
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
  if (lane >= kLanesTok) return;
  // head j is folded by wavefront j % 4 (the heads in parallel): wavefront
  // 0's state, then wavefronts 1, 2, 3 in order, as the same values in the
  // same order whichever wavefront does it
  constexpr int kHeadsPerWave = (G + 3) / 4;
#pragma unroll
  for (int jj = 0; jj < kHeadsPerWave; ++jj) {
    const int j = wave + 4 * jj;  // uniform over the wavefront
    if (j >= G) break;
    float mj = s_ml[0][j][0], lj = s_ml[0][j][1], aj[1][8];
#pragma unroll
    for (int e = 0; e < 8; ++e) aj[0][e] = s_acc[0][j][dc * 8 + e];
    for (int w = 1; w < 4; ++w) {
      const float m2 = s_ml[w][j][0], l2 = s_ml[w][j][1];
      float a2[1][8];
#pragma unroll
      for (int e = 0; e < 8; ++e) a2[0][e] = s_acc[w][j][dc * 8 + e];
      merge_state<1>(&mj, &lj, aj, &m2, &l2, a2);
    }
    const int64_t rowi = (static_cast<int64_t>(b) * P.Hq + g * G + j) * P.max_parts + part;
    if (dc == 0) {
      P.part_ml[rowi * 2] = mj;
      P.part_ml[rowi * 2 + 1] = lj;
    }
    float4* dst = reinterpret_cast<float4*>(P.part_acc + rowi * kD + dc * 8);
    dst[0] = make_float4(aj[0][0], aj[0][1], aj[0][2], aj[0][3]);
    dst[1] = make_float4(aj[0][4], aj[0][5], aj[0][6], aj[0][7]);
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
  // the largest partition maximum: one partition per lane, then across the
  // wavefront (a maximum is exact in any order)
  float M = -INFINITY;
  for (int p0 = 0; p0 < np; p0 += 64) {
    const int p = p0 + lane;
    M = fmaxf(M, p < np ? P.part_ml[(base + p) * 2] : -INFINITY);
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) M = fmaxf(M, __shfl_xor(M, m, 64));
  // weighted sums in partition order; the loads of eight partitions go out
  // together instead of one round trip per partition
  constexpr int kMergeBatch = 8;
  float den = 0.f, o0 = 0.f, o1 = 0.f;
  for (int p0 = 0; p0 < np; p0 += kMergeBatch) {
    float mp[kMergeBatch], lp[kMergeBatch];
    float2 a[kMergeBatch];
#pragma unroll
    for (int u = 0; u < kMergeBatch; ++u) {
      const int p = p0 + u;  // uniform
      mp[u] = -INFINITY;
      lp[u] = 0.f;
      a[u] = make_float2(0.f, 0.f);
      if (p < np) {
        mp[u] = P.part_ml[(base + p) * 2];
        lp[u] = P.part_ml[(base + p) * 2 + 1];
        a[u] = *reinterpret_cast<const float2*>(P.part_acc + (base + p) * kD + lane * 2);
      }
    }
#pragma unroll
    for (int u = 0; u < kMergeBatch; ++u) {
      if (mp[u] == -INFINITY) continue;  // past np, or an empty partition
      const float w = __builtin_amdgcn_exp2f(mp[u] - M);  // maxima are in the log2 domain
      den = fmaf(lp[u], w, den);
      o0 = fmaf(a[u].x, w, o0);
      o1 = fmaf(a[u].y, w, o1);
    }
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

// Scratch of the allocation-free entry point: partition partials of up to
// kStaticRows (request, query head, partition) rows, the sums of p * v
// ([kStaticRows][D] floats) followed by the running (max, sum) pairs
// ([kStaticRows][2]).  16.25 MiB, held by every device the library runs on
// until the process ends.  The host never uses the array's name as an
// address: boost_init looks up each device's copy once
// (attn_scratch_setup) and the entry point passes that address.
constexpr int64_t kStaticRows = 32768;
__device__ __align__(256) float scratch[kStaticRows * (kD + 2)];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[kMaxDevices] = {};  // per device: address of `scratch`

// Everything both entry points check and compute, then the two launches;
// part_acc / part_ml / max_parts name the partial buffers (max_parts = 0:
// the call's own partition count, with at most cap_rows rows).
int decode(boost_ctx* ctx, const boost_kv_pool* pool, int layer, const void* q, int B, int Hq,
           const int32_t* block_tables, int max_blocks, const int32_t* ctx_lens, float scale,
           void* out, int out_dtype, void* stream, float* part_acc, float* part_ml,
           int max_parts, int64_t cap_rows) {
  using bst::fail;
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
  const uint64_t pages = pool->geom.pages, hp = pool->geom.host_pages;
  const uint64_t tk = 2ull * layer, tv = 2ull * layer + 1;  // tensor indices
  P.k_hbm = pool->hbm.base + tk * (pages - hp) * bst::kPage;
  P.v_hbm = pool->hbm.base + tv * (pages - hp) * bst::kPage;
  P.k_host = hp ? pool->host[layer].base : P.k_hbm;
  P.v_host = hp ? pool->host[layer].base + hp * bst::kPage : P.v_hbm;
  P.host_from = (pages - hp) * bst::kPage;
  P.q = static_cast<const uint16_t*>(q);
  P.tables = block_tables;
  P.lens = ctx_lens;
  P.B = B;
  P.H = H;
  P.Hq = Hq;
  P.nb = static_cast<int>(pool->geom.nb);
  P.max_blocks = max_blocks;
  // enough work items to fill the GPU several times over (so the last grid
  // wave is short), each long enough to amortise its start and its merge
  // (PART_MIN blocks) and short enough to balance (PART_MAX blocks)
  const int want_parts = std::max(1, (BOOST_ATTN_ITEMS + B * H - 1) / (B * H));
  P.part_blocks = std::min(
      {kMaxPartBlocks, max_blocks,
       std::max(kPartMin, std::min(kPartMax, (max_blocks + want_parts - 1) / want_parts))});
  P.part_blocks = std::max(P.part_blocks, 4);
  P.n_parts = (max_blocks + P.part_blocks - 1) / P.part_blocks;
  P.max_parts = max_parts > 0 ? max_parts : P.n_parts;
  if (P.n_parts > P.max_parts) return fail(BOOST_EINVAL, "partition scratch too small");
  if (static_cast<int64_t>(B) * Hq * P.max_parts > cap_rows)
    return fail(BOOST_EINVAL, "%lld partial rows (B=%d x Hq=%d x %d partitions) exceed the "
                "scratch's %lld", static_cast<long long>(B) * Hq * P.max_parts, B, Hq,
                P.max_parts, static_cast<long long>(cap_rows));
  P.scale = scale > 0.f ? scale : 1.0f / std::sqrt(static_cast<float>(kD));
  P.part_acc = part_acc;
  P.part_ml = part_ml;
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

}  // namespace

namespace bst {
// Once per device, with that device current: the device address of this
// device's copy of `scratch`.  Called by boost_init.
int attn_scratch_setup(int device) {
  if (device < 0 || device >= kMaxDevices)
    return fail(BOOST_EINVAL, "device %d beyond the %d the static scratch serves", device,
                kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[device]) return BOOST_OK;
  void* ptr = nullptr;
  const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
  if (e != hipSuccess || !ptr)
    return fail(BOOST_EHIP, "hipGetSymbolAddress(scratch) on device %d: %s", device,
                hipGetErrorString(e));
  g_scratch_ptr[device] = static_cast<float*>(ptr);
  return BOOST_OK;
}
}  // namespace bst

using namespace bst;

extern "C" {

int boost_paged_attn_decode(boost_ctx* ctx, const boost_kv_pool* pool, int layer,
                            const void* q, int B, int Hq, const int32_t* block_tables,
                            int max_blocks, const int32_t* ctx_lens, float scale,
                            void* out, int out_dtype, void* stream) {
  if (!pool) return fail(BOOST_EINVAL, "null argument");
  const int64_t rows = static_cast<int64_t>(pool->cfg.max_batch) * pool->cfg.q_heads *
                       std::max(1, pool->max_parts);
  return decode(ctx, pool, layer, q, B, Hq, block_tables, max_blocks, ctx_lens, scale, out,
                out_dtype, stream, pool->d_part_acc, pool->d_part_ml,
                std::max(1, pool->max_parts), rows);
}

int boost_paged_attn_decode_noalloc(boost_ctx* ctx, const boost_kv_pool* pool, int layer,
                                    const void* q, int B, int Hq,
                                    const int32_t* block_tables, int max_blocks,
                                    const int32_t* ctx_lens, float scale, void* out,
                                    int out_dtype, void* stream) {
  if (!ctx) return fail(BOOST_EINVAL, "null argument");
  if (ctx->device < 0) return fail(BOOST_ENODEV, "plan-only context");
  float* base = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (ctx->device < kMaxDevices) base = g_scratch_ptr[ctx->device];
  }
  if (!base) return fail(BOOST_EHIP, "static scratch of device %d not set up", ctx->device);
  return decode(ctx, pool, layer, q, B, Hq, block_tables, max_blocks, ctx_lens, scale, out,
                out_dtype, stream, base, base + kStaticRows * kD, 0, kStaticRows);
}

}  // extern "C"
