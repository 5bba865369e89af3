// a4: decode GEMV over tiered pages, y[b, n] = sum_k W[n, k] x[b, k].
//
// W is an [N, K] row-major bf16 matrix placed page by page on HBM or host
// (§3.1 modulo placement).  The work unit of a workgroup is a group of rows
// restricted to ONE page, so a workgroup reads one tier for its whole life
// (§3.2 CTA-level confinement: a workgroup never mixes tiers).  A row that
// straddles a page boundary is split-K across the two workgroups of those
// pages; each stores its partial sum and a small second kernel adds them in a
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

#include "lds_dma.h"
#include "runtime.h"

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int64_t kPageElems = static_cast<int64_t>(bst::kPage / 2);

struct GemvParams {
  const char* const* page_table;
  const uint8_t* tiers;  // tier of every page
  const int32_t* hbm_pages;
  const int32_t* host_pages;
  // the same in closed form where the tensor's map is modulo placement:
  // page p is on host iff (p / lay_SP) % lay_M == lay_M - 1 (lay_M = 0: no
  // host page), each tier's pages sit in page order in one slab; lay_M < 0:
  // read the tables
  const char* hbm_base;
  const char* host_base;
  int lay_M;
  int lay_SP;
  int n_pages;
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
  int B;     // batch rows of x and y
  int join;  // 1: a cut row between two pages of one tier is summed by one unit
  int tail_first;  // 1: the last unit of every page is dispatched before the others
  int S;     // K slices per row group (matrix-core path; 1 = no split)
  float* ws;  // S > 1: [S][B][N] partials, then [(n_pages + 1) * 2][S][B] of cut rows
  float* partial;  // [(n_pages + 1) boundaries][2 sides][kMaxGemvBatch]
  // host side only: a caller's buffer for the K slices (the layout of ws,
  // summed by the consumer instead of split_reduce) and its size in floats
  float* slices;
  int64_t slice_floats;
};

// Page lookups: the closed form of modulo placement where the tensor has it
// (no dependent load before a unit's first weight load), else the tables.
__device__ __forceinline__ const char* page_addr(const GemvParams& P, int p) {
  if (P.lay_M < 0) return P.page_table[p];
  if (P.lay_M == 0) return P.hbm_base + static_cast<int64_t>(p) * bst::kPage;
  const int g = p / P.lay_SP, before = g / P.lay_M;  // host superpages before g's group
  if (g % P.lay_M == P.lay_M - 1)
    return P.host_base + (static_cast<int64_t>(before) * P.lay_SP + p % P.lay_SP) * bst::kPage;
  return P.hbm_base + (static_cast<int64_t>(p) - static_cast<int64_t>(before) * P.lay_SP) *
                          bst::kPage;
}
__device__ __forceinline__ uint8_t page_tier(const GemvParams& P, int p) {
  if (P.lay_M < 0) return P.tiers[p];
  return P.lay_M > 0 && (p / P.lay_SP) % P.lay_M == P.lay_M - 1 ? BOOST_TIER_HOST
                                                                 : BOOST_TIER_HBM;
}
// the i-th HBM page and the k-th host page in page order
__device__ __forceinline__ int hbm_page(const GemvParams& P, int i) {
  if (P.lay_M < 0) return P.hbm_pages[i];
  if (P.lay_M == 0) return i;
  const int per = (P.lay_M - 1) * P.lay_SP;  // HBM pages of a group of M superpages
  return (i / per) * P.lay_M * P.lay_SP + i % per;
}
__device__ __forceinline__ int host_page(const GemvParams& P, int k) {
  if (P.lay_M < 0) return P.host_pages[k];
  return (k / P.lay_SP) * P.lay_M * P.lay_SP + (P.lay_M - 1) * P.lay_SP + k % P.lay_SP;
}

__device__ __forceinline__ float lo_bf16(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t v) {
  return __uint_as_float(v & 0xffff0000u);
}

typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
// a.lo * b.lo + a.hi * b.hi + c for two packed bf16 pairs (products of bf16
// values are exact in fp32; the sum is accumulated in fp32)
__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                         __builtin_bit_cast(bf16x2_t, b), c, false);
}

// 8-element dot product of two 16-byte bf16 vectors, accumulated into acc in
// element order
__device__ __forceinline__ float dot8(const uint4& w, const uint4& x, float acc) {
  acc = dot2(w.x, x.x, acc);
  acc = dot2(w.y, x.y, acc);
  acc = dot2(w.z, x.z, acc);
  acc = dot2(w.w, x.w, acc);
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

// A row cut by page boundary `bnd` (between pages bnd-1 and bnd) is summed by
// two workgroups, one per page; each stores its partial sum here (side 0 = the
// part on the earlier page) and split_fixup adds them after the main kernel.
template <int B>
__device__ __forceinline__ void store_split(const GemvParams& P, int bnd, int side,
                                            const float* v) {
  float* slot = P.partial + (static_cast<int64_t>(bnd) * 2 + side) * bst::kMaxGemvBatch;
#pragma unroll
  for (int b = 0; b < B; ++b) slot[b] = v[b];
}

// Raw buffer resource over `bytes` bytes at `base` (CDNA: offsets at or past
// num_records read as zero, with no fault).  Word 3 selects 32-bit data.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base,
                                                            uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0,
                                           static_cast<int>(bytes), 0x00020000);
}

// Cache policy of weight loads: 2 = non-temporal (streamed once per token,
// no reuse to keep in L2).
#ifndef BOOST_W_AUX
#define BOOST_W_AUX 2
#endif
template <int AUX = 0>
__device__ __forceinline__ uint4 load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  auto v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, AUX);
  return *reinterpret_cast<uint4*>(&v);
}

// The same for a base and size the caller knows to be uniform over the
// wavefront: taken through readfirstlane, so the descriptor lives in scalar
// registers even where the compiler cannot prove the uniformity itself
// (otherwise every load through it becomes a loop over distinct descriptors).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc_uniform(const void* base,
                                                                    uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a >> 32));
  const uint32_t n = __builtin_amdgcn_readfirstlane(bytes);
  return make_rsrc(reinterpret_cast<const void*>((static_cast<uint64_t>(hi) << 32) | lo), n);
}

// Offsets at or above this are outside every resource used here (a page is
// 2 MiB, x is at most 8 * 512 K elements), so the load returns zero.
constexpr uint32_t kOOB = 0x80000000u;

// Most K slices a matrix-core call splits a row group into.
#ifndef BOOST_MFMA_MAX_SLICES
#define BOOST_MFMA_MAX_SLICES 8
#endif
constexpr int kMaxSlices = BOOST_MFMA_MAX_SLICES;

// Accumulate this wavefront's columns [k_beg, k_end) of its RW rows from
// the page behind resource wr; row i's column 0 sits at byte offset ro[i]
// (offsets outside the page read as zero).
template <int B, int RW, int UN>
__device__ __forceinline__ void accumulate(__amdgpu_buffer_rsrc_t wr,
                                           __amdgpu_buffer_rsrc_t xr, const uint32_t* ro,
                                           int64_t K, int64_t k_beg, int64_t k_end, int lane,
                                           float (*acc)[B]) {
  constexpr int kStep = 64 * 8;  // columns covered by one load of a wavefront
  for (int64_t kb = k_beg; kb < k_end; kb += kStep * UN) {
    uint4 wv[UN][RW], xv[UN][B];
#pragma unroll
    for (int u = 0; u < UN; ++u) {
      const int64_t kc = kb + u * kStep + lane * 8;
      const uint32_t oob = kc < k_end ? 0u : kOOB;
      const uint32_t kc2 = static_cast<uint32_t>(kc * 2);
#pragma unroll
      for (int b = 0; b < B; ++b)
        xv[u][b] = load16(xr, (static_cast<uint32_t>(b * K * 2) + kc2) | oob);
#pragma unroll
      for (int i = 0; i < RW; ++i) wv[u][i] = load16<BOOST_W_AUX>(wr, (ro[i] + kc2) | oob);
    }
#pragma unroll
    for (int u = 0; u < UN; ++u)
#pragma unroll
      for (int i = 0; i < RW; ++i)
#pragma unroll
        for (int b = 0; b < B; ++b) acc[i][b] = dot8(wv[u][i], xv[u][b], acc[i][b]);
  }
}

// One unit: a group of rows of page `page`, restricted to the page's bytes.
// The wavefronts of the workgroup form (kWaves / KS) row slots of RW rows;
// the KS wavefronts of a slot split K into KS contiguous column ranges
// (split-K inside the workgroup) and combine their partial sums through LDS
// in a fixed order.  The page's buffer resource covers exactly its valid
// bytes, so columns of a cut row that lie on the neighbouring page, and
// columns past K, read as zero without a branch.
//
// A row cut by a page boundary belongs to the earlier page's unit when both
// pages are in the same tier (it reads the next page too and adds the two
// parts itself); when the tiers differ each page's unit stores its part and
// split_fixup adds them, so no workgroup ever reads two tiers.
template <int B, int RW, int UN, int KS>
__device__ void gemv_unit(const GemvParams& P, int page, int j, float* lds) {
  constexpr int kSlots = kWaves / KS;
  constexpr int kRowsWg = kSlots * RW;
  const int64_t K = P.K;
  const int64_t total = static_cast<int64_t>(P.N) * K;
  const int64_t pe0 = static_cast<int64_t>(page) * kPageElems;
  const int64_t pe1 = min(pe0 + kPageElems, total);
  const int64_t r_lo = pe0 / K;
  const int64_t r_hi = (pe1 - 1) / K;  // inclusive
  const int64_t rbase = r_lo + static_cast<int64_t>(j) * kRowsWg;
  if (rbase > r_hi) return;  // uniform over the workgroup
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int slot = wave / KS, part = wave % KS;
  const int64_t r0 = rbase + slot * RW;
  // tiers are read only by the (few) units that hold a row cut by a page
  // boundary, so the common unit starts its loads without waiting on them
  const bool cut_first = rbase == r_lo && r_lo * K < pe0;
  const bool cut_last = rbase + kRowsWg > r_hi && (r_hi + 1) * K > pe1;
  bool prev_same = false, next_same = false;
  if (cut_first || cut_last) {
    const uint8_t tier = page_tier(P, page);
    prev_same = cut_first && page_tier(P, page - 1) == tier;
    next_same = cut_last && page + 1 < P.n_pages && page_tier(P, page + 1) == tier;
  }

  const __amdgpu_buffer_rsrc_t wr =
      make_rsrc(page_addr(P, page), static_cast<uint32_t>((pe1 - pe0) * 2));
  const __amdgpu_buffer_rsrc_t xr =
      make_rsrc(P.x, static_cast<uint32_t>(B * K * 2));
  // 0 = whole row here, 1 = tail of a row begun on the previous page,
  // 2 = head of a row ending on the next page, 3 = skipped
  int kind[RW];
  uint32_t ro[RW], ro2[RW];
  bool join = false;
#pragma unroll
  for (int i = 0; i < RW; ++i) {
    const int64_t r = r0 + i;
    const int64_t e0 = r * K;
    kind[i] = r > r_hi ? 3 : (e0 < pe0 ? (prev_same ? 3 : 1) : (e0 + K > pe1 ? 2 : 0));
    ro[i] = kind[i] == 3 ? kOOB : static_cast<uint32_t>((e0 - pe0) * 2);
    ro2[i] = kOOB;
    if (kind[i] == 2 && next_same) {
      ro2[i] = static_cast<uint32_t>((e0 - pe1) * 2);  // wraps: columns before pe1 read 0
      join = true;
    }
  }

  float acc[RW][B], acc2[RW][B];
#pragma unroll
  for (int i = 0; i < RW; ++i)
#pragma unroll
    for (int b = 0; b < B; ++b) acc[i][b] = acc2[i][b] = 0.f;

  constexpr int kStep = 64 * 8;
  // this wavefront's columns: [k_beg, k_end), k_beg a multiple of kStep
  const int64_t kper = (((K + KS - 1) / KS) + kStep - 1) / kStep * kStep;
  const int64_t k_beg = part * kper;
  const int64_t k_end = min(K, k_beg + kper);
  accumulate<B, RW, UN>(wr, xr, ro, K, k_beg, k_end, lane, acc);
  if (join) {  // uniform over the slot (same rows, same page): the next page's part
    const int64_t pe2 = min(pe1 + kPageElems, total);
    const __amdgpu_buffer_rsrc_t wr2 =
        make_rsrc(page_addr(P, page + 1), static_cast<uint32_t>((pe2 - pe1) * 2));
    accumulate<B, RW, UN>(wr2, xr, ro2, K, k_beg, k_end, lane, acc2);
  }

  float v[RW][B], v2[RW][B];
#pragma unroll
  for (int i = 0; i < RW; ++i)
#pragma unroll
    for (int b = 0; b < B; ++b) {
      v[i][b] = wave_sum(acc[i][b]);
      v2[i][b] = join ? wave_sum(acc2[i][b]) : 0.f;
    }

  if constexpr (KS > 1) {
    // partial sums of the KS column ranges meet in LDS; the slot's first
    // wavefront adds them in range order (each page part separately)
    float* l1 = lds;
    float* l2 = lds + kWaves * RW * B;
    if (lane == 0)
#pragma unroll
      for (int i = 0; i < RW; ++i)
#pragma unroll
        for (int b = 0; b < B; ++b) {
          l1[(wave * RW + i) * B + b] = v[i][b];
          l2[(wave * RW + i) * B + b] = v2[i][b];
        }
    __syncthreads();
    if (part == 0 && lane == 0)
#pragma unroll
      for (int i = 0; i < RW; ++i)
#pragma unroll
        for (int b = 0; b < B; ++b) {
          float s1 = l1[(wave * RW + i) * B + b], s2 = l2[(wave * RW + i) * B + b];
#pragma unroll
          for (int q = 1; q < KS; ++q) {
            s1 += l1[((wave + q) * RW + i) * B + b];
            s2 += l2[((wave + q) * RW + i) * B + b];
          }
          v[i][b] = s1;
          v2[i][b] = s2;
        }
    __syncthreads();  // LDS is reused by the next unit of a persistent worker
  }
  if (part != 0 || lane != 0) return;
#pragma unroll
  for (int i = 0; i < RW; ++i) {
    const int64_t r = r0 + i;
    if (kind[i] == 0) {
#pragma unroll
      for (int b = 0; b < B; ++b) store_y(P, b, r, v[i][b]);
    } else if (kind[i] == 1) {
      store_split<B>(P, page, 1, v[i]);  // tail of a row begun on a page of the other tier
    } else if (kind[i] == 2) {
      if (ro2[i] != kOOB) {
#pragma unroll
        for (int b = 0; b < B; ++b) store_y(P, b, r, v[i][b] + v2[i][b]);
      } else {
        store_split<B>(P, page + 1, 0, v[i]);  // head of a row ending on the other tier
      }
    }
  }
}

// Unit `idx` of a list of n pages (the HBM pages in page order, or with
// all_pages every page) with U units each.  Normally page idx / U, unit idx % U.  With tail_first the first n
// indices are the last non-empty unit of every page and the rest the other
// units in page order: the last unit of a page holds the row cut by the page
// boundary, which it sums over both pages when they are in one tier, so it
// reads twice as many steps as the others; dispatched first it overlaps
// them instead of running alone at the end of the launch.
template <int kRowsWg>
__device__ __forceinline__ void unit_of(const GemvParams& P, bool all_pages, int n, int U,
                                        int idx, int& page, int& j) {
  if (!P.tail_first) {
    page = all_pages ? idx / U : hbm_page(P, idx / U);
    j = idx % U;
    return;
  }
  const int i = idx < n ? idx : (idx - n) / (U - 1);
  page = all_pages ? i : hbm_page(P, i);
  const int64_t total = static_cast<int64_t>(P.N) * P.K;
  const int64_t pe0 = static_cast<int64_t>(page) * kPageElems;
  const int64_t pe1 = min(pe0 + kPageElems, total);
  const int last = static_cast<int>(((pe1 - 1) / P.K - pe0 / P.K) / kRowsWg);
  if (idx < n) {
    j = last;
  } else {
    const int k = (idx - n) % (U - 1);
    j = k < last ? k : k + 1;
  }
}

template <int B, int RW, int UN, int KS>
__global__ __launch_bounds__(kThreads) void gemv_kernel(GemvParams P) {
  __shared__ float lds[2 * kWaves * RW * B];
  constexpr int kRowsWg = (kWaves / KS) * RW;
  const int bid = blockIdx.x;
  const int U = P.units_per_page;
  int page, j;
  if (P.address_order) {
    unit_of<kRowsWg>(P, true, P.n_pages, U, bid, page, j);
    gemv_unit<B, RW, UN, KS>(P, page, j, lds);
  } else if (bid < P.host_workers) {
    const int n_host_units = P.n_host_pages * U;
    for (int v = bid; v < n_host_units; v += P.host_workers)
      gemv_unit<B, RW, UN, KS>(P, host_page(P, v / U), v % U, lds);
  } else {
    unit_of<kRowsWg>(P, false, P.n_hbm_pages, U, bid - P.host_workers, page, j);
    gemv_unit<B, RW, UN, KS>(P, page, j, lds);
  }
}

// y of every row cut by a page boundary: part on the earlier page plus part
// on the later page, in that order.  One lane per (boundary, batch row).
__global__ __launch_bounds__(256) void split_fixup(GemvParams P, int n_pages, int B) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  const int bnd = 1 + t / B, b = t % B;
  if (bnd >= n_pages) return;
  const int64_t e = static_cast<int64_t>(bnd) * kPageElems;
  if (e % P.K == 0) return;  // this boundary falls between rows
  if (P.join && page_tier(P, bnd - 1) == page_tier(P, bnd)) return;  // summed by one workgroup
  const float* s0 = P.partial + static_cast<int64_t>(bnd) * 2 * bst::kMaxGemvBatch;
  store_y(P, b, e / P.K, s0[b] + s0[bst::kMaxGemvBatch + b]);
}

// ---------------------------------------------------------------------------
// Skinny GEMM on the matrix cores for batches above the GEMV's range.
//
// Same page-confined units, schedules and split-row handling as the GEMV; the
// contraction runs on v_mfma_f32_16x16x32_bf16.  A unit is 16 * RT rows of
// one page and one slice of K; the four wavefronts of the workgroup split the
// slice into four contiguous column ranges.  Per 32-column step a wavefront
// holds, for each 16-row tile, one A fragment (lane l: row l % 16, columns
// 8 (l / 16) .. +8 of the step, 16 bytes) and, for each 16-wide batch tile,
// one B fragment of x with the same column mapping (lane l: batch row
// l % 16), and issues RT * BT MFMAs.  The column order inside a step is the
// instruction's, identical for both operands, so every product pairs
// W[n, k] with x[b, k].
//
// The four partial tiles meet in LDS in wavefront order (0, 1, 2, 3), so the
// reduction order is fixed.  Rows cut by a page boundary store their part in
// the split buffer and split_fixup adds the two parts; with K split over S
// workgroups every part goes to the context workspace and split_reduce adds
// the slices in order.  (Wavefronts that each own rows over the whole slice,
// sharing x through L1, measured 25-30 % slower: four times longer
// wavefronts and a quarter of the units.)
//
// Cache policy of the matrix-core path's weight loads: 0 = default.  A
// fragment covers 64 bytes of each of 16 rows, so the other half of every
// 128-byte line is read by the next column step; streaming (non-temporal)
// loads lose that half before it is used and fetch it from HBM again.
#ifndef BOOST_MFMA_W_AUX
#define BOOST_MFMA_W_AUX 0
#endif
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;

__device__ __forceinline__ bf16x8_t as_bf16x8(const uint4& v) {
  return __builtin_bit_cast(bf16x8_t, v);
}

// Weights through LDS (WL, one row tile per wavefront): each wavefront
// streams its 16 rows row-contiguously (one load instruction = 512 bytes of
// each of two rows), writes the 16 x 256 column chunk into a private LDS tile
// (16-byte chunks XOR-swizzled by row so both the writes and the fragment
// reads are free of bank conflicts) and reads the A fragments back from there.
constexpr int kWlCols = 256;                          // columns per chunk
constexpr int kWlTileFloats = 16 * kWlCols * 2 / 4;   // one wavefront's tile

template <int BT, int RT>
constexpr int mfma_lds_floats() { return 16 * BT * (16 * RT + 1); }

template <int BT, int RT, int UN, bool WL>
__device__ void mfma_unit(const GemvParams& P, int page, int unit, float* lds) {
  const int j = unit / P.S, slice = unit % P.S;
  constexpr int R = 16 * RT;  // rows of a unit
  constexpr int LS = R + 1;   // LDS stride between batch rows (floats)
  const int64_t K = P.K;
  const int64_t total = static_cast<int64_t>(P.N) * K;
  const int64_t pe0 = static_cast<int64_t>(page) * kPageElems;
  const int64_t pe1 = min(pe0 + kPageElems, total);
  const int64_t r_lo = pe0 / K;
  const int64_t r_hi = (pe1 - 1) / K;  // inclusive
  const int64_t rbase = r_lo + static_cast<int64_t>(j) * R;
  if (rbase > r_hi) return;  // uniform over the workgroup
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int lrow = lane & 15, lgrp = lane >> 4;

  const __amdgpu_buffer_rsrc_t wr =
      make_rsrc(page_addr(P, page), static_cast<uint32_t>((pe1 - pe0) * 2));
  const __amdgpu_buffer_rsrc_t xr =
      make_rsrc(P.x, static_cast<uint32_t>(static_cast<int64_t>(P.B) * K * 2));
  uint32_t xo[BT];
#pragma unroll
  for (int t = 0; t < BT; ++t) {
    const int b = 16 * t + lrow;
    xo[t] = b < P.B ? static_cast<uint32_t>(b * K * 2) : kOOB;
  }

  f32x4_t acc[RT][BT];
#pragma unroll
  for (int a = 0; a < RT; ++a)
#pragma unroll
    for (int t = 0; t < BT; ++t) acc[a][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  constexpr int kStep = 32;
  // this unit's K slice, then this wavefront's quarter of it
  const int64_t ksl = (K + P.S - 1) / P.S;
  const int64_t kslice = (ksl + kWaves * kStep - 1) / (kWaves * kStep) * (kWaves * kStep);
  const int64_t s_beg = slice * kslice;
  const int64_t s_end = min(K, s_beg + kslice);
  const int64_t kper = kslice / kWaves;
  const int64_t k_beg = min(s_end, s_beg + wave * kper);
  const int64_t k_end = min(s_end, k_beg + kper);

  if constexpr (WL) {
    static_assert(RT <= 2, "LDS-staged weights take one or two row tiles");
    constexpr int kLd = 8 * RT;  // load instructions per chunk (two rows each)
    uint4* tile = reinterpret_cast<uint4*>(lds + mfma_lds_floats<BT, RT>()) +
                  wave * (RT * kWlTileFloats / 4);
    // load instruction i: rows 2i and 2i+1 (lanes 0-31 / 32-63), 16 bytes
    // each; a row begun on the previous page gets a wrapped (huge) offset,
    // so its columns before the page read as zero
    uint32_t lo[kLd];
#pragma unroll
    for (int i = 0; i < kLd; ++i) {
      const int64_t r = rbase + 2 * i + (lane >> 5);
      lo[i] = r > r_hi ? kOOB : static_cast<uint32_t>((r * K - pe0) * 2);
    }
    const int wr_chunk = lane & 31;
    uint4 wv[kLd];
    auto load_chunk = [&](int64_t kb) {
      const int64_t kc = kb + 8 * wr_chunk;
      const uint32_t oob = kc < k_end ? 0u : kOOB;
      const uint32_t kc2 = static_cast<uint32_t>(kc * 2);
#pragma unroll
      for (int i = 0; i < kLd; ++i) wv[i] = load16<BOOST_MFMA_W_AUX>(wr, (lo[i] + kc2) | oob);
    };
    if (k_beg < k_end) load_chunk(k_beg);
    constexpr int kChunkSteps = kWlCols / kStep;
#pragma unroll 1
    for (int64_t kb = k_beg; kb < k_end; kb += kWlCols) {
#pragma unroll
      for (int i = 0; i < kLd; ++i) {
        const int rr = 2 * i + (lane >> 5);
        tile[rr * 32 + (wr_chunk ^ (rr & 15))] = wv[i];
      }
      // this chunk's x fragments, then the next chunk's weights: the MFMAs
      // below wait only for the former (the wait counter is in order)
      uint4 xv[kChunkSteps][BT];
#pragma unroll
      for (int st = 0; st < kChunkSteps; ++st) {
        const int64_t kc = kb + st * kStep + 8 * lgrp;
        const uint32_t oob = kc < k_end ? 0u : kOOB;
        const uint32_t kc2 = static_cast<uint32_t>(kc * 2);
#pragma unroll
        for (int t = 0; t < BT; ++t) xv[st][t] = load16(xr, (xo[t] + kc2) | oob);
      }
      load_chunk(kb + kWlCols);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int st = 0; st < kChunkSteps; ++st)
#pragma unroll
        for (int ra = 0; ra < RT; ++ra) {
          const uint4 a = tile[(16 * ra + lrow) * 32 + ((4 * st + lgrp) ^ lrow)];
#pragma unroll
          for (int t = 0; t < BT; ++t)
            acc[ra][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                as_bf16x8(a), as_bf16x8(xv[st][t]), acc[ra][t], 0, 0, 0);
        }
    }
  } else {
    // byte offset of column 0 of this lane's row in every row tile (wrapped
    // for a row begun on the previous page, as above)
    uint32_t ro[RT];
#pragma unroll
    for (int a = 0; a < RT; ++a) {
      const int64_t r = rbase + 16 * a + lrow;
      ro[a] = r > r_hi ? kOOB : static_cast<uint32_t>((r * K - pe0) * 2);
    }
    // Column groups (UN steps of 32) with their weight and x fragments are
    // loaded one group ahead: the group a step consumes is always the oldest
    // set of outstanding loads, so the in-order wait counter lets the next
    // group stay in flight while its MFMAs run.  Loads past k_end read zero.
    constexpr int64_t kGroup = kStep * UN;
    struct Group {
      uint4 w[UN][RT];
      uint4 x[UN][BT];
    };
    auto load_group = [&](int64_t kb, Group& g) {
#pragma unroll
      for (int u = 0; u < UN; ++u) {
        const int64_t kc = kb + u * kStep + 8 * lgrp;
        const uint32_t oob = kc < k_end ? 0u : kOOB;
        const uint32_t kc2 = static_cast<uint32_t>(kc * 2);
#pragma unroll
        for (int a = 0; a < RT; ++a)
          g.w[u][a] = load16<BOOST_MFMA_W_AUX>(wr, (ro[a] + kc2) | oob);
#pragma unroll
        for (int t = 0; t < BT; ++t) g.x[u][t] = load16(xr, (xo[t] + kc2) | oob);
      }
    };
    auto mma = [&](const Group& g) {
#pragma unroll
      for (int u = 0; u < UN; ++u)
#pragma unroll
        for (int t = 0; t < BT; ++t)
#pragma unroll
          for (int a = 0; a < RT; ++a)
            acc[a][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                as_bf16x8(g.w[u][a]), as_bf16x8(g.x[u][t]), acc[a][t], 0, 0, 0);
    };
    // fixed register roles (copying a group whose loads are outstanding
    // would wait for them); both halves always run, a group past k_end being
    // zeros, so the loop has one exit and the accumulators one register set
    Group ga, gb;
    if (k_beg < k_end) load_group(k_beg, ga);
#pragma unroll 1
    for (int64_t kb = k_beg; kb < k_end; kb += 2 * kGroup) {
      load_group(kb + kGroup, gb);
      __builtin_amdgcn_sched_barrier(0);  // keep the prefetch ahead of the MFMAs
      mma(ga);
      load_group(kb + 2 * kGroup, ga);
      __builtin_amdgcn_sched_barrier(0);
      mma(gb);
    }
  }

  // output element (row 16a + 4 lgrp + e, batch 16t + lrow) of every tile;
  // LDS holds the unit's [batch][row] tile, summed over wavefronts in order
#pragma unroll 1
  for (int w = 0; w < kWaves; ++w) {
    if (wave == w) {
#pragma unroll
      for (int a = 0; a < RT; ++a)
#pragma unroll
        for (int t = 0; t < BT; ++t)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            float* q = lds + (16 * t + lrow) * LS + 16 * a + 4 * lgrp + e;
            *q = w == 0 ? acc[a][t][e] : *q + acc[a][t][e];
          }
    }
    __syncthreads();
  }
  for (int idx = threadIdx.x; idx < R * 16 * BT; idx += kThreads) {
    const int b = idx / R, i = idx % R;
    const int64_t r = rbase + i;
    if (b >= P.B || r > r_hi) continue;
    const float v = lds[b * LS + i];
    const int64_t e0 = r * K;
    const int side = e0 < pe0 ? 1 : (e0 + K > pe1 ? 0 : -1);  // cut row: its part's side
    if (P.S == 1) {
      if (side == 1)
        P.partial[(static_cast<int64_t>(page) * 2 + 1) * bst::kMaxGemvBatch + b] = v;
      else if (side == 0)
        P.partial[(static_cast<int64_t>(page + 1) * 2) * bst::kMaxGemvBatch + b] = v;
      else
        store_y(P, b, r, v);
    } else if (side < 0) {
      P.ws[(static_cast<int64_t>(slice) * P.B + b) * P.N + r] = v;
    } else {
      const int64_t bnd = side ? page : page + 1;
      P.ws[static_cast<int64_t>(P.S) * P.B * P.N +
           ((bnd * 2 + side) * P.S + slice) * P.B + b] = v;
    }
  }
  __syncthreads();  // LDS is reused by the next unit of a persistent worker
}

template <int BT, int RT, int UN, bool WL>
__global__ __launch_bounds__(kThreads) void mfma_kernel(GemvParams P) {
  __shared__ float lds[mfma_lds_floats<BT, RT>() + (WL ? kWaves * RT * kWlTileFloats : 0)];
  const int bid = blockIdx.x;
  const int U = P.units_per_page;
  if (P.address_order) {
    mfma_unit<BT, RT, UN, WL>(P, bid / U, bid % U, lds);
  } else if (bid < P.host_workers) {
    const int n_host_units = P.n_host_pages * U;
    for (int v = bid; v < n_host_units; v += P.host_workers)
      mfma_unit<BT, RT, UN, WL>(P, host_page(P, v / U), v % U, lds);
  } else {
    const int u = bid - P.host_workers;
    mfma_unit<BT, RT, UN, WL>(P, hbm_page(P, u / U), u % U, lds);
  }
}

// ---------------------------------------------------------------------------
// Matrix-core GEMM for larger batches: W and x streamed into LDS by
// direct-to-LDS loads.
//
// The unit is 64 RT rows of one page and one slice of K.  K is walked in
// stages of 64 columns through a ring of dma_stages() stages in LDS, and
// every byte of a stage, W rows and x rows alike, goes from memory straight
// into LDS (buffer_load ... lds): no register holds data in flight, so all
// but one stage of the ring stay in flight per workgroup, and x crosses the
// L2 -> CU path once per workgroup.  Each wavefront reads its A fragments
// (lane l: row l % 16 of a 16-row tile, columns 8 (l / 16) .. + 8 of a
// 32-column step) and B fragments (the same mapping over batch rows) from
// LDS and ends with the full sums of its tiles over the slice, so there is
// no cross-wavefront reduction; rows cut by a page boundary and split-K
// slices go through the same partial buffers as the other matrix-core path.
// One such load instruction moves 1 KiB: lane i writes LDS
// bytes [16 i, 16 i + 16) of the block at M0, and a lane chooses which global
// 16 bytes it fetches, so an instruction reads 8 whole 128-byte rows of a
// stage and lays them out swizzled: row r (0..7) of block b keeps its
// 16-byte chunk c at position c ^ r ^ (b & 1), so the 16 rows of a fragment
// read at one chunk (rows 0..7 from an even block, 8..15 from the next) sit
// at 16 distinct 16-byte positions modulo 256 bytes.  The compiler does not
// see these loads (inline assembly: it would otherwise wait for all of them
// before any LDS read); the waits on them are explicit, in issue
// order: before stage s is read, each wavefront waits until only the later
// stages' loads are outstanding, then the workgroup barrier makes every
// wavefront's part of the stage visible and frees the slot read in the
// previous step, which the next loads overwrite.  Out-of-range lanes (rows
// past the page, columns outside the page or the slice, batch rows past B)
// write zeros into LDS, as out-of-range register loads return zeros.
constexpr int kDmaBlk = 1024;  // 8 rows x 128 bytes
constexpr int kDmaLds = 160000;  // LDS bytes a ring may take
// bytes of one stage: W rows, then x rows (stages of 128 columns, one
// barrier per 128 columns, were 2-7 % slower on the 8B shapes at batch
// 32..256)
template <int BT, int RT>
constexpr int dma_stage_bytes() { return (8 * RT + 2 * BT) * kDmaBlk; }
// as many stages as fit, up to BOOST_GEMM_DMA_NS (deeper rings, up to 16
// stages, were no faster on the 8B and 70B shapes)
#ifndef BOOST_GEMM_DMA_NS
#define BOOST_GEMM_DMA_NS 4
#endif
template <int BT, int RT>
constexpr int dma_stages() {
  return kDmaLds / dma_stage_bytes<BT, RT>() >= BOOST_GEMM_DMA_NS ? BOOST_GEMM_DMA_NS
                                                                  : kDmaLds / dma_stage_bytes<BT, RT>();
}

// Row groups of the 2-D arrangement of the NW wavefronts over a unit's
// 4 RT row tiles and BT batch tiles: the one that reads the fewest fragments
// per 32-column step (4 RT / WR + BT / (NW / WR)), ties to more row groups
template <int BT, int RT, int NW = 4>
constexpr int dma_wave_rows() {
  int best = -1, cost = 1 << 30;
  for (int wr = NW; wr >= 1; wr /= 2) {
    const int wb = NW / wr;
    if ((4 * RT) % wr || BT % wb) continue;
    const int c = 4 * RT / wr + BT / wb;
    if (c < cost) best = wr, cost = c;
  }
  return best;
}

using bst::load16_lds;
using bst::vmcnt_imm;

// HOST: the unit is one 16-row tile of a unit (sub-unit unit_in % (4 RT) of
// unit unit_in / (4 RT)), so a page read over the host link, whose loads wait
// far longer than HBM's, spreads over 4 RT times more workgroups; every
// output still sums the same columns in the same order, so the results do
// not depend on which pages are on the host.
template <int BT, int RT, bool HOST = false, int NW = 4>
__device__ __forceinline__ void gemm_dma_unit(const GemvParams& P, int page_in, int unit_in,
                                              char* ring) {
  static_assert((2 * BT) % NW == 0, "x blocks are spread evenly over the wavefronts");
  static_assert((8 * RT) % NW == 0, "W blocks are spread evenly over the wavefronts");
  constexpr int kNs = dma_stages<BT, RT>();
  constexpr int kSb = dma_stage_bytes<BT, RT>();
  constexpr int kXq = 2 * BT / NW;            // x blocks loaded per wavefront and stage
  constexpr int kWq = HOST ? 1 : 8 * RT / NW;  // W blocks loaded per wavefront and stage
  constexpr int kLoads = kWq + kXq;        // load instructions per wavefront and stage
  static_assert(kNs >= 2, "ring of at least two stages");
  const int page = __builtin_amdgcn_readfirstlane(page_in);
  const int uin = __builtin_amdgcn_readfirstlane(unit_in);
  const int unit = HOST ? uin / (4 * RT) : uin;
  const int j = unit / P.S, slice = unit % P.S;
  constexpr int R = 64 * RT;
  const int64_t K = P.K;
  const int64_t total = static_cast<int64_t>(P.N) * K;
  const int64_t pe0 = static_cast<int64_t>(page) * kPageElems;
  const int64_t pe1 = min(pe0 + kPageElems, total);
  const int64_t r_lo = pe0 / K;
  const int64_t r_hi = (pe1 - 1) / K;  // inclusive
  const int64_t rbase =
      r_lo + static_cast<int64_t>(j) * R + (HOST ? 16 * (uin % (4 * RT)) : 0);
  if (rbase > r_hi) return;  // uniform over the workgroup
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
  const int lane = threadIdx.x & 63;
  const int lrow = lane & 15, lgrp = lane >> 4;

  const __amdgpu_buffer_rsrc_t wr =
      make_rsrc_uniform(page_addr(P, page), static_cast<uint32_t>((pe1 - pe0) * 2));
  const __amdgpu_buffer_rsrc_t xr =
      make_rsrc_uniform(P.x, static_cast<uint32_t>(static_cast<int64_t>(P.B) * K * 2));

  const int64_t ksl = (K + P.S - 1) / P.S;
  const int64_t kslice = (ksl + 63) / 64 * 64;
  const int64_t k_beg = min(K, slice * kslice);
  const int64_t k_end = min(K, k_beg + kslice);
  const int nst = static_cast<int>((k_end - k_beg + 63) / 64);

  // loads: lane i of an instruction for block b fetches row i / 8 of the
  // block and the chunk it stores at position i % 8, i.e. chunk
  // (i % 8) ^ (i / 8) ^ (b & 1); W blocks 2 T + h (tile T, rows 8 h ..),
  // wavefront w loading blocks w kWq .. w kWq + kWq - 1; x blocks
  // 8 RT + NW q + wave (an even base: parity of wave).  A host sub-unit has
  // one tile: wavefronts 0 and 1 load its blocks 0 and 1, and the others
  // issue an out-of-range load into the unused block 2, so every wavefront
  // issues the same number of loads per stage.
  const int brow = lane >> 3;
  const int c0 = (lane & 7) ^ brow;  // chunk at parity 0; parity 1: c0 ^ 1
  uint32_t ro[kWq];
  int wblk[kWq], wpar[kWq];
#pragma unroll
  for (int i = 0; i < kWq; ++i) {
    const int blk = HOST ? min(wave, 2) : wave * kWq + i;
    const int h = HOST ? (wave & 1) : (blk & 1);
    const int64_t r = rbase + 8 * blk + brow;  // block blk holds rows 8 blk ..
    const bool live = !HOST || wave < 2;
    ro[i] = (!live || r > r_hi) ? kOOB
                                : static_cast<uint32_t>((r * K - pe0) * 2) + 16 * (c0 ^ h);
    wblk[i] = blk;
    wpar[i] = h;
  }
  const int cx = c0 ^ (wave & 1);
  uint32_t xo[kXq];
#pragma unroll
  for (int q = 0; q < kXq; ++q) {
    const int b = 8 * (wave + NW * q) + brow;
    xo[q] = b < P.B ? static_cast<uint32_t>(static_cast<int64_t>(b) * K * 2) + 16 * cx : kOOB;
  }
  auto issue = [&](int s, int slot) {  // stage s into ring slot `slot`
    const int64_t kb = 64 * static_cast<int64_t>(s);
    // a chunk at or past k_end (a multiple of 8) reads zeros
    const int64_t kc0 = k_beg + kb + 8 * c0, kc1 = k_beg + kb + 8 * (c0 ^ 1);
    const uint32_t oob0 = kc0 < k_end ? 0u : kOOB, oob1 = kc1 < k_end ? 0u : kOOB;
    const uint32_t oobx = (wave & 1) ? oob1 : oob0;
    const uint32_t kb2 = static_cast<uint32_t>((k_beg + kb) * 2);
    const char* st = ring + slot * kSb;
#pragma unroll
    for (int i = 0; i < kWq; ++i)
      load16_lds(wr, (ro[i] + kb2) | (wpar[i] ? oob1 : oob0), st + wblk[i] * kDmaBlk);
#pragma unroll
    for (int q = 0; q < kXq; ++q)
      load16_lds(xr, (xo[q] + kb2) | oobx, st + (8 * RT + wave + NW * q) * kDmaBlk);
  };

  // fragment reads: lane l takes row l % 16 of a tile (block 2 tile + h,
  // h = l % 16 / 8, block row l % 8) and 8 columns at chunk 4 sub + l / 16
  // of the stage, at position chunk ^ row ^ h
  const int r8 = lrow & 7, hb = lrow >> 3;
  const int fo = hb * kDmaBlk + r8 * 128;
  const int fx0 = ((lgrp ^ r8 ^ hb) << 4), fx1 = fx0 ^ 64;  // position, sub 0 / 1
  // products: the NW wavefronts form a WR x (NW / WR) grid over the unit's
  // 4 RT row tiles and BT batch tiles; wavefront w takes row tiles
  // [RW (w / WB), + RW) and batch tiles [BW (w % WB), + BW)
  // (a host sub-unit: one row tile, the batch tiles over min(NW, BT)
  // wavefronts; the others only load)
  constexpr int WR = HOST ? 1 : dma_wave_rows<BT, RT, NW>();
  static_assert(WR > 0, "no wavefront grid fits the unit");
  constexpr int WB = HOST ? (BT < NW ? BT : NW) : NW / WR;
  constexpr int RW = (HOST ? 1 : 4 * RT) / WR, BW = BT / WB;
  const int t_row = RW * (wave / WB), t_bat = BW * (wave % WB);
  const bool computes = !HOST || wave < WB;  // uniform over the wavefront
  const int wa = 2 * t_row * kDmaBlk + fo;
  const int xa = (8 * RT + 2 * t_bat) * kDmaBlk + fo;

  f32x4_t acc[RW][BW];
#pragma unroll
  for (int a = 0; a < RW; ++a)
#pragma unroll
    for (int t = 0; t < BW; ++t) acc[a][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  constexpr int TG = BW < 4 ? BW : 4;  // x fragments live at once
  auto mma = [&](const char* st) {
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {  // the stage's two 32-column steps
      const int fx = sub ? fx1 : fx0;
      uint4 wf[RW];
#pragma unroll
      for (int a = 0; a < RW; ++a)
        wf[a] = *reinterpret_cast<const uint4*>(st + wa + a * 2 * kDmaBlk + fx);
#pragma unroll
      for (int t0 = 0; t0 < BW; t0 += TG) {
        uint4 xf[TG];
#pragma unroll
        for (int u = 0; u < TG; ++u)
          xf[u] = *reinterpret_cast<const uint4*>(st + xa + (t0 + u) * 2 * kDmaBlk + fx);
#pragma unroll
        for (int u = 0; u < TG; ++u)
#pragma unroll
          for (int a = 0; a < RW; ++a)
            acc[a][t0 + u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                as_bf16x8(wf[a]), as_bf16x8(xf[u]), acc[a][t0 + u], 0, 0, 0);
      }
    }
  };

#pragma unroll
  for (int s = 0; s < kNs - 1; ++s) issue(s, s);  // stages past the slice: zeros
  int slot = 0, fill = kNs - 1;
#pragma unroll 1
  for (int s = 0; s < nst; ++s) {
    __builtin_amdgcn_s_waitcnt(vmcnt_imm<(kNs - 2) * kLoads>());  // stage s landed
    __syncthreads();  // ... for every wavefront; slot `fill` is no longer read
    issue(s + kNs - 1, fill);
    if (computes) mma(ring + slot * kSb);
    slot = slot + 1 == kNs ? 0 : slot + 1;
    fill = fill + 1 == kNs ? 0 : fill + 1;
  }
  __builtin_amdgcn_s_waitcnt(vmcnt_imm<0>());  // the loads issued past the slice
  __syncthreads();  // LDS is reused by the next unit of a persistent worker

  if (!computes) return;
#pragma unroll
  for (int a = 0; a < RW; ++a)
#pragma unroll
    for (int t = 0; t < BW; ++t) {
      const int b = 16 * (t_bat + t) + lrow;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t r = rbase + 16 * (t_row + a) + 4 * lgrp + e;
        if (b >= P.B || r > r_hi) continue;
        const float v = acc[a][t][e];
        const int64_t e0 = r * K;
        const int side = e0 < pe0 ? 1 : (e0 + K > pe1 ? 0 : -1);  // cut row: its part's side
        if (P.S == 1) {
          if (side == 1)
            P.partial[(static_cast<int64_t>(page) * 2 + 1) * bst::kMaxGemvBatch + b] = v;
          else if (side == 0)
            P.partial[(static_cast<int64_t>(page + 1) * 2) * bst::kMaxGemvBatch + b] = v;
          else
            store_y(P, b, r, v);
        } else if (side < 0) {
          P.ws[(static_cast<int64_t>(slice) * P.B + b) * P.N + r] = v;
        } else {
          const int64_t bnd = side ? page : page + 1;
          P.ws[static_cast<int64_t>(P.S) * P.B * P.N +
               ((bnd * 2 + side) * P.S + slice) * P.B + b] = v;
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
}

template <int BT, int RT, int NW>
__global__ __launch_bounds__(64 * NW) void gemm_dma_kernel(GemvParams P) {
  __shared__ __attribute__((aligned(16))) char ring[dma_stages<BT, RT>() * dma_stage_bytes<BT, RT>()];
  const int bid = blockIdx.x;
  const int U = P.units_per_page;
  if (P.address_order) {
    gemm_dma_unit<BT, RT, false, NW>(P, bid / U, bid % U, ring);
  } else if (bid < P.host_workers) {
    const int Uh = U * 4 * RT;  // 16-row sub-units per host page
    const int n_host_sub = P.n_host_pages * Uh;
    for (int v = bid; v < n_host_sub; v += P.host_workers)
      gemm_dma_unit<BT, RT, true, NW>(P, host_page(P, v / Uh), v % Uh, ring);
  } else {
    const int u = bid - P.host_workers;
    gemm_dma_unit<BT, RT, false, NW>(P, hbm_page(P, u / U), u % U, ring);
  }
}

// Wavefronts per workgroup of the direct-to-LDS GEMM: eight (two per SIMD,
// sharing the one ring of the workgroup) from BOOST_GEMM_NW8_BT batch tiles,
// and for 128-row units from BOOST_GEMM_NW8_RT2_BT.  At 16 batch tiles
// (B = 129..256) eight took the 8B matrices 3-12 % faster (B = 256: gate_up
// 110 -> 102 us, down 92 -> 81 us); at 4 and 8 tiles (B = 49..64, 113..128)
// they took the 128-row units 5-8 % faster (down 39 -> 37 us at B = 64;
// gate_up 69 -> 65 us, down 55 -> 50 us at B = 128) while the 64-row units
// of qkv and o were -10..+5 % (kept at four).
#ifndef BOOST_GEMM_NW8_BT
#define BOOST_GEMM_NW8_BT 16
#endif
#ifndef BOOST_GEMM_NW8_RT2_BT
#define BOOST_GEMM_NW8_RT2_BT 4
#endif

// y of a split-K call: the S slice partials of every (batch row, row) in
// slice order; a row cut by a page boundary adds its earlier page's slices,
// then its later page's.  One lane per (b, n).
__global__ __launch_bounds__(256) void split_reduce(GemvParams P) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= static_cast<int64_t>(P.B) * P.N) return;
  const int b = static_cast<int>(t / P.N);
  const int64_t r = t % P.N;
  const int64_t e0 = r * P.K;
  const int64_t p0 = e0 / kPageElems, p1 = (e0 + P.K - 1) / kPageElems;
  // all S loads go out together (a loop over a run-time S would wait for
  // each in turn), then the sums in slice order
  float v = 0.f;
  if (p0 == p1) {
    float part[kMaxSlices];
#pragma unroll
    for (int s = 0; s < kMaxSlices; ++s)
      part[s] = s < P.S ? P.ws[(static_cast<int64_t>(s) * P.B + b) * P.N + r] : 0.f;
#pragma unroll
    for (int s = 0; s < kMaxSlices; ++s)
      if (s < P.S) v += part[s];
  } else {
    const float* cut = P.ws + static_cast<int64_t>(P.S) * P.B * P.N;
    float part0[kMaxSlices], part1[kMaxSlices];
#pragma unroll
    for (int s = 0; s < kMaxSlices; ++s) {
      part0[s] = s < P.S ? cut[((p1 * 2 + 0) * P.S + s) * P.B + b] : 0.f;
      part1[s] = s < P.S ? cut[((p1 * 2 + 1) * P.S + s) * P.B + b] : 0.f;
    }
    float v1 = 0.f;
#pragma unroll
    for (int s = 0; s < kMaxSlices; ++s)
      if (s < P.S) {
        v += part0[s];
        v1 += part1[s];
      }
    v += v1;
  }
  store_y(P, b, r, v);
}

#ifndef BOOST_GEMV_UN1
#define BOOST_GEMV_UN1 8
#endif
// Rows per wavefront and loads in flight per row, by batch size.
// Rows per wavefront (an x chunk is reused for every row) and load steps in
// flight, by batch size: more rows per wavefront as the batch grows keeps the
// x loads per weight load, and the registers, bounded.
#ifndef BOOST_GEMV_RW_BIG
#define BOOST_GEMV_RW_BIG 4
#endif
#ifndef BOOST_GEMV_UN_BIG
#define BOOST_GEMV_UN_BIG 1
#endif
// Batch 1 with a row split over four wavefronts (rows longer than 12K
// columns): each wavefront's x slice differs from its neighbours', so x misses
// the L1 cache (counters: as many L2 requests for x as for the weights) and
// would be fetched from L2 once per row; two rows per wavefront reuse one x
// slice from registers (8B down projection 22.2 -> 21.2 us, 70B 44.0 ->
// 42.1 us; with a row over two wavefronts it did not pay), with eight load
// steps in flight per row (four: 21.8 us, eight: 21.4, sixteen: 30.4 at
// half the occupancy).
#ifndef BOOST_GEMV_RW1_LONG
#define BOOST_GEMV_RW1_LONG 2
#endif
#ifndef BOOST_GEMV_UN1_LONG
#define BOOST_GEMV_UN1_LONG 8
#endif
#ifndef BOOST_GEMV_RW1
#define BOOST_GEMV_RW1 1
#endif
template <int B, int KS>
struct Shape {
  static constexpr int RW = B == 1 ? (KS > 2 ? BOOST_GEMV_RW1_LONG : BOOST_GEMV_RW1)
                                   : (B == 2 ? 2 : (B <= 4 ? 4 : BOOST_GEMV_RW_BIG));
  static constexpr int UN = B == 1 ? (KS > 2 ? BOOST_GEMV_UN1_LONG : BOOST_GEMV_UN1)
                                   : (B <= 4 ? 2 : BOOST_GEMV_UN_BIG);
};

// Wavefronts per row (split-K inside the workgroup) for a row of K columns:
// enough that each wavefront reads a few KiB of a row, so long rows do not
// serialise many round trips in one wavefront.
#ifndef BOOST_GEMV_KS_MAX
#define BOOST_GEMV_KS_MAX 4
#endif
#ifndef BOOST_GEMV_KS2_ABOVE
#define BOOST_GEMV_KS2_ABOVE 6144
#endif
#ifndef BOOST_GEMV_KS4_ABOVE
#define BOOST_GEMV_KS4_ABOVE 12288
#endif
inline int k_splits(int K) {
  const int ks = K <= BOOST_GEMV_KS2_ABOVE ? 1 : (K <= BOOST_GEMV_KS4_ABOVE ? 2 : 4);
  return ks < BOOST_GEMV_KS_MAX ? ks : BOOST_GEMV_KS_MAX;
}

#ifndef BOOST_HOST_UNITS_PER_WORKER
#define BOOST_HOST_UNITS_PER_WORKER 16
#endif
// Host workers for host_units units on host pages: by default n_cu / 16.
// The matrix-core kernels, whose workgroups keep fewer bytes in flight, take
// one per BOOST_HOST_UNITS_PER_WORKER host units, up to n_cu / 8 (70B step at
// batch 8: 427.6 -> 419.2 ms).  The GEMV's workgroups already keep the link
// busy; more of them slowed the HBM units beside them (2 GiB tensor, 8 host
// pages: 360 -> 432 us).  Never more workers than host units.
int host_worker_count(const boost_ctx* ctx, int64_t host_units, bool matrix_core) {
  const int64_t h_lo = std::max(1, ctx->n_cu / 16);
  const int64_t h_hi = matrix_core ? std::max(1, ctx->n_cu / 8) : h_lo;
  const int64_t h_want = (host_units + BOOST_HOST_UNITS_PER_WORKER - 1) / BOOST_HOST_UNITS_PER_WORKER;
  const int64_t h = ctx->gemv_host_workers > 0 ? ctx->gemv_host_workers
                                               : std::min(h_hi, std::max(h_lo, h_want));
  return static_cast<int>(std::min(h, host_units));
}

// Units per page and grid size for units of rows_wg rows; fills in
// P.units_per_page, P.host_workers and P.address_order.  Returns -1 if the
// grid is too large.
int64_t plan_grid(GemvParams& P, int n_pages, int rows_wg, const boost_ctx* ctx,
                  bool matrix_core) {
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
    P.host_workers = host_worker_count(ctx, host_units, matrix_core);
    grid = P.host_workers + static_cast<int64_t>(P.n_hbm_pages) * P.units_per_page;
  }
  return grid > 0x7fffffff ? -1 : grid;
}

// Largest S (halving from `want`) whose partials ([S][B][N] plus the cut
// rows' parts) fit the context's workspace or the caller's slice buffer.
int fit_slices(const GemvParams& P, int n_pages, int want, const boost_ctx* ctx) {
  int S = want;
  const uint64_t per = static_cast<uint64_t>(P.B) * (P.N + 2ull * (n_pages + 1));
  const uint64_t cap = P.slices ? static_cast<uint64_t>(P.slice_floats) : ctx->gemm_ws_floats;
  while (S > 1 && S * per > cap) S /= 2;
  return S;
}

int launch_fixup(GemvParams& P, int n_pages, bool need_fixup, hipStream_t s) {
  if (need_fixup) {
    const int lanes = (n_pages - 1) * P.B;
    hipLaunchKernelGGL(split_fixup, dim3((lanes + 255) / 256), dim3(256), 0, s, P,
                       n_pages, P.B);
    BOOST_HIP(hipGetLastError());
  }
  return BOOST_OK;
}

#ifndef BOOST_GEMV_TAIL_FIRST
#define BOOST_GEMV_TAIL_FIRST 1
#endif
template <int B, int KS>
int launch(GemvParams& P, int n_pages, bool need_fixup, const boost_ctx* ctx, hipStream_t s) {
  constexpr int RW = Shape<B, KS>::RW, UN = Shape<B, KS>::UN;
  const int64_t grid = plan_grid(P, n_pages, RW * (kWaves / KS), ctx, false);
  if (grid < 0) return bst::fail(BOOST_EINVAL, "grid too large");
  // rows cut by page boundaries: their units go first (see unit_of)
  P.tail_first = kPageElems % P.K != 0 && P.units_per_page >= 2 ? BOOST_GEMV_TAIL_FIRST : 0;
  hipLaunchKernelGGL((gemv_kernel<B, RW, UN, KS>), dim3(static_cast<unsigned>(grid)),
                     dim3(kThreads), 0, s, P);
  BOOST_HIP(hipGetLastError());
  return launch_fixup(P, n_pages, need_fixup, s);
}

// Row tiles per unit and column steps in flight by batch tiles (16 rows of x
// each): more accumulators as the batch grows, fewer loads in flight.
// Matrix-core shapes by batch tiles (16 rows of x each), from a sweep over the
// 8B and 70B matrices at B = 16..256:
//   BT <= 2: weights staged through LDS (row-contiguous streaming beat the
//            A-fragment pattern by 10-25 %);
//   BT 3..8: four 16-row tiles per wavefront (each x fragment serves four
//            MFMAs) when that still gives about one workgroup per CU, else
//            two (the smaller matrices need the extra workgroups more);
//   BT > 8:  two row tiles (four would need 256 accumulators per lane).
// Split K over S workgroups when the row groups alone give fewer than two
// workgroups per CU (small matrices at large batch); each slice keeps at
// least 512 columns, and the partials must fit the context's workspace.
template <int BT, int RT, int UN, bool WL>
int launch_mfma_shape(GemvParams& P, int n_pages, bool need_fixup, const boost_ctx* ctx,
                      hipStream_t s) {
  P.S = 1;
  int64_t grid = plan_grid(P, n_pages, 16 * RT, ctx, true);
  if (grid < 0) return bst::fail(BOOST_EINVAL, "grid too large");
  const int64_t units = static_cast<int64_t>(n_pages) * P.units_per_page;
  int S = 1;
  while (S < kMaxSlices && units * S < 2 * ctx->n_cu && P.K / (2 * S) >= 512) S *= 2;
  S = fit_slices(P, n_pages, S, ctx);
  if (S > 1) {
    P.S = S;
    P.ws = P.slices ? P.slices : ctx->gemm_ws;
    P.units_per_page *= S;
    grid = P.address_order ? static_cast<int64_t>(n_pages) * P.units_per_page
                           : P.host_workers + static_cast<int64_t>(P.n_hbm_pages) *
                                                  P.units_per_page;
  }
  hipLaunchKernelGGL((mfma_kernel<BT, RT, UN, WL>), dim3(static_cast<unsigned>(grid)),
                     dim3(kThreads), 0, s, P);
  BOOST_HIP(hipGetLastError());
  if (S == 1) return launch_fixup(P, n_pages, need_fixup, s);
  if (P.slices) return BOOST_OK;  // the consumer sums the slices
  const int64_t lanes = static_cast<int64_t>(P.B) * P.N;
  hipLaunchKernelGGL(split_reduce, dim3(static_cast<unsigned>((lanes + 255) / 256)), dim3(256),
                     0, s, P);
  BOOST_HIP(hipGetLastError());
  return BOOST_OK;
}

// Matrix-core shapes by batch tiles (16 rows of x each), from a sweep over the
// 8B and 70B matrices at B = 16..256:
//   BT <= 2: weights staged through LDS (row-contiguous streaming beat the
//            A-fragment pattern by 10-25 %);
//   BT 3..8: four 16-row tiles per wavefront (each x fragment serves four
//            MFMAs) when that still gives about one workgroup per CU, else
//            two (the smaller matrices need the extra workgroups more);
//   BT > 8:  two row tiles (four would need 256 accumulators per lane).
// The direct-to-LDS GEMM: units of 64 RT rows (RT = 2 where a page holds at
// least 128 rows, else 1), split-K over workgroups as above.
// Workgroups per four CUs that split-K aims for
#ifndef BOOST_GEMM_WG_X4
#define BOOST_GEMM_WG_X4 3
#endif
template <int BT, int RT>
int launch_gemm_shape(GemvParams& P, int n_pages, bool need_fixup, const boost_ctx* ctx,
                      hipStream_t s) {
  P.S = 1;
  int64_t grid = plan_grid(P, n_pages, 64 * RT, ctx, true);
  if (grid < 0) return bst::fail(BOOST_EINVAL, "grid too large");
  const int64_t units = static_cast<int64_t>(n_pages) * P.units_per_page;
  // split K over S workgroups until there are about three workgroups per
  // four CUs, and while a slice is longer than 16K columns (from a sweep of
  // RT and S over the 8B and 70B matrices at batch 32..256: fewer, fuller
  // workgroups beat more split-K, whose fp32 partials are extra traffic)
  int S = 1;
  while (S < kMaxSlices && P.K / (2 * S) >= 512 &&
         (units * S < ctx->n_cu * BOOST_GEMM_WG_X4 / 4 || P.K / S > 16384))
    S *= 2;
  S = fit_slices(P, n_pages, S, ctx);
  if (S > 1) {
    P.S = S;
    P.ws = P.slices ? P.slices : ctx->gemm_ws;
    P.units_per_page *= S;
  }
  if (P.address_order) {
    grid = static_cast<int64_t>(n_pages) * P.units_per_page;
  } else {
    // host pages run as 16-row sub-units (4 RT per unit)
    const int64_t host_sub = static_cast<int64_t>(P.n_host_pages) * P.units_per_page * 4 * RT;
    P.host_workers = host_worker_count(ctx, host_sub, true);
    grid = P.host_workers + static_cast<int64_t>(P.n_hbm_pages) * P.units_per_page;
  }
  if (grid > 0x7fffffff) return bst::fail(BOOST_EINVAL, "grid too large");
  if constexpr ((BT >= BOOST_GEMM_NW8_BT || (BT >= BOOST_GEMM_NW8_RT2_BT && RT == 2)) && BT % 4 == 0)
    hipLaunchKernelGGL((gemm_dma_kernel<BT, RT, 8>), dim3(static_cast<unsigned>(grid)),
                       dim3(8 * 64), 0, s, P);
  else
    hipLaunchKernelGGL((gemm_dma_kernel<BT, RT, 4>), dim3(static_cast<unsigned>(grid)),
                       dim3(kThreads), 0, s, P);
  BOOST_HIP(hipGetLastError());
  if (S == 1) return launch_fixup(P, n_pages, need_fixup, s);
  if (P.slices) return BOOST_OK;  // the consumer sums the slices
  const int64_t lanes = static_cast<int64_t>(P.B) * P.N;
  hipLaunchKernelGGL(split_reduce, dim3(static_cast<unsigned>((lanes + 255) / 256)), dim3(256),
                     0, s, P);
  BOOST_HIP(hipGetLastError());
  return BOOST_OK;
}

template <int BT>
int launch_gemm(GemvParams& P, int n_pages, bool need_fixup, const boost_ctx* ctx,
                hipStream_t s) {
  // 128-row units where a page fills them and they still give a workgroup
  // per CU (three per four CUs above four batch tiles, where halving x's
  // share of the ring counts for more: 8B gate_up's 224 units take 64-row
  // units at B = 64, 58.2 against 61.3 us, but keep 128-row units at B = 128
  // and 256, 70.5 and 92.9 against 83.4 and 119.0), or where a page holds
  // 64..127 rows (one unit per page either way); 64-row units otherwise.
  const int64_t rpp = kPageElems / P.K;  // whole rows per page
  // rows a page meets at most: one more than it holds whole when rows
  // straddle page boundaries
  const int64_t meet = std::min<int64_t>(P.N, rpp + (kPageElems % P.K != 0));
  const int64_t u2 = static_cast<int64_t>(n_pages) * ((meet + 127) / 128);
  const int64_t enough = BT > 4 ? ctx->n_cu * 3 / 4 : ctx->n_cu;
  if ((rpp >= 128 && u2 >= enough) || (rpp >= 64 && rpp < 128))
    return launch_gemm_shape<BT, 2>(P, n_pages, need_fixup, ctx, s);
  return launch_gemm_shape<BT, 1>(P, n_pages, need_fixup, ctx, s);
}

// Smallest batch-tile count that takes the direct-to-LDS GEMM
#ifndef BOOST_GEMM_MIN_BT
#define BOOST_GEMM_MIN_BT 2
#endif

template <int BT>
int launch_mfma(GemvParams& P, int n_pages, bool need_fixup, const boost_ctx* ctx,
                hipStream_t s) {
  if constexpr (BT >= BOOST_GEMM_MIN_BT) {
    return launch_gemm<BT>(P, n_pages, need_fixup, ctx, s);
  } else if constexpr (BT <= 2) {
    // two row tiles share each x fragment above 8 batch rows on matrices of
    // at least 2^25 elements (8B at B = 12..16: gate_up 54.5 -> 50.4 us,
    // down 42.0 -> 36.6 us); smaller matrices need the workgroups of one
    // (qkv, o: 19-27 % slower with two), and at B = 7..8 the two are even
    if (P.B > 8 && static_cast<int64_t>(P.N) * P.K >= (int64_t{1} << 25))
      return launch_mfma_shape<BT, 2, 1, true>(P, n_pages, need_fixup, ctx, s);
    return launch_mfma_shape<BT, 1, 1, true>(P, n_pages, need_fixup, ctx, s);
  } else if constexpr (BT <= 8) {
    // workgroups with 64-row units: pages x units per page (a page meets at
    // most kPageElems / K + 1 rows)
    const int64_t per_page = std::min<int64_t>(P.N, kPageElems / P.K + 1);
    if (static_cast<int64_t>(n_pages) * ((per_page + 63) / 64) >= ctx->n_cu * 3 / 4)
      return launch_mfma_shape<BT, 4, 1, false>(P, n_pages, need_fixup, ctx, s);
    return launch_mfma_shape<BT, 2, 2, false>(P, n_pages, need_fixup, ctx, s);
  } else {
    return launch_mfma_shape<BT, 2, 1, false>(P, n_pages, need_fixup, ctx, s);
  }
}

// Smallest batch that runs on the matrix cores (smaller ones use the GEMV):
// from batch 7 the one-tile matrix-core unit beats the dot2 GEMV on every
// 8B and 70B matrix; at 5 and 6 it depends on the shape.
#ifndef BOOST_MFMA_MIN_B
#define BOOST_MFMA_MIN_B 7
#endif
constexpr int kMfmaMinBatch = BOOST_MFMA_MIN_B;

template <int B>
int launch_b(GemvParams& P, int n_pages, bool need_fixup, const boost_ctx* ctx,
             hipStream_t s) {
  switch (k_splits(P.K)) {
    case 1: return launch<B, 1>(P, n_pages, need_fixup, ctx, s);
    case 2: return launch<B, 2>(P, n_pages, need_fixup, ctx, s);
    default: return launch<B, 4>(P, n_pages, need_fixup, ctx, s);
  }
}

}  // namespace

using namespace bst;

namespace {

int dispatch(GemvParams& P, const boost_tensor* W, int K, int B, const boost_ctx* ctx,
             hipStream_t s);

// The decode GEMV behind both entry points: y, or with `slices` the split-K
// partial sums in fp32 in the layout of ws (S reported through n_slices).
int decode_gemv(boost_ctx* ctx, const boost_tensor* W, int N, int K, const void* x, int B,
                void* y, int y_dtype, float* slices, int64_t slice_floats, int* n_slices,
                void* stream) {
  if (!ctx || !W || !x || !y) return fail(BOOST_EINVAL, "null argument");
  if (ctx->device < 0) return fail(BOOST_ENODEV, "plan-only context");
  if (N < 1 || K < 8 || K % 8) return fail(BOOST_EINVAL, "N=%d K=%d (K %% 8 == 0)", N, K);
  if (static_cast<uint64_t>(K) * 2 > kPage)
    return fail(BOOST_EINVAL, "row of %d elements exceeds a page", K);
  if (B < 1 || B > kMaxGemvBatch)
    return fail(BOOST_EINVAL, "B=%d outside [1, %d]", B, kMaxGemvBatch);
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
  P.hbm_base = W->hbm.base;
  P.host_base = W->host.base;
  P.lay_M = W->lay_M;
  P.lay_SP = W->lay_SP;
  P.n_hbm_pages = static_cast<int>(W->hbm_pages.size());
  P.n_host_pages = static_cast<int>(W->host_pages.size());
  P.address_order = ctx->gemv_schedule == BOOST_SCHED_ADDRESS;
  P.N = N;
  P.K = K;
  P.x = static_cast<const uint16_t*>(x);
  P.y = y;
  P.y_bf16 = y_dtype == BOOST_DTYPE_BF16;
  P.partial = W->d_partial;
  P.slices = slices;
  P.slice_floats = slice_floats;
  P.B = B;
  const int r = dispatch(P, W, K, B, ctx, static_cast<hipStream_t>(stream));
  if (r == BOOST_OK && n_slices) *n_slices = std::max(1, P.S);
  return r;
}

int dispatch(GemvParams& P, const boost_tensor* W, int K, int B, const boost_ctx* ctx,
             hipStream_t s) {
  const int n = static_cast<int>(W->n_pages);
  P.n_pages = n;
  P.tiers = W->d_tiers;
  if (B >= kMfmaMinBatch) {
    // every row cut by a page boundary goes through split_fixup
    P.join = 0;
    bool fix = false;
    for (int b = 1; b < n && !fix; ++b) fix = (static_cast<int64_t>(b) * kPageElems) % K != 0;
    switch ((B + 15) / 16) {
      case 1: return launch_mfma<1>(P, n, fix, ctx, s);
      case 2: return launch_mfma<2>(P, n, fix, ctx, s);
      case 3:
      case 4: return launch_mfma<4>(P, n, fix, ctx, s);
      case 5:
      case 6:
      case 7:
      case 8: return launch_mfma<8>(P, n, fix, ctx, s);
      default: return launch_mfma<16>(P, n, fix, ctx, s);
    }
  }
  // split_fixup is needed only where a cut row crosses a tier boundary
  P.join = 1;
  bool fix = false;
  if (kPageElems % K != 0)
    for (int b = 1; b < n && !fix; ++b)
      fix = (static_cast<int64_t>(b) * kPageElems) % K != 0 && W->tiers[b - 1] != W->tiers[b];
  switch (B) {
    case 1: return launch_b<1>(P, n, fix, ctx, s);
    case 2: return launch_b<2>(P, n, fix, ctx, s);
    case 3: return launch_b<3>(P, n, fix, ctx, s);
    case 4: return launch_b<4>(P, n, fix, ctx, s);
    case 5: return launch_b<5>(P, n, fix, ctx, s);
    case 6: return launch_b<6>(P, n, fix, ctx, s);
    case 7: return launch_b<7>(P, n, fix, ctx, s);
    default: return launch_b<8>(P, n, fix, ctx, s);
  }
}

}  // namespace

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
  return decode_gemv(ctx, W, N, K, x, B, y, y_dtype, nullptr, 0, nullptr, stream);
}

int boost_gemv_slices_floats(int N, int K, int B, int max_slices, uint64_t* floats) {
  if (!floats) return fail(BOOST_EINVAL, "null argument");
  if (N < 1 || K < 1 || B < 1 || max_slices < 1)
    return fail(BOOST_EINVAL, "N=%d K=%d B=%d max_slices=%d", N, K, B, max_slices);
  const uint64_t pages = (static_cast<uint64_t>(N) * K + kPageElems - 1) / kPageElems;
  *floats = static_cast<uint64_t>(max_slices) * B * (N + 2 * (pages + 1));
  return BOOST_OK;
}

int boost_decode_gemv_slices(boost_ctx* ctx, const boost_tensor* W, int N, int K,
                             const void* x, int B, float* slices, int max_slices,
                             int* n_slices, void* stream) {
  if (!slices || !n_slices) return fail(BOOST_EINVAL, "null argument");
  if (max_slices < 1 || max_slices > BOOST_MAX_GEMV_SLICES)
    return fail(BOOST_EINVAL, "max_slices %d outside [1, %d]", max_slices, BOOST_MAX_GEMV_SLICES);
  if (reinterpret_cast<uintptr_t>(slices) & 15)
    return fail(BOOST_EINVAL, "slices must be 16-byte aligned");
  uint64_t cap = 0;
  if (int rc = boost_gemv_slices_floats(N, K, B, max_slices, &cap)) return rc;
  *n_slices = 0;
  return decode_gemv(ctx, W, N, K, x, B, slices, BOOST_DTYPE_F32, slices,
                     static_cast<int64_t>(cap), n_slices, stream);
}

}  // extern "C"
