/*
 * boost_cap.h -- C-ABI of the tiered-memory (HBM + pinned host) decode path.
 *
 * Method: BOOST, "Concurrent Access to Host Memory and HBM to Accelerate LLM
 * Inference".  Weights are placed page by page on two tiers by modulo page
 * placement (MPP); the KV pool is split linearly between the tiers with KV
 * heads outermost and handed out by a wave-aware allocator (DSR); hand-written
 * CDNA4 kernels read every operand through a device page table so that each
 * workgroup streams from exactly one tier.
 *
 * Conventions
 *   - Every call returns 0 (BOOST_OK) or a negative BOOST_E* code; nothing
 *     throws across the ABI.  boost_last_error() gives a message for the last
 *     failing call of the calling thread.
 *   - A "page" is 2 MiB (BOOST_PAGE_BYTES), the GPU page size the paper places
 *     (§1, §4.4).  Tier codes: BOOST_TIER_HBM = 0, BOOST_TIER_HOST = 1.
 *   - Device pointers are plain addresses in the current HIP device's address
 *     space; `stream` is a hipStream_t passed as void* (NULL = default stream).
 *   - The library owns placed tensors, KV pools and their page tables and
 *     frees them in *_free / *_destroy.  The caller owns activations, queries,
 *     outputs, block tables, context lengths and streams.
 *   - Decode calls (boost_decode_gemv, boost_kv_write, boost_paged_attn_decode)
 *     are asynchronous on `stream`, never synchronise and never allocate; the
 *     first call on a tensor or pool may be made inside HIP graph capture.
 *     Two decode calls that use the same tensor or pool must be ordered on one
 *     stream (they share the tensor's split-row scratch).
 *   - Allocator calls (boost_kv_alloc / boost_kv_free) are CPU-only
 *     bookkeeping and are not thread-safe: one scheduler thread per pool.
 */
#ifndef BOOST_CAP_H
#define BOOST_CAP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define BOOST_OK 0
#define BOOST_EINVAL (-22) /* bad argument (null, zero size, shape, range)    */
#define BOOST_ENOMEM (-12) /* allocation or HBM budget failure                */
#define BOOST_EAGAIN (-11) /* KV pool cannot serve the request now (§4.3)     */
#define BOOST_ENODEV (-19) /* call needs a device but the context is plan-only */
#define BOOST_EHIP (-5)    /* a HIP runtime call failed                       */

#define BOOST_TIER_HBM 0
#define BOOST_TIER_HOST 1

#define BOOST_DTYPE_F32 0
#define BOOST_DTYPE_BF16 1

/* Placement kinds of boost_plan_contrast */
#define BOOST_PLACE_MPP 0        /* modulo placement, restarted per tensor  */
#define BOOST_PLACE_MPP_GLOBAL 1 /* modulo pattern continued across tensors */
#define BOOST_PLACE_LINEAR 2     /* first pages HBM, last floor(n/M) host   */
#define BOOST_PLACE_RANDOM 3     /* BAPP-R: each page host w.p. 1/M         */

#define BOOST_PAGE_BYTES (2ull * 1024ull * 1024ull)

typedef struct boost_ctx boost_ctx;
typedef struct boost_tensor boost_tensor;
typedef struct boost_kv_pool boost_kv_pool;

/* Message of the calling thread's last failing call ("" if none). */
const char *boost_last_error(void);

/* ABI version (major * 100 + minor). */
int boost_version(void);

/* ------------------------------------------------------------------ context */

/* Open a context on HIP device `device` (>= 0), or a plan-only context with
 * device = -1: plan-only contexts serve the placement planner and the KV
 * allocator bookkeeping and return BOOST_ENODEV from every call that touches
 * a GPU.  *out is owned by the caller and released with boost_shutdown.
 * Errors: EINVAL (null out, bad device), EHIP. */
int boost_init(int device, boost_ctx **out);
int boost_shutdown(boost_ctx *ctx);

/* Device facts: compute units and HIP device id (-1 when plan-only). */
int boost_ctx_info(const boost_ctx *ctx, int *device, int *n_cu);

/* Host backing of host-tier pages: 1 = coherent (fine-grained, uncached on
 * the GPU; default), 0 = non-coherent.  Affects pages placed afterwards. */
int boost_set_host_coherent(boost_ctx *ctx, int coherent);

/* NUMA node of host-tier pages (§4.4 binds every 2 MB host region to a
 * chosen node).  BOOST_NUMA_DEVICE (default): HIP's choice, the node nearest
 * the GPU; node >= 0: pages placed afterwards (weights, KV pool, calibration
 * buffers) are pinned while the calling thread's memory policy binds them to
 * that node, and the thread's previous policy is put back after each
 * allocation.  Errors: EINVAL (null ctx, node not online; a refused policy
 * call surfaces as EINVAL from the allocating call). */
#define BOOST_NUMA_DEVICE (-1)
int boost_set_host_numa(boost_ctx *ctx, int node);

/* Host NUMA facts (any output may be NULL): the NUMA node of the context's
 * GPU (-1 when the platform reports none or the context is plan-only), the
 * number of online nodes, and the node set by boost_set_host_numa. */
int boost_host_numa_info(const boost_ctx *ctx, int *device_node, int *n_nodes,
                         int *node);

/* ------------------------------------------------------- a0: calibration */

/* Measure alpha (§2.3: host read bandwidth over HBM read bandwidth; the paper
 * measures each tier's peak separately, §5.1).  One streaming-read kernel
 * reads a device buffer of `hbm_bytes` and a pinned, device-mapped host buffer
 * of `host_bytes` (both allocated and freed inside the call, so this call
 * synchronises and must not be captured), `iters` timed passes each after one
 * warm-up pass; the best of a small sweep is kept for each tier (HBM: static
 * slices over 4..32 workgroups per compute unit, and persistent workers, one
 * per compute unit, dealt 256 KiB chunks round robin, swept before and after
 * the host tier; host: 16..1024 workgroups).
 * Outputs (any may be NULL): GB/s (1e9 B/s) of each tier and alpha.
 * Errors: EINVAL (sizes < 64 MiB, iters < 1), ENODEV, ENOMEM, EHIP. */
int boost_calibrate(boost_ctx *ctx, uint64_t hbm_bytes, uint64_t host_bytes,
                    int iters, double *hbm_gbps, double *host_gbps,
                    double *alpha);

/* Read bandwidth (GB/s) of one streaming pass over `bytes` at device address
 * `src` with `grid` workgroups of 256 lanes, timed over `iters` passes on the
 * default stream (synchronises).  Used by calibration and tier probes.
 * Errors: EINVAL (null, bytes not a multiple of 4 KiB, grid < 1), ENODEV, EHIP. */
int boost_stream_read_gbps(boost_ctx *ctx, const void *src, uint64_t bytes,
                           int grid, int iters, double *gbps);

/* One point of the concurrent two-tier streaming probe. */
typedef struct boost_cap_point {
  uint64_t hbm_bytes;   /* bytes read from the HBM buffer */
  uint64_t host_bytes;  /* bytes read from the host buffer */
  int32_t hbm_wgs;      /* workgroups that stream the HBM bytes */
  int32_t host_wgs;     /* workgroups that stream the host bytes (0 for DMA) */
  int32_t host_stride;  /* host workgroups are 0, s, 2s, ...: 1 spreads them over
                           the XCDs, 8 puts them on one XCD */
  int32_t host_depth;   /* 16-byte loads per lane in flight on host: 1, 2, 4, 8 */
  int32_t host_policy;  /* host-load cache policy: 0 non-temporal (the kernels'),
                           1 default, 2 system-coherent */
  int32_t dma;          /* 1: the host bytes move by a host -> HBM copy on a
                           second stream, started with the HBM-only launch */
  int32_t hbm_chunk_kib;  /* 0: each HBM workgroup streams one contiguous slice;
                           > 0 (a multiple of 4): the HBM workgroups are
                           persistent and take chunks of this many KiB from a
                           queue (an atomic counter) until none is left */
  int32_t chunk_static; /* with hbm_chunk_kib > 0: 0 every chunk from the
                           queue; 1 the chunks dealt to the persistent workers
                           round robin, no queue; 2 each worker's first chunk
                           is its own index, the rest from the queue; 3 as 1,
                           with every workgroup holding 96 KiB of LDS so that
                           no two share a compute unit (host depth 8,
                           non-temporal host loads, no DMA) */
} boost_cap_point;

/* Concurrent two-tier streaming probe (the bound §3 "CAP" measures with a
 * streaming kernel whose workgroups read the host tier and HBM at once, swept
 * over the host share; §6.1 notes that the compute units must be able to keep
 * both tiers busy together).  Allocates an HBM buffer of hbm_bytes and a
 * pinned, device-mapped host buffer of host_bytes (coherent or not as set by
 * boost_set_host_coherent; plus an HBM staging buffer of host_bytes when a
 * point uses DMA), then for each of n_points points launches one kernel of
 * host_wgs + hbm_wgs workgroups, `iters` timed launches after one warm-up.
 * Static slices start on 1 KiB boundaries (the last ones shorter or empty).
 * Host workgroups stream host_bytes of the host buffer (contiguous slices,
 * the point's depth and cache policy), the others hbm_bytes of the HBM buffer
 * (16-byte non-temporal loads, 8 per lane in flight, contiguous slices).
 * results[16 i .. 16 i + 15] receive, each the median over the `iters` launches:
 *   0: GB/s of both tiers' bytes per launch (events; for DMA points over the
 *      longer of the launch and the copy),
 *   1: microseconds per launch (events),
 *   2: HBM tier GB/s inside the launch: hbm_bytes / (last HBM workgroup's end -
 *      the launch's first workgroup start), from each workgroup's clock,
 *   3: host tier GB/s: inside the launch the same way, or bytes over the
 *      copy's event time for DMA points (0 when unused),
 *   4: microseconds from the first workgroup start to the last end,
 *   5: microseconds from the first start to the median HBM workgroup's end,
 *   6: microseconds of the copy (DMA points), else 0,
 *   7: microseconds from the first start to the last HBM workgroup's end,
 *   8 + x: the same for the HBM workgroups that ran on XCD x (hardware
 *      register XCC_ID), x = 0..7 (0 when none ran there).
 * Synchronises; allocates and frees its buffers (load-time tool).
 * Errors: EINVAL (null, sizes beyond the buffers, bytes not a multiple of 16,
 * bytes without workgroups, a slice over 2 GiB, a stride outside [1, 64] or
 * whose host workgroups fall past the grid, a depth or policy out of range, a
 * DMA point with host workgroups, a chunk size out of range), ENODEV, ENOMEM,
 * EHIP. */
int boost_cap_sweep(boost_ctx *ctx, uint64_t hbm_bytes, uint64_t host_bytes,
                    int n_points, const boost_cap_point *points, int iters,
                    double *results);

/* C1: modulus M = K + 1 with K = ceil(1/alpha) (§3.1 modulo placement, §4.4
 * ceil rule keeping the host share at or below alpha).  alpha in (0, 1].
 * Errors: EINVAL. */
int boost_modulus_from_alpha(double alpha, uint32_t *M);

/* ----------------------------------------------------- a1: weight placement */

/* Superpage size in pages, lcm(footprint, page) / page (§3.2, §4.4); 1 when
 * footprint is 0. Errors: EINVAL (null). */
int boost_superpage_pages(uint64_t footprint_bytes, uint32_t *S);

/* C2: modulo page placement of one tensor of `bytes` bytes (§3.1, §4.4):
 * n = ceil(bytes / 2 MiB) pages; superpage j = pages [jS, (j+1)S); superpage j
 * is on host iff j mod M == M - 1.  The phase restarts for every tensor
 * (§3.1), so a tensor with fewer than M superpages has no host page.
 * Writes min(n, tier_cap) tier codes to tier_out (may be NULL) and n to
 * *n_pages.  Pure CPU.  Errors: EINVAL (bytes 0, M < 2, null n_pages). */
int boost_plan_mpp(uint64_t bytes, uint32_t M, uint64_t footprint_bytes,
                   uint8_t *tier_out, uint64_t tier_cap, uint64_t *n_pages);

/* Contrast placements of one tensor for the comparisons the paper draws
 * against modulo placement (§2.6 bandwidth-aware random placement BAPP-R and
 * Linux weighted interleaving, §5.6, §5.7 proportional interleave).  n =
 * ceil(bytes / 2 MiB) pages; page i is on host iff
 *   BOOST_PLACE_MPP         i mod M == M - 1 (same map as boost_plan_mpp, S=1);
 *   BOOST_PLACE_MPP_GLOBAL  (phase + i) mod M == M - 1, where phase is the
 *                           number of pages of the tensors placed before this
 *                           one: the modulo pattern is not restarted per tensor
 *                           (an interleave blind to kernel boundaries, §2.6);
 *   BOOST_PLACE_LINEAR      i >= n - floor(n / M) (the linear split of §4.2
 *                           applied to a weight tensor);
 *   BOOST_PLACE_RANDOM      uniforms[i] * M < 1 (fp64), with uniforms[0..n) in
 *                           [0, 1) drawn by the caller (BAPP-R, §2.6).
 * phase and uniforms are ignored by the kinds that do not use them (uniforms
 * may then be NULL).  Writes min(n, tier_cap) codes to tier_out (may be NULL)
 * and n to *n_pages.  Pure CPU.  Errors: EINVAL (bytes 0, M < 2, unknown
 * kind, null n_pages, RANDOM without uniforms). */
int boost_plan_contrast(int kind, uint64_t bytes, uint32_t M, uint64_t phase,
                        const double *uniforms, uint8_t *tier_out,
                        uint64_t tier_cap, uint64_t *n_pages);

/* C3: modulus under an HBM budget.  The paper always places about an alpha
 * share on host; when the weights exceed a budget we keep the modulo rule and
 * take the largest M in [2, M_alpha] whose HBM-resident pages (whole pages,
 * every tensor placed on its own) fit in hbm_budget_bytes.  footprints may be
 * NULL (all 0).  Errors: EINVAL, ENOMEM (even M = 2 does not fit). */
int boost_modulus_from_budget(const uint64_t *tensor_bytes,
                              const uint64_t *footprints, size_t n_tensors,
                              uint64_t hbm_budget_bytes, uint32_t M_alpha,
                              uint32_t *M);

/* Place one weight tensor by MPP (§3.1, §4.4): plan the tier map, back HBM
 * pages with one device slab and host pages with pinned, device-mapped host
 * memory, copy `bytes` bytes from `src` (host or device address; the bytes are
 * copied, src stays the caller's) and upload a device page table.  The last
 * partial page is zero-filled.  Synchronises (load time only, §4.4).
 * *out is released with boost_tensor_free.
 * Errors: EINVAL, ENODEV, ENOMEM, EHIP. */
int boost_place_weights(boost_ctx *ctx, const void *src, uint64_t bytes,
                        uint32_t M, uint64_t footprint_bytes,
                        boost_tensor **out);

/* Same with an explicit tier map of n_pages codes (n_pages must equal
 * ceil(bytes / 2 MiB)): all-HBM, all-host and contrast placements. */
int boost_place_weights_map(boost_ctx *ctx, const void *src, uint64_t bytes,
                            const uint8_t *tiers, uint64_t n_pages,
                            boost_tensor **out);

/* Tier map and page count of a placed tensor (tier_out may be NULL). */
int boost_tensor_tiers(const boost_tensor *t, uint8_t *tier_out,
                       uint64_t tier_cap, uint64_t *n_pages);

/* The closed form of t's tier map that the GEMV kernels use to find a page
 * (§3.1: placement by page index modulo M over superpages of SP pages):
 * page p is on host iff (p / SP) % M == M - 1, *M = 0 when no page is on
 * host; *M = -1 when the map has no such form (arbitrary maps, staged views),
 * and the kernels read the page tables instead.  Errors: EINVAL (null). */
int boost_tensor_layout(const boost_tensor *t, int32_t *M, int32_t *SP);

/* Copy `bytes` bytes starting at logical offset `offset` of a placed tensor
 * back to host memory `dst` through its page table (checks, synchronises). */
int boost_tensor_read(const boost_tensor *t, uint64_t offset, void *dst,
                      uint64_t bytes);

int boost_tensor_free(boost_tensor *t);

/* ------------------------------------------- a6: prefetch-to-HBM baseline */

/* Prefetch baseline (§2.5 "Prefetching", §5.1 evaluated policies): data that
 * lives on host is copied into HBM before use and read from there, so every
 * staged byte also costs an HBM write.  boost_staged_view makes a view of a
 * placed tensor whose HBM pages are the tensor's own and whose host pages are
 * replaced by staging pages in caller-owned device memory `staging` (at least
 * n_host_pages * 2 MiB bytes, 16-byte aligned).  The view holds no copy of the
 * HBM pages, must be freed (boost_tensor_free) before the tensor, and reads
 * only HBM in decode calls.  Errors: EINVAL (staging too small), ENODEV, EHIP. */
int boost_staged_view(boost_ctx *ctx, const boost_tensor *t, void *staging,
                      uint64_t staging_bytes, boost_tensor **view);

/* Copy the source tensor's host pages into the view's staging pages
 * (host-to-device DMA) on `stream`; a decode call on the view ordered after
 * it reads the staged bytes.  No-op for a view of a tensor with no host page.
 * Errors: EINVAL (not a view), EHIP. */
int boost_prefetch(boost_ctx *ctx, const boost_tensor *view, void *stream);

/* ------------------------------------------------------ a4: decode GEMV */

/* Work-unit schedule of the GEMV (library-wide):
 *   BOOST_SCHED_ADDRESS: workgroups take units in address order, blind to
 *     tiers (the transparent kernel of §3.1: a wave's host share comes only
 *     from placement);
 *   BOOST_SCHED_CAP: CTA specialisation (§3.2): `host_workers` persistent
 *     workgroups, dispatched first, stream every host-page unit while all
 *     other workgroups stream HBM-page units, so host and HBM reads overlap in
 *     every wave (§3 "CAP").  host_workers = 0 picks the default: n_cu / 16
 *     for the GEMV (B <= 6); for the matrix-core kernels one worker per 16
 *     host units of the tensor, at least n_cu / 16 and at most n_cu / 8
 *     (from B = 17 a host unit is one 16-row tile of a work unit, so a host
 *     page spreads over more workers).  Never more workers than host units. */
#define BOOST_SCHED_ADDRESS 0
#define BOOST_SCHED_CAP 1
int boost_gemv_set_schedule(boost_ctx *ctx, int schedule, int host_workers);

/* y[b, n] = sum_k W[n, k] * x[b, k] (§3.1 handwritten matmul; §4.4 up/down
 * projections).  W: placed tensor holding an [N, K] row-major bf16 matrix
 * (nn.Linear layout; bytes must equal N*K*2).  x: device bf16 [B, K]
 * contiguous.  y: device [B, N] contiguous, fp32 (y_dtype BOOST_DTYPE_F32) or
 * bf16 rounded to nearest even (BOOST_DTYPE_BF16).  Accumulation is fp32 and
 * the reduction order is fixed, so results are bitwise reproducible and do
 * not depend on the placement or the schedule.  1 <= B <= 256, K % 8 == 0,
 * N >= 1.  Batches up to 6 run as a GEMV on the vector units; larger ones as a
 * skinny GEMM on the matrix cores (the batch sizes of §5.10), with
 * the same page-confined work units; a matrix too small to fill the GPU at a
 * large batch has K split over several workgroups whose partials go to a
 * workspace owned by the context (64 MiB, allocated by boost_init) and are
 * summed in slice order by a second kernel.  Calls on one context must
 * therefore be ordered (one stream, or streams joined by events): two
 * overlapping split calls would share the workspace.  x must be 16-byte
 * aligned, y 4-byte.
 * Errors: EINVAL, ENODEV, EHIP (launch failure). */
int boost_decode_gemv(boost_ctx *ctx, const boost_tensor *W, int N, int K,
                      const void *x, int B, void *y, int y_dtype, void *stream);

/* The same product with the split-K reduction left to the consumer (§3.1
 * matmul; the fold saves the reduction launch and its round trip through
 * HBM between the projection and the element-wise step after it).  Writes
 * the split-K partial sums to `slices` (caller-owned device memory of
 * boost_gemv_slices_floats(N, K, B, max_slices) floats, 16-byte aligned) and
 * their count S to *n_slices (host int).  Layout: fp32 [S][B][N], then, for
 * every row of W that crosses a 2 MiB page (rows r with r K and r K + K - 1
 * on different pages), its two parts: part h (0: the columns on the earlier
 * page, 1: on the later) of slice s for batch row b at
 * [S B N + ((p 2 + h) S + s) B + b], p the page holding the row's last
 * column.  y[b, n] equals, bit for bit, what boost_decode_gemv returns
 * (fp32): for a row on one page, slices[s][b][n] added over s = 0..S-1 in
 * that order to 0.0f; for a cut row, the parts h = 0 so added, plus the parts
 * h = 1 so added.  S == 1 means slices[0] is y itself (cut rows included).
 * S is chosen as boost_decode_gemv chooses it, halved until it is at most
 * max_slices; it depends only on the shapes, the placement and the context,
 * so it is known on the host when the call returns.
 * It touches no workspace of the context: the partials live in `slices`, and
 * with S == 1 the parts of rows cut between pages of different tiers are
 * staged in a buffer of the tensor W, so calls on different streams may
 * overlap unless they use the same W.
 * 1 <= max_slices <= BOOST_MAX_GEMV_SLICES.  Other arguments and errors as
 * boost_decode_gemv. */
#define BOOST_MAX_GEMV_SLICES 8
int boost_decode_gemv_slices(boost_ctx *ctx, const boost_tensor *W, int N, int K,
                             const void *x, int B, float *slices, int max_slices,
                             int *n_slices, void *stream);

/* Floats a slice buffer of boost_decode_gemv_slices needs for an [N, K]
 * matrix at batch B and up to max_slices slices (host-only arithmetic).
 * Errors: EINVAL (null output, a size below 1). */
int boost_gemv_slices_floats(int N, int K, int B, int max_slices, uint64_t *floats);

/* ------------------------------------------- a2/a3: KV pool and allocator */

/* KV pool placement modes. */
#define BOOST_KV_LPP 0      /* linear page placement, last 1/M of pages on host */
#define BOOST_KV_ALL_HBM 1  /* every page in HBM (HBM-only baseline) */
#define BOOST_KV_ALL_HOST 2 /* every page on host (stress / capacity bound) */
/* Linear split at a capacity budget: each K (and V) tensor keeps its first
 * floor(hbm_budget_bytes / (2 * layers * 2 MiB)) pages in HBM and the rest of
 * its pages on host (the high-throughput setting of §5.2, where the batch
 * grows past what HBM holds and the overflow KV lives on host).  When the
 * tail spans several head regions, blocks carry c or c + 1 host heads, the
 * mixing of §4.5. */
#define BOOST_KV_BUDGET 3

/* Request / block types of the allocator (§4.3). */
#define BOOST_KV_LOCAL 0 /* all-local: no head on host (fewer host heads) */
#define BOOST_KV_SHH 1   /* single-head-host (more host heads when H > M) */

typedef struct boost_kv_cfg {
  uint32_t layers;             /* layers sharing one block id space */
  uint32_t kv_heads;           /* H */
  uint32_t head_dim;           /* D: 64 or 128 */
  uint32_t block_tokens;       /* tokens per block: 16 (§4.3) */
  uint32_t n_blocks;           /* blocks wanted; rounded up so every head's
                                  region is whole pages */
  uint32_t M;                  /* host share of pages 1/M (BOOST_KV_LPP) */
  int32_t tier_mode;           /* BOOST_KV_* */
  uint32_t q_heads;            /* Hq, a multiple of H (attention scratch) */
  uint32_t max_batch;          /* largest B of a decode call (scratch) */
  uint32_t max_blocks_per_seq; /* widest block-table row (scratch) */
  uint64_t hbm_budget_bytes;   /* HBM bytes of the whole pool (BOOST_KV_BUDGET) */
} boost_kv_cfg;

typedef struct boost_kv_info {
  uint32_t nb_pool;               /* blocks in the pool */
  uint32_t blocks_per_page;       /* head-blocks per 2 MiB page */
  uint64_t pages_per_tensor;      /* pages of one layer's K (or V) */
  uint64_t host_pages_per_tensor; /* of which on host (the LPP tail) */
  uint32_t n_shh;                 /* blocks on the SHH list */
  uint32_t shh_host_heads;        /* host heads of an SHH block */
  uint32_t local_host_heads;      /* host heads of an all-local block */
  double tau;                     /* n_shh / nb_pool: the greedy threshold */
} boost_kv_info;

typedef struct boost_kv_usage {
  uint32_t free_shh, free_local;  /* free blocks on each list */
  uint64_t used_blocks;           /* blocks held by requests */
  uint64_t used_host_head_blocks; /* sum of host heads over held blocks */
  uint32_t requests, shh_requests;
} boost_kv_usage;

/* Create a KV pool (§4.2 LPP; §4.5 heads-outermost layout).  Every layer has
 * a K and a V tensor laid out [H][NB][T][D] bf16 with NB rounded up so each
 * head's region is whole 2 MiB pages; the last floor(pages / M) pages of each
 * tensor are host-resident (BOOST_KV_LPP), so a block's host heads are the
 * heads whose region reaches into that tail.  Blocks with the larger host-head
 * count form the SHH list, the rest the all-local list (§4.3, §4.5).  On a
 * device context the pages are backed (HBM slab + pinned host pages) and a
 * device page table is uploaded; on a plan-only context only the allocator
 * exists.  Errors: EINVAL (shape, M < 2 for LPP, head-block not dividing a
 * page), ENOMEM, EHIP. */
int boost_kv_pool_create(boost_ctx *ctx, const boost_kv_cfg *cfg,
                         boost_kv_pool **out);
int boost_kv_pool_info(const boost_kv_pool *pool, boost_kv_info *info);
int boost_kv_pool_destroy(boost_kv_pool *pool);

/* Host heads (0..H) of one block.  Errors: EINVAL (block out of range). */
int boost_kv_block_host_heads(const boost_kv_pool *pool, int32_t block,
                              uint32_t *n_host_heads);

/* Append n_blocks blocks to request `request_id` (§4.3 wave-aware block
 * fulfillment).  A new request takes the SHH type when the free-SHH fraction
 * exceeds tau (strictly) and SHH blocks are free, else all-local if any are
 * free, else SHH; an existing request keeps its type.  Blocks come from the
 * list of the request's type, lowest id first; when that list empties the
 * request switches to the other list and stays there (sticky fallback).  The
 * call is all-or-nothing: with fewer than n_blocks free blocks nothing changes
 * and BOOST_EAGAIN is returned (the scheduler decides, §4.3).  block_ids_out
 * receives n_blocks ids in allocation order.  CPU only.
 * Errors: EINVAL (n_blocks 0, null), EAGAIN. */
int boost_kv_alloc(boost_kv_pool *pool, uint64_t request_id, uint32_t n_blocks,
                   int32_t *block_ids_out);

/* Return every block of the request to its list and forget the request.
 * Errors: EINVAL (unknown request). */
int boost_kv_free(boost_kv_pool *pool, uint64_t request_id);

/* Current type (BOOST_KV_LOCAL / BOOST_KV_SHH) of a live request. */
int boost_kv_request_type(const boost_kv_pool *pool, uint64_t request_id,
                          int *type);
int boost_kv_stats(const boost_kv_pool *pool, boost_kv_usage *out);

/* ------------------------------------------------ a5: paged attention */

/* Write n tokens of one layer into the pool: token i goes to slot
 * slots[i] = block * T + offset (negative slots are skipped, slots past the
 * pool are ignored).  k, v: device bf16 [n, H, D] contiguous; slots: device
 * int32 [n].  Asynchronous on `stream`.  Errors: EINVAL, ENODEV, EHIP. */
int boost_kv_write(boost_ctx *ctx, const boost_kv_pool *pool, int layer,
                   const int32_t *slots, const void *k, const void *v, int n,
                   void *stream);

/* GQA decode attention over the pool (§3.3 KV head chunks per workgroup;
 * §4.5 paged layout):  for request b and query head h (KV head g = h / (Hq/H))
 *   o[b,h,:] = sum_t softmax_t(scale * q[b,h,:] . k[b,t,g,:]) v[b,t,g,:]
 * over t < ctx_lens[b], where token t of request b lives in block
 * block_tables[b * max_blocks + t / T] at offset t % T.  Work item = (KV head,
 * request, context partition): the Hq/H query heads of a KV head share every
 * K/V load, partitions are merged by log-sum-exp in a fixed order, and items
 * of the heads that can hold host pages are dispatched first.
 * q: device bf16 [B, Hq, D]; block_tables: device int32 [B, max_blocks];
 * ctx_lens: device int32 [B]; out: device [B, Hq, D] fp32 or bf16.
 * scale <= 0 selects 1/sqrt(D).  A block id outside [0, nb_pool) at a
 * position inside the context is skipped: its 16 tokens are left out of the
 * softmax (no read, no weight), as if they were not in the context; a row
 * whose every token is skipped, or ctx_lens[b] = 0, gives a zero row.
 * 1 <= B <= max_batch,
 * Hq == q_heads of the pool, max_blocks <= max_blocks_per_seq.
 * Errors: EINVAL, ENODEV, EHIP. */
int boost_paged_attn_decode(boost_ctx *ctx, const boost_kv_pool *pool, int layer,
                            const void *q, int B, int Hq,
                            const int32_t *block_tables, int max_blocks,
                            const int32_t *ctx_lens, float scale, void *out,
                            int out_dtype, void *stream);

/* Allocation-free variant of boost_paged_attn_decode, for callers that cannot
 * allocate device memory or use a pool's scratch (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * arguments, kernels and bits, but the partition partials live in a
 * fixed-size static device array of the library (16.25 MiB per device, held
 * until the process ends) instead of the pool's scratch.  The call allocates
 * nothing.  Limit: B * Hq * partitions <= 32768 partial rows, where the
 * partition count is the one the call picks from max_blocks, B and the KV
 * heads (batch 64 x 32 query heads at up to 4096 tokens, or batch 256 x 32 at
 * up to 8192, fit); larger calls fail with BOOST_EINVAL.  Every call on one
 * GPU shares that GPU's array: calls that overlap on one GPU (on different
 * streams, or from different pools or threads) race and must be ordered by
 * the caller.  Nothing in the array needs to start at zero (each call writes
 * every partial it reads).  Errors: as boost_paged_attn_decode, and EINVAL
 * beyond the limit. */
int boost_paged_attn_decode_noalloc(boost_ctx *ctx, const boost_kv_pool *pool,
                                    int layer, const void *q, int B, int Hq,
                                    const int32_t *block_tables, int max_blocks,
                                    const int32_t *ctx_lens, float scale,
                                    void *out, int out_dtype, void *stream);

/* -------------------------------------------- a6: glue of a full decode step */

/* The paper measures whole decode steps of Llama-style models (§5.1) without
 * restating the model; these operators complete a pre-norm step around the
 * GEMV and attention calls.  The residual stream is fp32 [B, d]; operands of
 * products and of attention are bf16.  All calls are asynchronous on
 * `stream`, allocate nothing and fail with EINVAL on bad sizes or nulls and
 * ENODEV on a plan-only context. */

/* out[b, :] = embedding row tokens[b] of the placed [V, d] bf16 tensor E
 * (read through its page table), as fp32.  A token outside [0, V) gives a
 * zero row. */
int boost_embed_gather(boost_ctx *ctx, const boost_tensor *E, int V, int d,
                       const int32_t *tokens, int B, float *out, void *stream);

/* out[b, i] = bf16(x[b, i] / sqrt(mean_i x[b, i]^2 + eps) * w[i]).
 * x fp32 [B, d], w bf16 [d], out bf16 [B, d]. */
int boost_rmsnorm(boost_ctx *ctx, const float *x, const void *w, int B, int d,
                  float eps, void *out, void *stream);

/* x[b, i] += r[b, i] (fp32, in place), then out = the RMSNorm of the new x
 * exactly as boost_rmsnorm computes it: the same bits as boost_residual_add
 * followed by boost_rmsnorm, in one launch (the step's residual add and the
 * next norm).  r fp32 [B, d], 16-byte aligned (EINVAL otherwise). */
int boost_add_rmsnorm(boost_ctx *ctx, float *x, const float *r, const void *w, int B,
                      int d, float eps, void *out, void *stream);

/* boost_add_rmsnorm with r handed over as the S split-K slices of
 * boost_decode_gemv_slices for a [d, K] matrix (the layout documented there,
 * 16-byte aligned): r is their sum in the order given there, so x and out get
 * the same bits as boost_decode_gemv followed by boost_add_rmsnorm.
 * 1 <= S <= BOOST_MAX_GEMV_SLICES, K >= 1 (the producing matrix's). */
int boost_add_rmsnorm_slices(boost_ctx *ctx, float *x, const float *r, int S, int K,
                             const void *w, int B, int d, float eps, void *out,
                             void *stream);

/* Split the fused qkv output fp32 [B, (Hq + 2H) D] (query heads, then key
 * heads, then value heads) into bf16 q [B, Hq, D], k [B, H, D], v [B, H, D],
 * rotating query and key heads by RoPE at positions[b]: element i pairs with
 * i + D/2 and turns by positions[b] * theta^(-2i/D). */
int boost_rope_qkv(boost_ctx *ctx, const float *qkv, const int32_t *positions,
                   int B, int Hq, int H, int D, double theta, void *q, void *k,
                   void *v, void *stream);

/* Append the new token of every request to one layer of the pool: token b
 * at position positions[b] goes to block block_tables[b][positions[b] / T],
 * offset positions[b] % T.  k, v bf16 [B, H, D].  Positions or blocks
 * outside the table / pool are skipped. */
int boost_kv_append(boost_ctx *ctx, const boost_kv_pool *pool, int layer,
                    const int32_t *block_tables, int max_blocks,
                    const int32_t *positions, const void *k, const void *v,
                    int B, void *stream);

/* boost_rope_qkv followed by boost_kv_append in one launch: the query heads
 * go to q (bf16 [B, Hq, D]) and the rotated key and converted value heads
 * straight into the token's slot of the pool (H and D are the pool's), with
 * the same bits and the same skipping rules as the two calls. */
int boost_rope_kv_append(boost_ctx *ctx, const boost_kv_pool *pool, int layer,
                         const float *qkv, const int32_t *positions, int B, int Hq,
                         double theta, const int32_t *block_tables, int max_blocks,
                         void *q, void *stream);

/* boost_rope_kv_append with qkv handed over as the S split-K slices of
 * boost_decode_gemv_slices for a [(Hq + 2H) D, K] matrix (the layout
 * documented there): every element is their sum in the order given there, so
 * q and the pool get the same bits as boost_decode_gemv followed by
 * boost_rope_kv_append.  1 <= S <= BOOST_MAX_GEMV_SLICES, K >= 1. */
int boost_rope_kv_append_slices(boost_ctx *ctx, const boost_kv_pool *pool, int layer,
                                const float *qkv, int S, int K, const int32_t *positions,
                                int B, int Hq, double theta, const int32_t *block_tables,
                                int max_blocks, void *q, void *stream);

/* out[b, j] = bf16(silu(gu[b, j]) * gu[b, F + j]) for the fused gate_up
 * output fp32 [B, 2F] (gate rows first). */
int boost_silu_mul(boost_ctx *ctx, const float *gu, int B, int F, void *out,
                   void *stream);

/* x[i] += y[i] for n fp32 values. */
int boost_residual_add(boost_ctx *ctx, float *x, const float *y, int64_t n,
                       void *stream);

/* ids[b] = argmax_j logits[b, j] (fp32 [B, V]); ties give the lowest index. */
int boost_argmax(boost_ctx *ctx, const float *logits, int B, int V, int32_t *ids,
                 void *stream);

#ifdef __cplusplus
}
#endif

#endif /* BOOST_CAP_H */
