/*
 * tensorcast_hip.h -- C ABI of the MI355X (gfx950) data path beneath the
 * tensor lifecycle primitives of TensorCast (arXiv 2608.06007).
 *
 * The paper's runtime moves tensor states between engine-resident layouts and
 * transfer locations: a request's paged KV blocks are exported with publish()
 * and loaded back with hydrate(); a tensor-parallel rank materializes only
 * its slice of each weight through view(slice) + tensor_dict(); replicas move
 * in batches through prefetch_many(); transform_into() transforms a tensor by
 * a `spec` rule while filling an instance-owned buffer (Sec. 3.2, Table 2).
 * This library is the device-side hot path of those operations: descriptor
 * driven gathers and scatters between device layouts and contiguous buffers
 * (including resharding between tensor-parallel layouts), a bf16 -> fp8 E4M3
 * cast with one fp32 scale per 128x128 tile as one concrete transform_into
 * rule, and its inverse; per-fragment integrity digests for the pipeline's
 * verify stage; and the pinned staging that moves such bytes between host
 * memory and the device (Sec. 5).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Pointers are DEVICE pointers unless a comment says "host".  All device
 *   buffers belong to the caller (the paper's caller-leased ownership,
 *   Sec. 3.2 "Artifact") and must stay valid until the work enqueued on
 *   `stream` has completed.  The library keeps no pointer after returning.
 * - Calls are asynchronous and stream-ordered: they validate arguments on the
 *   host, enqueue kernels on `stream` and return, without waiting for the
 *   device.  n == 0 enqueues nothing.  The exceptions say so: the calls that
 *   hand a device-computed number back to the host (tc_plan_fragments,
 *   tc_plan_status) and the host staging calls.  The library allocates
 *   nothing that outlives a call, on the device or the host, apart from a
 *   stager's own ring (created and destroyed by the caller) and the fixed
 *   device array behind tc_cast_fp8_blockscaled_noalloc.
 * - Calls are pure functions of their inputs, so re-running one after a
 *   failure is safe (the paper's idempotent retry, Sec. 3.2 "Plan").
 * - Errors: TC_ERR_INVALID_ARGUMENT for null pointers, negative sizes,
 *   geometry that cannot be valid, and fragment, item or task counts above
 *   2^33 (the plan kernels' grids grow with them); TC_ERR_WORKSPACE for a workspace that is
 *   too small; TC_ERR_HOST_RESOURCES when host memory (for validation or
 *   host tables) or host threads cannot be had; no C++ exception leaves the
 *   library; TC_ERR_HIP when the HIP runtime rejects a launch (the HIP
 *   error code is then available from tc_last_hip_error()).  With validation
 *   on (tc_set_validate(1) or TC_VALIDATE=1 in the environment) the calls
 *   also copy the descriptors to the host, synchronize the stream, and
 *   report ids out of range (TC_ERR_OUT_OF_RANGE) and aliasing writes
 *   (TC_ERR_ALIAS) before launching; without it those are preconditions.
 * - HIP graph capture: with validation off, every call that only enqueues
 *   kernels may be captured and the graph replayed: tc_gather_blocks,
 *   tc_scatter_blocks, tc_plan_fragments_async, tc_copy_fragments,
 *   tc_copy_planned, tc_copy_planned_digest, tc_digest_planned, the
 *   block-scaled cast and its inverse (one-call, prepare and planned forms)
 *   and tc_cast_fp8_scaled.  They issue no memset and no host
 *   synchronization; host-side tables travel by value in the kernel launches,
 *   so a graph keeps the values it captured.  tc_plan_fragments and
 *   tc_plan_status (they read the device back) and the staging calls must not
 *   be captured.
 */
#ifndef TENSORCAST_HIP_H
#define TENSORCAST_HIP_H

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TC_OK = 0,
  TC_ERR_INVALID_ARGUMENT = 1,
  TC_ERR_OUT_OF_RANGE = 2,
  TC_ERR_ALIAS = 3,
  TC_ERR_HIP = 4,
  TC_ERR_WORKSPACE = 5,
  TC_ERR_HOST_RESOURCES = 6 /* host memory or threads could not be had */
} tc_status;

/* Largest number of regions a block pool may have. */
#define TC_MAX_REGIONS 256

/* ------------------------------------------------------------------------
 * Paged KV blocks: publish / hydrate (Sec. 3.2 "Operation", Table 2;
 * KV pages as high-cardinality Artifacts, Sec. 4.2 and Sec. 6.3)
 *
 * An engine keeps its KV cache in `num_regions` regions (one per layer and
 * K|V; region r = 2*layer + kv).  Inside a region, block b starts at byte
 * b * block_stride and holds block_bytes bytes.  Regions may be separate
 * allocations, or views into one allocation (for [2][blocks][...] or
 * [blocks][2][...] engine layouts, choose base and stride accordingly).
 * The transfer buffer is id-major, then region-major: the block of id i in
 * region r sits at byte (i * num_regions + r) * block_bytes, so one block's
 * KV for all layers is contiguous.
 * ------------------------------------------------------------------------ */
typedef struct {
  const uint64_t* region_base; /* host array [num_regions]: device address of each region */
  int32_t num_regions;         /* 1 .. TC_MAX_REGIONS */
  int64_t num_blocks;          /* blocks per region; ids must lie in [0, num_blocks) */
  int64_t block_bytes;         /* bytes per block and region, > 0 */
  int64_t block_stride;        /* bytes between consecutive blocks, >= block_bytes */
} tc_block_pool;
/* Every call that takes a pool returns TC_ERR_INVALID_ARGUMENT, before any
 * work is enqueued, for a pool outside these bounds, a null region address,
 * or byte extents beyond 2^63 - 1 (num_blocks * block_stride, num_regions *
 * block_bytes, or a batch's n * num_regions * block_bytes). */

/* publish: out[i][r][0:B] = region_r[ids[i]*stride : +B] for i < n, r < R.
 * ids: device int32[n]; repeated ids are allowed.  out: device buffer of
 * n * num_regions * block_bytes bytes that must not overlap the pool. */
tc_status tc_gather_blocks(const tc_block_pool* pool, const int32_t* ids, int64_t n,
                           void* out, hipStream_t stream);

/* hydrate: region_r[ids[i]*stride : +B] = in[i][r][0:B] for i < n, r < R.
 * ids must be distinct (else the result depends on write order; checked as
 * TC_ERR_ALIAS in validation mode).  in must not overlap the pool. */
tc_status tc_scatter_blocks(const tc_block_pool* pool, const int32_t* ids, int64_t n,
                            const void* in, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Fragment lists: batched replica moves (prefetch_many, Table 2) and the
 * transfer stage of the materialization pipeline (Sec. 5).
 *
 * Each descriptor copies len bytes from src_base + src_off to
 * dst_base + dst_off.  Destination ranges must be pairwise disjoint and must
 * not overlap any source range (this is a copy, not a memmove).  There is no
 * alignment requirement; 16-byte-aligned fragments take the fast path.
 * len == 0 is allowed.
 * ------------------------------------------------------------------------ */
typedef struct {
  uint64_t src_off; /* bytes from src_base */
  uint64_t dst_off; /* bytes from dst_base */
  uint64_t len;     /* bytes */
} tc_fragment;

/* Recommended bytes of device workspace for a plan of n descriptors.  A
 * plan cuts every fragment into tasks of at most `piece` bytes (1 KiB, or the
 * next power of two, at most 2^30, that keeps the task table inside the
 * workspace) and spreads the tasks over the whole GPU, one task per wave.
 * With 1 KiB pieces every task after a fragment's first starts on a 128-byte
 * line of the destination, so a fragment may take one task more.  A
 * task costs 32 bytes (the packed task and its digest slot) plus 16 bytes per
 * 1024 tasks; a descriptor costs at most ~48 bytes of planning scratch.  A
 * workspace with room for T >= n + 1 tasks accepts payloads up to
 * (T - n) * 2^30 bytes (beyond that the plan returns TC_ERR_WORKSPACE); this
 * size has room for 4n + 2^23 tasks, which keeps 1 KiB pieces for payloads
 * up to ~2 KiB per fragment plus 8 GiB.  Offsets plus lengths must stay below
 * 2^48. */
size_t tc_copy_fragments_workspace(int64_t n); /* 0 for n < 0 or n > 2^33 */
/* Smallest workspace a plan of n descriptors accepts (room for n + 1 tasks;
 * the task size then grows to fit, so payloads up to 2^30 bytes always fit).
 * Fewer, longer tasks use fewer waves: a copy needs tens of thousands of
 * tasks to fill the GPU, which the recommended size provides. */
size_t tc_copy_fragments_workspace_min(int64_t n);

/* Copy every fragment: a plan (tc_plan_fragments_async) and a copy that
 * takes the plan's task count on the device (tc_copy_planned with
 * TC_TASKS_FROM_PLAN).  frags: device tc_fragment[n].  workspace: device
 * buffer, 256-byte aligned.  Fully asynchronous: the piece size, the
 * destination reordering and the task count are decided by the planning
 * kernels, and the copy's grid is bounded by the workspace's capacity.  The
 * workspace may be reused once the stream has passed the copy.
 * Failures the plan finds on the device -- a non-empty fragment whose source
 * or destination range ends past 2^48 (TC_ERR_OUT_OF_RANGE), a payload the
 * workspace cannot hold even with pieces of 2^30 bytes (TC_ERR_WORKSPACE) --
 * copy nothing and are reported by tc_plan_status on this workspace;
 * argument errors are returned at once. */
tc_status tc_copy_fragments(const void* src_base, void* dst_base, const tc_fragment* frags,
                            int64_t n, void* workspace, size_t workspace_bytes,
                            hipStream_t stream);

/* Plan once, copy many times (a rank's weight-slice list is fixed for a
 * model).  tc_plan_fragments_async enqueues the plan for frags into
 * workspace and returns.  tc_plan_fragments does the same and then waits for
 * it: it returns the plan's status (the device-found failures above) and its
 * task count in *total_tasks (host).  tc_copy_planned then copies with the
 * plan -- asynchronously, as often as wanted -- for any src/dst bases, while
 * the workspace is kept unchanged.  total_tasks is the plan's count (the
 * copy's grid is then sized exactly), or TC_TASKS_FROM_PLAN (the kernel reads
 * it from the plan, no host round trip; a failed plan copies nothing).
 * total_tasks == 0 means there is nothing to copy; a count larger than the
 * workspace's task table can hold is TC_ERR_WORKSPACE. */
#define TC_TASKS_FROM_PLAN UINT64_MAX
tc_status tc_plan_fragments_async(const tc_fragment* frags, int64_t n, void* workspace,
                                  size_t workspace_bytes, hipStream_t stream);
tc_status tc_plan_fragments(const tc_fragment* frags, int64_t n, void* workspace,
                            size_t workspace_bytes, uint64_t* total_tasks /* host, out */,
                            hipStream_t stream);
tc_status tc_copy_planned(const void* src_base, void* dst_base, const void* workspace,
                          size_t workspace_bytes, uint64_t total_tasks, hipStream_t stream);
/* The status of the plan last written into workspace (TC_OK,
 * TC_ERR_OUT_OF_RANGE, TC_ERR_WORKSPACE, or TC_ERR_INVALID_ARGUMENT for more
 * than 2^33 tasks), and its task count in *total_tasks (host; 0 unless
 * TC_OK).  Waits for `stream` to reach that point.  workspace must hold a
 * plan. */
tc_status tc_plan_status(const void* workspace, size_t workspace_bytes,
                         uint64_t* total_tasks /* host, out, may be NULL */, hipStream_t stream);

/* Integrity digests (the "verify integrity" stage of the materialization
 * pipeline, Sec. 5).  The paper names the stage but no checksum; this
 * library's digest of a fragment with bytes b_0 .. b_(len-1) is the pair
 *   S1 = sum_i b_i            (mod 2^64)
 *   S2 = sum_i (i + 1) * b_i  (mod 2^64)
 * which changes when any single byte changes and when two differing bytes
 * swap places (a Fletcher-style position-weighted sum, computable in parallel
 * over any cut of the fragment).
 *
 * tc_copy_planned_digest: tc_copy_planned with the same plan, that also
 * writes the digest of every planned fragment, taken over the bytes it
 * copies, into digests[2f], digests[2f + 1] (device uint64_t[2n], 8-byte
 * aligned; fragments in the order given to tc_plan_fragments).  n must be
 * the plan's descriptor count.  The copy reads each source byte once and
 * writes it once; the digests cost 32 bytes of workspace traffic per task
 * and a short reduction.  The workspace is written (its digest slots), so
 * two digest calls with one workspace must not overlap in time; the plan
 * itself is left unchanged.  Asynchronous.
 *
 * tc_digest_planned: the digests alone, read from base at the fragments'
 * source offsets (side TC_DIGEST_SRC: what a publisher records) or at their
 * destination offsets (TC_DIGEST_DST: what a reader checks after the copy).
 * Nothing is written outside digests and the workspace's digest slots.
 *
 * Errors: TC_ERR_INVALID_ARGUMENT for n < 0, null pointers with work to do, a
 * misaligned workspace or digest array, and (when validating) a header that
 * disagrees with n or total_tasks; TC_ERR_WORKSPACE if total_tasks exceeds
 * the workspace's task capacity for n descriptors. */
#define TC_DIGEST_SRC 0
#define TC_DIGEST_DST 1
tc_status tc_copy_planned_digest(const void* src_base, void* dst_base, void* workspace,
                                 size_t workspace_bytes, uint64_t total_tasks, int64_t n,
                                 uint64_t* digests, hipStream_t stream);
tc_status tc_digest_planned(const void* base, int32_t side, void* workspace,
                            size_t workspace_bytes, uint64_t total_tasks, int64_t n,
                            uint64_t* digests, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Tensor-parallel views: view(slice) + tensor_dict() (Table 2; each rank
 * retrieves only its slice of every weight, Sec. 6.1 and 6.2).
 *
 * A weight is a row-major matrix [rows][cols] of elem_bytes-byte elements
 * in a source buffer.  `split` says which of its dimensions the
 * tensor-parallel group divides: TC_SPLIT_ROWS gives rank r the rows
 * [r*rows/tp, (r+1)*rows/tp) (column-parallel layers), TC_SPLIT_COLS the
 * columns [r*cols/tp, (r+1)*cols/tp) (row-parallel layers), TC_SPLIT_NONE the
 * whole matrix.  The rank's slice is written densely row-major at dst_off
 * with row stride dst_ld elements.
 * These two builders run on the host and only describe the moves.
 * ------------------------------------------------------------------------ */
typedef enum { TC_SPLIT_NONE = 0, TC_SPLIT_ROWS = 1, TC_SPLIT_COLS = 2 } tc_split;

typedef struct {
  uint64_t src_off;   /* byte offset of element [0][0] of the full matrix */
  int64_t rows, cols; /* full matrix shape in elements */
  int64_t src_ld;     /* elements between source rows (>= cols) */
  uint64_t dst_off;   /* byte offset of the rank's slice in the destination */
  int64_t dst_ld;     /* elements between destination rows (>= slice cols) */
  int32_t elem_bytes; /* 1, 2, 4 or 8 */
  int32_t split;      /* tc_split */
} tc_tp_view;

/* Host: number of fragments tc_tp_fragments produces for these views
 * (-1 on invalid arguments: tp < 1, rank outside [0, tp), a split dimension
 * not divisible by tp, ld too small, bad elem_bytes). */
int64_t tc_tp_fragment_count(const tc_tp_view* views /* host */, int64_t n_views, int32_t tp,
                             int32_t rank);

/* Host: write the fragments that materialize rank `rank`'s slices into
 * out (host array with room for `capacity` entries); *written receives the
 * count.  Rows that are contiguous in both source and destination are merged
 * into one fragment. */
tc_status tc_tp_fragments(const tc_tp_view* views /* host */, int64_t n_views, int32_t tp,
                          int32_t rank, tc_fragment* out /* host */, int64_t capacity,
                          int64_t* written /* host */);

/* ------------------------------------------------------------------------
 * Cross-layout reshard: a weight stored as the slices of a src_tp-way
 * tensor-parallel split is rearranged into one rank's slice of a dst_tp-way
 * split along the same dimension (resharding checkpoint tensors into the
 * layouts other parallel configurations need, Sec. 2.1; rank-specific
 * resharding with view() and transform_into(), Sec. 7).
 *
 * Source rank s holds its slice densely row-major at byte src_off[s] of the
 * source buffer: rows [s*rows/src_tp, (s+1)*rows/src_tp) for TC_SPLIT_ROWS,
 * columns [s*cols/src_tp, ...) for TC_SPLIT_COLS, the whole matrix for
 * TC_SPLIT_NONE (then only src_off[0] is read).  The destination rank's slice
 * is written densely row-major at byte dst_off of the destination buffer.
 * Slices of consecutive views placed back to back give fused layouts (for
 * example q, k, v of one rank stacked by rows).  Host builder only; the moves
 * run through tc_plan_fragments / tc_copy_planned.
 * ------------------------------------------------------------------------ */
typedef struct {
  const uint64_t* src_off; /* host array [src_tp]: byte offset of each source rank's slice */
  int64_t rows, cols;      /* full matrix shape in elements */
  int32_t elem_bytes;      /* 1, 2, 4 or 8 */
  int32_t split;           /* tc_split, the same dimension on both sides */
  int32_t src_tp;          /* ranks of the source split (>= 1) */
  int32_t reserved;        /* 0 */
  uint64_t dst_off;        /* byte offset of the destination rank's slice */
} tc_reshard_view;

/* Host: number of fragments tc_reshard_fragments produces (-1 on invalid
 * arguments: a null src_off, tp < 1, rank out of range, a split dimension
 * not divisible by src_tp or dst_tp, bad elem_bytes). */
int64_t tc_reshard_fragment_count(const tc_reshard_view* views /* host */, int64_t n_views,
                                  int32_t dst_tp, int32_t dst_rank);

/* Host: write the fragments that build rank dst_rank's slices of a
 * dst_tp-way split into out (room for `capacity`); *written gets the count.
 * Contiguous runs are merged: a row split needs one fragment per overlapping
 * source rank, a column split one per row and overlapping source rank. */
tc_status tc_reshard_fragments(const tc_reshard_view* views /* host */, int64_t n_views,
                               int32_t dst_tp, int32_t dst_rank, tc_fragment* out /* host */,
                               int64_t capacity, int64_t* written /* host */);

/* ------------------------------------------------------------------------
 * transform_into with an fp8 spec (Table 2, Sec. 3.2): bf16 -> OCP FP8 E4M3
 * with one fp32 scale per 128x128 tile, for weight synchronization
 * (Sec. 6.2).  The paper fixes no numeric format; this rule is:
 *   per tile (edge tiles partial), amax = max |x| over its elements;
 *   finite tile, amax > 0: s = RN_f32(amax / 448), q = E4M3(RN_f32(x / s));
 *   finite tile, amax = 0: s = 0, q = sign bit of x (0x00 or 0x80);
 *   tile holding Inf/NaN:  s = NaN (0x7FC00000), every q = 0x7F.
 * E4M3(v): nearest finite E4M3 value with ties to even mantissa, |v| >= 448
 * saturating to +-448 (0x7E/0xFE), NaN -> 0x7F.  x / s is a correctly
 * rounded binary32 division; subnormal scales are kept.
 * ------------------------------------------------------------------------ */
typedef struct {
  uint64_t src_off;   /* bf16 elements from src_base to element [0][0] */
  int64_t rows, cols; /* matrix shape (elements) */
  int64_t src_ld;     /* bf16 elements between source rows (>= cols) */
  uint64_t dst_off;   /* bytes from dst_base to code [0][0] */
  int64_t dst_ld;     /* bytes between destination rows (>= cols) */
  uint64_t scale_off; /* floats from scale_base to scale [0][0] */
  int64_t scale_ld;   /* floats between rows of the scale grid (>= ceil(cols/128)) */
} tc_cast_item;

/* Host: the cast item for rank `rank`'s slice of a bf16 weight described by
 * a view (elem_bytes must be 2; view.dst_off is taken as the code offset in
 * bytes), with its scale grid at scale_off (row stride = its tile columns).
 * Returns TC_ERR_INVALID_ARGUMENT for the same reasons as
 * tc_tp_fragment_count. */
tc_status tc_tp_cast_item(const tc_tp_view* view /* host */, int32_t tp, int32_t rank,
                          uint64_t scale_off, tc_cast_item* out /* host */);

/* Host: cast items (for tc_cast_fp8_blockscaled) that build rank dst_rank's
 * fp8 slices of a dst_tp-way split straight from bf16 source slices of a
 * src_tp-way split: the reshard and the transform_into rule in one pass
 * (rank-specific resharding with view() + transform_into(), Sec. 7).  Views
 * as for tc_reshard_fragments with elem_bytes 2 and BYTE offsets: src_off[s]
 * of each bf16 source slice (even), dst_off of the fp8 destination slice
 * (one byte per element, densely row-major); scale_off[i] (host) is the
 * float offset of view i's scale grid, ceil(rows_d/128) x ceil(cols_d/128)
 * row-major for the destination slice's shape rows_d x cols_d.  One item per
 * overlapping source slice.  The destination's tiles are those of its own
 * slice, so every boundary between two source slices must lie on a multiple
 * of 128 from the destination slice's first row (row split) or column (column
 * split); otherwise, and for elem_bytes != 2 or an odd src_off, the count is
 * -1 and the builder returns TC_ERR_INVALID_ARGUMENT.  TC_ERR_WORKSPACE if
 * `capacity` items do not fit. */
int64_t tc_reshard_cast_item_count(const tc_reshard_view* views /* host */, int64_t n_views,
                                   int32_t dst_tp, int32_t dst_rank);
tc_status tc_reshard_cast_items(const tc_reshard_view* views /* host */,
                                const uint64_t* scale_off /* host [n_views] */, int64_t n_views,
                                int32_t dst_tp, int32_t dst_rank, tc_cast_item* out /* host */,
                                int64_t capacity, int64_t* written);

/* Bytes of device workspace tc_cast_fp8_blockscaled needs for n items. */
size_t tc_cast_fp8_workspace(int64_t n_items);
/* Bytes of a workspace that also holds a per-tile table for these items
 * (HOST array): 32 bytes for every full 128x128 tile, after the item table.
 * With it the streaming kernels find each tile's rows with one load instead
 * of searching the items (on a 70B-shaped shard about 4% faster for the
 * cast and 5% for its inverse, which then splits each tile over four
 * workgroups).  Any
 * workspace of at least tc_cast_fp8_workspace(n_items) bytes works; the
 * table is built whenever the workspace has room for it.  0 for an invalid
 * item or more than 2^33 items. */
size_t tc_cast_fp8_workspace_tiles(const tc_cast_item* items /* host */, int64_t n_items);

/* A tile table made by tc_cast_fp8_prepare or tc_dequant_fp8_prepare (host
 * struct, filled by the library): the item count, the tiles of the
 * streaming path and of the element-wise path, the residues mod 16 of the
 * input and output bases the table was made for (a tile's path depends on
 * its rows' alignment), and whether the workspace also holds the per-tile
 * table (1) or not (0). */
typedef struct {
  int64_t n_items;
  uint64_t full_tiles;
  uint64_t edge_tiles;
  uint32_t in_align;
  uint32_t out_align;
  uint32_t tiled;
  uint32_t reserved; /* 0 */
} tc_tile_plan;

/* Cast every item.  items: HOST array tc_cast_item[n_items] (a model has a
 * few hundred); the library writes it, with its tile offsets, into the
 * device workspace (256-byte aligned) by small kernels that carry the table
 * in their launch arguments, so the host array may be reused as soon as the
 * call returns and nothing is staged or allocated.  Destination codes and
 * scale grids of different items must not overlap one another or the
 * source.  tile must be 128.  Source rows are read through src_ld, so a
 * strided slice of a full weight is cast in place without a gather.  The
 * workspace may be reused once the stream has passed the call.
 * This is tc_cast_fp8_prepare followed by tc_cast_fp8_planned. */
tc_status tc_cast_fp8_blockscaled(const void* src_base, void* dst_base, float* scale_base,
                                  const tc_cast_item* items, int64_t n_items, int32_t tile,
                                  void* workspace, size_t workspace_bytes, hipStream_t stream);

/* The two halves, for casts repeated with one item list (a rank's weights
 * at every synchronization, Sec. 6.2): tc_cast_fp8_prepare checks the items
 * (same errors as tc_cast_fp8_blockscaled), enqueues the table's writes into
 * the workspace and fills *plan (host).  tc_cast_fp8_planned then launches
 * only the cast kernels, as often as wanted while the workspace is kept, for
 * any bases with the residues mod 16 recorded in the plan
 * (TC_ERR_INVALID_ARGUMENT otherwise).  A plan with tiled = 1 needs a
 * workspace that still holds the per-tile table (TC_ERR_WORKSPACE
 * otherwise); tiled above 1 is TC_ERR_INVALID_ARGUMENT. */
tc_status tc_cast_fp8_prepare(const void* src_base, const void* dst_base, const tc_cast_item* items,
                              int64_t n_items, int32_t tile, void* workspace,
                              size_t workspace_bytes, tc_tile_plan* plan /* host, out */,
                              hipStream_t stream);
tc_status tc_cast_fp8_planned(const void* src_base, void* dst_base, float* scale_base,
                              const void* workspace, size_t workspace_bytes,
                              const tc_tile_plan* plan /* host */, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * tc_cast_fp8_blockscaled without a workspace.  The tile table lives in a
 * fixed array of device memory that the library holds on each device it
 * runs on, 332,288 bytes, until the process ends; nothing is allocated, on
 * the device or the host.  The array used is that of the device that runs
 * `stream` (the current device for the null stream).  At most TC_NOALLOC_MAX_ITEMS items: more is
 * TC_ERR_WORKSPACE, before anything is enqueued.  Validation mode does not
 * apply (its checks need host memory).  Every call on one device rewrites
 * that device's array, so two calls that overlap in time on one device race:
 * serialize them (for example, issue them on one stream).  Other arguments
 * and errors as for tc_cast_fp8_blockscaled. */
#define TC_NOALLOC_MAX_ITEMS 4096
tc_status tc_cast_fp8_blockscaled_noalloc(const void* src_base, void* dst_base, float* scale_base,
                                          const tc_cast_item* items /* host */, int64_t n_items,
                                          int32_t tile, hipStream_t stream);

/* q[i] = E4M3(RN_f32(bf16(src[i]) / scale)) for i < n, one given scale (no
 * amax).  Quotients that overflow saturate; NaN gives 0x7F. */
tc_status tc_cast_fp8_scaled(const void* src_bf16, int64_t n, float scale, void* dst_e4m3,
                             hipStream_t stream);

/* ------------------------------------------------------------------------
 * The inverse rule: E4M3 codes with their per-tile fp32 scales back to bf16,
 * so fp8 artifacts can be resharded or consumed by bf16 engines (resharding
 * into other layouts, Sec. 2.1; rank-specific transform_into, Sec. 7):
 *   y = RN_bf16(RN_f32(E4M3value(q) * s)), s the scale of q's 128x128 tile;
 *   a NaN product (code 0x7F/0xFF, NaN scale, 0 * Inf) gives 0x7FC0.
 * ------------------------------------------------------------------------ */
typedef struct {
  uint64_t src_off;   /* bytes from the code base to code [0][0] */
  int64_t rows, cols; /* matrix shape (elements) */
  int64_t src_ld;     /* bytes between code rows (>= cols) */
  uint64_t dst_off;   /* bf16 elements from dst_base to element [0][0] */
  int64_t dst_ld;     /* bf16 elements between destination rows (>= cols) */
  uint64_t scale_off; /* floats from scale_base to scale [0][0] */
  int64_t scale_ld;   /* floats between rows of the scale grid (>= ceil(cols/128)) */
} tc_dequant_item;

/* Bytes of device workspace tc_dequant_fp8_blockscaled needs for n items. */
size_t tc_dequant_fp8_workspace(int64_t n_items);
/* The same with room for the per-tile table, as tc_cast_fp8_workspace_tiles. */
size_t tc_dequant_fp8_workspace_tiles(const tc_dequant_item* items /* host */, int64_t n_items);

/* Dequantize every item.  items: HOST array, written into the workspace
 * like the cast's.  The bf16 destinations must not overlap one another or the
 * sources.  tile must be 128.  This is tc_dequant_fp8_prepare followed by
 * tc_dequant_fp8_planned, the same split as the cast's (the plan's input
 * base is the codes', its output base the bf16 destination's). */
tc_status tc_dequant_fp8_blockscaled(const void* codes_base, const float* scale_base,
                                     void* dst_base, const tc_dequant_item* items /* host */,
                                     int64_t n_items, int32_t tile, void* workspace,
                                     size_t workspace_bytes, hipStream_t stream);
tc_status tc_dequant_fp8_prepare(const void* codes_base, const void* dst_base,
                                 const tc_dequant_item* items /* host */, int64_t n_items,
                                 int32_t tile, void* workspace, size_t workspace_bytes,
                                 tc_tile_plan* plan /* host, out */, hipStream_t stream);
tc_status tc_dequant_fp8_planned(const void* codes_base, const float* scale_base, void* dst_base,
                                 const void* workspace, size_t workspace_bytes,
                                 const tc_tile_plan* plan /* host */, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Host <-> device staging: the materialization pipeline's pinned streaming
 * buffers and asynchronous copy streams (Sec. 5; the same mechanism serves
 * the parallel read streams of weight loading, Sec. 6.2), for bytes that live
 * in host memory -- a transfer buffer kept in host DRAM, or a host-memory
 * tier.
 *
 * A stager is bound to the device current when it is created.  It owns
 * `slots` pinned host buffers of `slot_bytes` each (hipHostMalloc), a copy
 * stream of default priority, and `host_threads` host threads (counting the
 * caller) that copy between pageable memory and the pinned slots.  Zero
 * selects the defaults: 32 MiB slots, 4 slots, 4 threads.  Pageable bytes
 * travel in slot-sized chunks: while the DMA engine moves chunk k over PCIe,
 * the host threads copy chunk k + 1 and the device scatters or gathers the
 * chunk before.  With TC_HOST_PINNED the caller's host buffer is itself
 * pinned (hipHostMalloc) and the DMA reads or writes it directly.
 *
 * One call at a time per stager (an internal lock serializes callers).  The
 * stager allocates no device memory: device staging is the caller's
 * dev_stage buffer, cut into up to 8 slots of whole ids.
 *
 * Ordering: each call starts after the work already enqueued on `stream`;
 * device results are ordered before later work on `stream`.
 *   tc_stage_h2d / tc_hydrate_from_host return once the host source may be
 *     reused (every host copy out of it has finished) -- except with
 *     TC_HOST_PINNED, where the source must stay unchanged until `stream`
 *     has passed the call (as for hipMemcpyAsync).
 *   tc_stage_d2h / tc_publish_to_host return when host_dst holds the bytes.
 *
 * tc_hydrate_from_host: host_src holds n * num_regions * block_bytes bytes in
 *   the layout tc_gather_blocks writes (id-major, then region); the blocks
 *   are scattered into the pool exactly as tc_scatter_blocks would (ids
 *   distinct).  tc_publish_to_host is the inverse: the pool's blocks of ids,
 *   gathered, land in host_dst.
 *
 * Errors: TC_ERR_INVALID_ARGUMENT for null pointers with work to do, unknown
 * flags, a bad pool, a call from another device than the stager's;
 * TC_ERR_WORKSPACE if one id's blocks (num_regions * block_bytes) exceed a
 * slot or dev_stage cannot hold one chunk; validation-mode errors as for the
 * block calls, checked over the whole id list.
 * ------------------------------------------------------------------------ */
#define TC_HOST_PINNED 1
typedef struct tc_stager tc_stager;
tc_status tc_stager_create(size_t slot_bytes, int32_t slots, int32_t host_threads,
                           tc_stager** out);
/* Waits for the stager's copies, then frees everything it owns.  No other
 * thread may be inside a call on this stager (its lock is freed too). */
tc_status tc_stager_destroy(tc_stager* stager);
/* host_src (bytes) -> dev_dst (bytes). */
tc_status tc_stage_h2d(tc_stager* stager, const void* host_src, void* dev_dst, size_t bytes,
                       int32_t flags, hipStream_t stream);
/* dev_src (bytes) -> host_dst (bytes); blocks until host_dst is complete. */
tc_status tc_stage_d2h(tc_stager* stager, const void* dev_src, void* host_dst, size_t bytes,
                       int32_t flags, hipStream_t stream);
tc_status tc_hydrate_from_host(tc_stager* stager, const tc_block_pool* pool, const int32_t* ids,
                               int64_t n, const void* host_src, int32_t flags, void* dev_stage,
                               size_t dev_stage_bytes, hipStream_t stream);
tc_status tc_publish_to_host(tc_stager* stager, const tc_block_pool* pool, const int32_t* ids,
                             int64_t n, void* host_dst, int32_t flags, void* dev_stage,
                             size_t dev_stage_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Same-host zero-copy sharing between processes (HIP IPC): the Unified
 * Tensor Pool exposes device tensors of co-hosted instances to one another
 * without copies (Sec. 4.2, Sec. 5), and a warm start consumes
 * pre-materialized weights that way (Sec. 6.1).  Every call above accepts
 * an imported address like any other device pointer, so an engine can, for
 * example, gather KV blocks straight out of another process's pool.
 *
 * tc_ipc_export: a handle for the device range [dev_ptr, dev_ptr + bytes),
 *   which must lie inside one allocation of this process (IPC shares whole
 *   allocations; the handle records the range's offset in it).  The handle
 *   is plain bytes: send it to another process on this host by any channel.
 *   The exporter must keep the allocation alive while importers use it.
 *   TC_ERR_INVALID_ARGUMENT for null arguments, memory that is not a device
 *   allocation of this process, and allocations of 2 GiB or more (opening a
 *   handle to such an allocation has been seen not to return on some ROCm
 *   drivers); TC_ERR_OUT_OF_RANGE for a range that leaves its allocation.
 * tc_ipc_open: maps the exporter's allocation on the current device and
 *   returns the range's address in this process in *dev_ptr.  A process may
 *   open a given handle once at a time.
 * tc_ipc_close: unmaps it (dev_ptr as returned by tc_ipc_open).  The
 *   exporter's memory is unaffected.
 * Runtime failures are TC_ERR_HIP (tc_last_hip_error() gives the code).
 * These calls are synchronous host calls; they enqueue nothing.
 * ------------------------------------------------------------------------ */
typedef struct {
  uint8_t handle[64];   /* the runtime's IPC handle of the allocation */
  uint64_t offset;      /* bytes from the allocation's base to the range */
  uint64_t bytes;       /* length of the range */
  uint64_t alloc_bytes; /* size of the allocation */
} tc_ipc_handle;
tc_status tc_ipc_export(const void* dev_ptr, size_t bytes, tc_ipc_handle* out /* host */);
tc_status tc_ipc_open(const tc_ipc_handle* handle /* host */, void** dev_ptr /* host, out */);
tc_status tc_ipc_close(const tc_ipc_handle* handle /* host */, void* dev_ptr);

/* ------------------------------------------------------------------------ */
const char* tc_status_string(tc_status status);
/* hipError_t of the most recent TC_ERR_HIP on the calling thread. */
int tc_last_hip_error(void);
/* 1: validate descriptors (synchronous, for debugging); 0: off. */
void tc_set_validate(int on);
int tc_get_validate(void);

#ifdef __cplusplus
}
#endif
#endif /* TENSORCAST_HIP_H */
