// Internal declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tensorcast_hip.h"

namespace tc {

// Fragment plans cut fragments into tasks of at most `piece` bytes, one task
// per wave (64 lanes x 16 B = 1 KiB per pass); the piece is the smallest
// power of two >= kMinPiece that keeps the task table within the workspace,
// at most kMaxPiece.
constexpr uint64_t kMinPiece = 1024;
constexpr uint64_t kMaxPiece = uint64_t(1) << 30;
// Descriptors handled by one workgroup of the planning kernels.
constexpr int kPlanPerBlock = 1024;

struct RegionTable {
  uint64_t base[TC_MAX_REGIONS];
};

// One task of a fragment plan, a byte run of at most `piece` bytes, packed in
// 16 bytes: src_off (48 bits) | dst_off (48 bits) | len (31 bits) | a flag
// set on the first task of each fragment.  Offsets must stay below 2^48
// (256 TiB).
struct Task {
  uint64_t lo;  // src_off | dst_off << 48
  uint64_t hi;  // dst_off >> 16 | len << 32 | first << 63
};
constexpr uint64_t kOffsetLimit = uint64_t(1) << 48;
constexpr uint64_t kTaskFirst = uint64_t(1) << 63;
__host__ __device__ inline uint64_t task_src(const Task& t) { return t.lo & (kOffsetLimit - 1); }
__host__ __device__ inline uint64_t task_dst(const Task& t) {
  return (t.lo >> 48) | ((t.hi & 0xFFFFFFFFu) << 16);
}
__host__ __device__ inline uint64_t task_len(const Task& t) { return (t.hi >> 32) & 0x7FFFFFFFu; }

// Header at the start of a fragment-plan workspace.
struct PlanHeader {
  uint64_t total_tasks;    // written by the planning kernels
  uint64_t piece;          // task size chosen for this plan
  uint64_t payload;        // sum of the fragment lengths
  uint64_t n;              // number of fragments planned
  uint64_t capacity;       // task-table entries that fit the workspace
  uint64_t dst_unordered;  // some fragment starts below its predecessor (destination side)
  uint64_t dst_end;        // largest dst_off + len of a non-empty fragment
  uint64_t permuted;       // the tasks follow the reordered list; perm maps back
  uint64_t cut;            // 127: tasks after a fragment's first start on a 128-byte
                           // destination line; 0: tasks start at multiples of the piece
  uint64_t out_of_range;   // some non-empty fragment ends past 2^48 (source or destination):
                           // its tasks could not hold the offsets, so nothing is planned
  uint64_t status;         // tc_status of the plan: TC_OK, TC_ERR_OUT_OF_RANGE (offsets past
                           // 2^48), TC_ERR_WORKSPACE (the tasks do not fit), or
                           // TC_ERR_INVALID_ARGUMENT (more than 2^33 tasks); total_tasks is 0
                           // unless TC_OK
  uint64_t recount;        // 1 KiB pieces overflowed the workspace: counted again with `piece`
  uint64_t shift;          // bucket size (log2 bytes) of a destination-ordered plan
};
// The planning kernels decide everything on the device (piece, reordering,
// status), so planning never waits for the host.  A copy launched with this
// task count reads the count from the plan's header on the device.
constexpr uint64_t kTasksFromPlan = ~uint64_t(0);

// Workspace layout: header | tasks[capacity] | digest slots[capacity] |
// windows[ceil(capacity / 1024)] | ... | tstart[n + 1] | block sums |
// [reordered fragments | perm | buckets].  The task table sits at a fixed
// offset so a copy needs only the workspace base; windows[j] holds the first
// and last fragment of tasks [1024 j, 1024 (j + 1)), written by the plan's
// expansion.  The planning scratch lives at the end and stays valid with the
// plan (the digest reduction reads tstart, windows and perm).
constexpr size_t kTasksOffset = 256;
static_assert(sizeof(PlanHeader) <= kTasksOffset, "the header fits before the task table");
constexpr size_t kTaskBytes = 32;  // a task and its 16-byte digest slot
constexpr uint64_t kWindowTasks = 1024;  // tasks per window of the expansion and the reduction
constexpr size_t kWindowBytes = 16;      // first and last fragment of a window
// Lists of at least this many fragments whose destinations are not in
// ascending order are planned in destination order (bucketed by address).
constexpr int64_t kReorderMin = 4096;
struct PlanLayout {
  size_t tstart, blocks, capacity, slots, windows;
  size_t sorted, perm, buckets, bucket_sums;  // valid when nbuckets > 0
  uint64_t nbuckets;                          // bucket capacity (0: no reordering)
};
PlanLayout plan_layout(int64_t n, size_t ws_bytes);
size_t frag_workspace_bytes(int64_t n);
size_t frag_workspace_min_bytes(int64_t n);

// TC_OK for hipSuccess; otherwise records the error for tc_last_hip_error()
// and returns TC_ERR_HIP.
tc_status hip_status(hipError_t e);

// A block pool the movers accept: 1..TC_MAX_REGIONS non-null regions, at
// least one block, stride >= block bytes, and byte extents (a region's
// blocks x stride, one id's regions x block bytes) within 63 bits.
bool pool_valid(const tc_block_pool* p);

// --- block gather / scatter --------------------------------------------
hipError_t launch_blocks(const RegionTable& tab, int32_t num_regions, int64_t block_bytes,
                         int64_t block_stride, const int32_t* ids, int64_t n, uint8_t* buf,
                         bool gather, bool aligned, hipStream_t s);

// --- fragments ---------------------------------------------------------
// Enqueue the whole plan of n fragments into the workspace (header, task
// table, windows, tstart; for long unordered lists the destination-ordered
// copy of the list and its permutation).  Every decision -- piece size,
// reordering, status -- is taken on the device; nothing waits for the host.
hipError_t launch_plan(const tc_fragment* frags, int64_t n, void* ws, const PlanLayout& L,
                       hipStream_t s);
// Copy with a plan.  total_tasks is the plan's count, or kTasksFromPlan: the
// kernel then reads it from the header and a bounded grid strides over the
// tasks (cap_tasks bounds the count, from the workspace size).
hipError_t launch_copy_tasks(const uint8_t* src, uint8_t* dst, const void* ws,
                             uint64_t total_tasks, uint64_t cap_tasks, hipStream_t s);
// Copy (mode 0) or only read (1: at the tasks' source offsets, 2: at their
// destination offsets) with a plan, and write each fragment's digest pair
// into digests[2n]: zero fill, per-task sums into the digest slots, then a
// reduction per fragment.  `src` is the buffer read in every mode.
hipError_t launch_copy_digest(const uint8_t* src, uint8_t* dst, void* ws, const PlanLayout& L,
                              int64_t n, uint64_t total, int mode, uint64_t* digests,
                              hipStream_t s);

// --- fp8 cast ----------------------------------------------------------
// Workspace: items | prefix of full (vector-path) tiles | prefix of the other
// tiles | per-item vector-path flag.  Byte offsets:
struct CastLayout {
  size_t items, full_prefix, edge_prefix, aligned, bytes;
};
CastLayout cast_layout(int64_t n_items);
size_t cast_workspace_bytes(int64_t n_items);
// A chunk of the tile table, passed by value as a kernel argument (3.3 KB,
// below the 4 KiB of kernel arguments a launch may carry).
constexpr int kTableChunkItems = 40;
constexpr int kItemWords = 8;  // a cast or inverse-cast item is eight 64-bit words
struct TableChunk {
  uint64_t words[kTableChunkItems * kItemWords];
  uint64_t fprefix[kTableChunkItems];
  uint64_t eprefix[kTableChunkItems];
  uint64_t first;            // index of the chunk's first item
  uint64_t ftotal, etotal;   // the table's totals, written after the last chunk
  uint32_t count;            // items in the chunk
  uint32_t last;             // 1 for the last chunk
  uint8_t aligned[kTableChunkItems];
};
static_assert(sizeof(TableChunk) <= 3584, "a chunk fits the kernel arguments");
// Enqueue the writes of one chunk of a table of n_items items into the
// workspace (the table's layout is cast_layout(n_items)).
hipError_t launch_tile_chunk(const TableChunk& c, int64_t n_items, void* ws, hipStream_t s);
// Optional per-tile table after the item table (at cast_layout(n).bytes):
// one entry per full tile, so that a workgroup finds its tile's rows with a
// single load instead of searching the items and dividing for the tile's
// row and column.  Offsets are in elements of each side (bf16 elements or
// code bytes); lds packs src_ld | dst_ld << 32 (both below 2^32).
struct TileEntry {
  uint64_t in_off, out_off, scale_idx, lds;
};
static_assert(sizeof(TileEntry) == 32, "tile entries are 32 bytes");
constexpr size_t kTileEntryBytes = sizeof(TileEntry);
// Fill the per-tile table of the full tiles from the item table already
// enqueued in the workspace (one thread per tile).
hipError_t launch_tile_expand(void* ws, int64_t n_items, uint64_t full_tiles, hipStream_t s);
// tiled: the workspace holds the per-tile table (full tiles read it).
hipError_t launch_cast_blockscaled(const uint16_t* src, uint8_t* dst, float* scales,
                                   const void* ws, int64_t n_items, uint64_t full_tiles,
                                   uint64_t edge_tiles, bool tiled, hipStream_t s);
hipError_t launch_cast_scaled(const uint16_t* src, int64_t n, float scale, uint8_t* dst,
                              hipStream_t s);
// The inverse cast uses the same workspace layout (its items are the same
// size as cast items).
hipError_t launch_dequant_blockscaled(const uint8_t* codes, const float* scales, uint16_t* dst,
                                      const void* ws, int64_t n_items, uint64_t full_tiles,
                                      uint64_t edge_tiles, bool tiled, hipStream_t s);

}  // namespace tc
