// Internal declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tensorcast_hip.h"

namespace tc {

// Fragments are cut into pieces of at most this many bytes; a wave copies
// one piece at a time.
constexpr uint64_t kPieceBytes = 16 * 1024;
// Tasks (pieces) a wave takes per visit of the plan.
constexpr int kTasksPerChunk = 8;
// Descriptors summed by one workgroup of the planning kernels.
constexpr int kPlanPerBlock = 1024;

struct RegionTable {
  uint64_t base[TC_MAX_REGIONS];
};

// Launch geometry of the current device.
struct DeviceInfo {
  int device;
  int cus;
};
hipError_t device_info(DeviceInfo* out);

// --- block gather / scatter --------------------------------------------
hipError_t launch_blocks(const RegionTable& tab, int32_t num_regions, int64_t block_bytes,
                         int64_t block_stride, const int32_t* ids, int64_t n, uint8_t* buf,
                         bool gather, bool aligned, hipStream_t s);

// --- fragments ---------------------------------------------------------
// Workspace layout (bytes): [0, 8*(n+1))       tstart: first task of each fragment, tstart[n] = total
//                            [.., + 8*nblocks)  per-block task sums, then their exclusive prefix
size_t frag_workspace_bytes(int64_t n);
hipError_t launch_plan_fragments(const tc_fragment* frags, int64_t n, void* ws, hipStream_t s);
hipError_t launch_copy_planned(const uint8_t* src, uint8_t* dst, const tc_fragment* frags,
                               int64_t n, const void* ws, const DeviceInfo& di, hipStream_t s);

// --- fp8 cast ----------------------------------------------------------
size_t cast_workspace_bytes(int64_t n_items);
hipError_t launch_cast_blockscaled(const uint16_t* src, uint8_t* dst, float* scales,
                                   const tc_cast_item* items, int64_t n_items, void* ws,
                                   const DeviceInfo& di, hipStream_t s);
hipError_t launch_cast_scaled(const uint16_t* src, int64_t n, float scale, uint8_t* dst,
                              hipStream_t s);

}  // namespace tc
