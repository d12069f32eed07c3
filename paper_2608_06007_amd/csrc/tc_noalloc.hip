// The block-scaled fp8 cast for callers that cannot allocate: the same
// kernels as tc_cast_fp8_blockscaled, with the tile table in a fixed array
// of device memory owned by the library instead of a caller workspace.
//
// `scratch` is a file-scope device array.  In host code its name is only a
// host-side stand-in, so the device address is looked up once per device
// with hipGetSymbolAddress (with that device current) and kept; every launch
// takes the address on the device of its stream.  Each device holds its own
// copy until the process ends.  Calls on one device share it: the table is
// rewritten by every call, so two calls that overlap in time on one device
// race.
#include <mutex>

#include "tc_device.h"


namespace tc {
namespace {

// cast_workspace_bytes(TC_NOALLOC_MAX_ITEMS): 4096 items of 64 bytes, two
// prefixes of 4097 words and 4096 flags, each part 256-byte aligned.
constexpr size_t kScratchBytes = 332288;
static_assert(TC_NOALLOC_MAX_ITEMS == 4096, "kScratchBytes holds the table of 4096 items");

static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];  // device address of `scratch` on each device (null: not yet)

// The address of `scratch` on the device that runs `stream` (the current
// device for the null stream), looked up with that device current on its
// first use there.
hipError_t scratch_for_stream(hipStream_t stream, void** out) {
  int dev = 0;
  hipError_t e = stream ? hipStreamGetDevice(stream, &dev) : hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    int cur = 0;
    e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev) {
      const hipError_t back = hipSetDevice(cur);
      if (e == hipSuccess) e = back;
    }
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace
}  // namespace tc

extern "C" tc_status tc_cast_fp8_blockscaled_noalloc(const void* src_base, void* dst_base,
                                                     float* scale_base, const tc_cast_item* items,
                                                     int64_t n_items, int32_t tile,
                                                     hipStream_t stream) {
  if (n_items < 0 || tile != 128) return TC_ERR_INVALID_ARGUMENT;
  if (n_items == 0) return TC_OK;
  if (n_items > TC_NOALLOC_MAX_ITEMS) return TC_ERR_WORKSPACE;
  if (tc::cast_workspace_bytes(TC_NOALLOC_MAX_ITEMS) > tc::kScratchBytes) return TC_ERR_WORKSPACE;
  void* ws = nullptr;
  hipError_t e = tc::scratch_for_stream(stream, &ws);
  if (e != hipSuccess) return tc::hip_status(e);
  tc_tile_plan plan;
  tc_status st = tc_cast_fp8_prepare(src_base, dst_base, items, n_items, tile, ws, tc::kScratchBytes,
                                     &plan, stream);
  if (st != TC_OK) return st;
  return tc_cast_fp8_planned(src_base, dst_base, scale_base, ws, tc::kScratchBytes, &plan, stream);
}
