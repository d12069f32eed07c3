// Same-host zero-copy sharing of device tensors between processes through
// HIP IPC: the paper's Unified Tensor Pool exposes tensors of co-hosted
// instances to one another without copies (Sec. 4.2, Sec. 5), and a warm
// start consumes pre-materialized weights that way (Sec. 6.1).
//
// A handle names the allocation that holds the exported range (IPC works on
// whole allocations) plus the range's offset and length in it.  The
// importer maps that allocation and gets the range's address in its own
// address space; the bytes are the exporter's, read and written in place.
#include <hip/hip_runtime.h>

#include <cstring>

#include "tc_internal.h"

static_assert(sizeof(hipIpcMemHandle_t) == sizeof(((tc_ipc_handle*)nullptr)->handle),
              "the handle carries the runtime's IPC handle verbatim");

namespace {
// On some ROCm drivers, opening a handle to an allocation of 2 GiB or more
// has been seen not to return; exports are limited to smaller allocations.
constexpr size_t kMaxIpcAllocation = (size_t(1) << 31) - 1;
}  // namespace

extern "C" {

tc_status tc_ipc_export(const void* dev_ptr, size_t bytes, tc_ipc_handle* out) {
  if (!dev_ptr || !out) return TC_ERR_INVALID_ARGUMENT;
  std::memset(out, 0, sizeof(*out));
  hipDeviceptr_t base = nullptr;
  size_t size = 0;
  hipError_t e = hipMemGetAddressRange(&base, &size, const_cast<void*>(dev_ptr));
  if (e != hipSuccess) {
    (void)hipGetLastError();  // not device memory of this process: not a sticky error
    return TC_ERR_INVALID_ARGUMENT;
  }
  const uintptr_t b = reinterpret_cast<uintptr_t>(base), p = reinterpret_cast<uintptr_t>(dev_ptr);
  if (p < b || p - b > size || bytes > size - (p - b)) return TC_ERR_OUT_OF_RANGE;
  if (size > kMaxIpcAllocation) return TC_ERR_INVALID_ARGUMENT;
  hipIpcMemHandle_t h;
  e = hipIpcGetMemHandle(&h, base);
  if (e != hipSuccess) return tc::hip_status(e);
  std::memcpy(out->handle, &h, sizeof(h));
  out->offset = uint64_t(p - b);
  out->bytes = uint64_t(bytes);
  out->alloc_bytes = uint64_t(size);
  return TC_OK;
}

tc_status tc_ipc_open(const tc_ipc_handle* handle, void** dev_ptr) {
  if (!handle || !dev_ptr) return TC_ERR_INVALID_ARGUMENT;
  *dev_ptr = nullptr;
  if (handle->alloc_bytes > kMaxIpcAllocation || handle->offset > handle->alloc_bytes ||
      handle->bytes > handle->alloc_bytes - handle->offset)
    return TC_ERR_INVALID_ARGUMENT;
  hipIpcMemHandle_t h;
  std::memcpy(&h, handle->handle, sizeof(h));
  void* base = nullptr;
  hipError_t e = hipIpcOpenMemHandle(&base, h, hipIpcMemLazyEnablePeerAccess);
  if (e != hipSuccess) return tc::hip_status(e);
  *dev_ptr = static_cast<uint8_t*>(base) + handle->offset;
  return TC_OK;
}

tc_status tc_ipc_close(const tc_ipc_handle* handle, void* dev_ptr) {
  if (!handle || !dev_ptr || reinterpret_cast<uintptr_t>(dev_ptr) < handle->offset)
    return TC_ERR_INVALID_ARGUMENT;
  return tc::hip_status(hipIpcCloseMemHandle(static_cast<uint8_t*>(dev_ptr) - handle->offset));
}

}  // extern "C"
