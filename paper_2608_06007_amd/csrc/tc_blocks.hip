// Paged-KV block gather and scatter for gfx950: the device half of publish
// (export a request's blocks into one contiguous transfer buffer) and
// hydrate (import them into another engine's pool).
#include "tc_device.h"

namespace tc {
namespace {

// ------------------------------------------------------------------------
// Block gather / scatter: work item w = 4 KiB tile k of chunk c = i*R + r
// (id i, region r).  One workgroup per tile; grid-stride only when the grid
// is capped.
// ------------------------------------------------------------------------
template <bool kGather>
__global__ __launch_bounds__(kThreads) void k_blocks_vec(const RegionTable tab, const int32_t R,
                                                        const int64_t B, const int64_t stride,
                                                        const int32_t* __restrict__ ids,
                                                        const uint64_t total_tiles,
                                                        const uint64_t tiles_per_chunk,
                                                        uint8_t* __restrict__ buf) {
  for (uint64_t b = blockIdx.x; b < total_tiles; b += gridDim.x) {
    const uint64_t w = xcd_grouped(b, total_tiles, kGather ? kXcdGroupGather : kXcdGroupScatter);
    const uint64_t c = w / tiles_per_chunk;
    const uint64_t k = w - c * tiles_per_chunk;
    const uint64_t i = c / uint64_t(R);
    const int32_t r = (int32_t)(c - i * uint64_t(R));
    uint8_t* pool = reinterpret_cast<uint8_t*>(tab.base[r]) + int64_t(ids[i]) * stride;
    uint8_t* xfer = buf + c * uint64_t(B);
    const int64_t off = int64_t(k) * kTileBytes + int64_t(threadIdx.x) * 16;
    if (off < B) {
      if (kGather)
        st_sc1(reinterpret_cast<u32x4*>(xfer + off), ld_nt_global(pool + off));
      else
        st_sc1_nt(reinterpret_cast<u32x4*>(pool + off), ld_nt(reinterpret_cast<const u32x4*>(xfer + off)));
    }
  }
}

// Pools whose bases, stride or block size are not 16-byte multiples: one
// workgroup per (id, region) chunk, its waves taking 1 KiB runs in turn, each
// copied at vector width whatever the alignment of its two ends.
template <bool kGather>
__global__ __launch_bounds__(kThreads) void k_blocks_bytes(const RegionTable tab, const int32_t R,
                                                          const int64_t B, const int64_t stride,
                                                          const int32_t* __restrict__ ids,
                                                          const uint64_t n_chunks,
                                                          uint8_t* __restrict__ buf) {
  const int lane = threadIdx.x & (kWaveLanes - 1);
  const int64_t w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  constexpr int64_t kRun = int64_t(kWaveLanes) * 16;
  for (uint64_t c = blockIdx.x; c < n_chunks; c += gridDim.x) {
    const uint64_t i = c / uint64_t(R);
    const int32_t r = (int32_t)(c - i * uint64_t(R));
    uint8_t* pool = reinterpret_cast<uint8_t*>(tab.base[r]) + int64_t(ids[i]) * stride;
    uint8_t* xfer = buf + c * uint64_t(B);
    const uint8_t* from = kGather ? pool : xfer;
    uint8_t* to = kGather ? xfer : pool;
    for (int64_t o = w * kRun; o < B; o += (kThreads / kWaveLanes) * kRun) {
      const uint64_t n = uint64_t(B - o < kRun ? B - o : kRun);
      if (kGather)
        wave_copy_any(from + o, to + o, n, lane, [](u32x4* p, u32x4 v) { st_sc1(p, v); });
      else
        wave_copy_any(from + o, to + o, n, lane, [](u32x4* p, u32x4 v) { st_sc1_nt(p, v); });
    }
  }
}

}  // namespace

hipError_t launch_blocks(const RegionTable& tab, int32_t R, int64_t B, int64_t stride,
                         const int32_t* ids, int64_t n, uint8_t* buf, bool gather, bool aligned,
                         hipStream_t s) {
  const uint64_t chunks = uint64_t(n) * uint64_t(R);
  if (aligned) {
    const uint64_t tpc = (uint64_t(B) + kTileBytes - 1) / kTileBytes;
    const uint64_t total = chunks * tpc;
    if (gather)
      hipLaunchKernelGGL(k_blocks_vec<true>, dim3(grid_for(total)), dim3(kThreads), 0, s, tab, R,
                         B, stride, ids, total, tpc, buf);
    else
      hipLaunchKernelGGL(k_blocks_vec<false>, dim3(grid_for(total)), dim3(kThreads), 0, s, tab, R,
                         B, stride, ids, total, tpc, buf);
  } else {
    if (gather)
      hipLaunchKernelGGL(k_blocks_bytes<true>, dim3(grid_for(chunks)), dim3(kThreads), 0, s, tab,
                         R, B, stride, ids, chunks, buf);
    else
      hipLaunchKernelGGL(k_blocks_bytes<false>, dim3(grid_for(chunks)), dim3(kThreads), 0, s, tab,
                         R, B, stride, ids, chunks, buf);
  }
  return hipGetLastError();
}

}  // namespace tc
