// Device helpers shared by the byte movers on gfx950: the paged-KV block
// moves (tc_blocks.hip), fragment plans (tc_plan.hip) and planned copies
// with their digests (tc_copy.hip).
//
// Design (measured on MI355X): the copies are HBM-bound, and the launch
// shape that streams best is a one-shot grid of small workgroups -- 256
// lanes, one 16-byte vector each, 4 KiB per workgroup -- with non-temporal
// loads and stores (the data is touched once) and a workgroup order that
// gives each XCD runs of consecutive tiles.  Workgroups are dealt to the 8
// XCDs round-robin by block index; without the regrouping every 32 KiB block
// would be split across all eight L2s and address translators.
#pragma once

#include "tc_internal.h"

namespace tc {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;  // 4 waves of 64 lanes
constexpr int kWaveLanes = 64;
constexpr int64_t kTileBytes = int64_t(kThreads) * 16;  // 4 KiB per workgroup
constexpr int kXcds = 8;
constexpr uint64_t kXcdGroup = 64;           // consecutive tiles per XCD run
constexpr uint64_t kXcdGroupScatter = 512;   // hydrate: longer runs stream its reads better
constexpr uint64_t kXcdGroupReordered = 256;  // task copies of destination-ordered plans

// Work item of block b when the 8 XCDs each take runs of G consecutive items
// (a bijection on [0, N); the last partial round keeps the identity order).
__device__ __forceinline__ uint64_t xcd_grouped(uint64_t b, uint64_t N, uint64_t G) {
  const uint64_t round = uint64_t(kXcds) * G;
  const uint64_t full = (N / round) * round;
  if (b >= full) return b;
  const uint64_t x = b % kXcds, l = b / kXcds;
  return (l / G) * round + x * G + (l % G);
}

__device__ __forceinline__ u32x4 ld_nt(const u32x4* p) { return __builtin_nontemporal_load(p); }
// The same load through a global-address-space pointer, for addresses the
// compiler cannot prove global (pool bases passed as integers): a global
// rather than a flat load.
typedef const u32x4 __attribute__((address_space(1))) global_u32x4;
__device__ __forceinline__ u32x4 ld_nt_global(const void* p) {
  return __builtin_nontemporal_load((global_u32x4*)p);
}
// Vector stores with the SC1 scope bit, alone (gather's contiguous output) or
// with NT (hydrate's scattered blocks, planned copies of ordered lists):
// measured +1-4% over plain non-temporal stores on those streams.  Plans
// built from unordered destination lists (small fragments with scattered
// sources, copied in destination order) store with plain NT: +8% there.
__device__ __forceinline__ void st_nt(u32x4* p, u32x4 v) { __builtin_nontemporal_store(v, p); }
//
// A store of more than 8 bytes reads its data registers after issue: a VALU
// write to them needs 2 wait states on this GPU.  The compiler inserts them
// for its own stores but cannot see into inline asm, so each asm store ends
// with s_nop 1 (2 wait states) before any later instruction of the wave.
__device__ __forceinline__ void st_sc1(u32x4* p, u32x4 v) {
  asm volatile("global_store_dwordx4 %0, %1, off sc1\n\ts_nop 1" ::"v"(p), "v"(v) : "memory");
}
__device__ __forceinline__ void st_sc1_nt(u32x4* p, u32x4 v) {
  asm volatile("global_store_dwordx4 %0, %1, off sc1 nt\n\ts_nop 1" ::"v"(p), "v"(v) : "memory");
}
// The planned copies' store: plain NT for a reordered plan, SC1 NT otherwise
// (plain is wave-uniform, read from the plan header).
__device__ __forceinline__ void st_task(u32x4* p, u32x4 v, bool plain) {
  if (plain)
    st_nt(p, v);
  else
    st_sc1_nt(p, v);
}

namespace {
// p[0 .. n) = 0: a fill kernel rather than hipMemsetAsync, so the calls that
// clear memory can be captured into a graph (digests with no task to run,
// the reorder's bucket counters).
[[maybe_unused]] __global__ __launch_bounds__(kThreads) void k_fill_zero(uint64_t* __restrict__ p,
                                                                         const uint64_t n) {
  for (uint64_t i = uint64_t(blockIdx.x) * kThreads + threadIdx.x; i < n;
       i += uint64_t(gridDim.x) * kThreads)
    p[i] = 0;
}
}  // namespace

// Tasks that one workgroup expands, and reduces: one window of the plan.
constexpr int kExpandPerBlock = int(kWindowTasks);

// Largest grid used for one launch; bigger jobs loop (grid-stride).
constexpr uint64_t kMaxGrid = uint64_t(1) << 24;

inline unsigned grid_for(uint64_t items) { return (unsigned)(items < kMaxGrid ? items : kMaxGrid); }

}  // namespace tc
