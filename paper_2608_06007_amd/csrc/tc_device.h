// Device helpers shared by the kernels for gfx950: the paged-KV block moves
// (tc_blocks.hip), fragment plans (tc_plan.hip), planned copies with their
// digests (tc_copy.hip), and the block-scaled cast and its inverse
// (tc_cast.hip, tc_dequant.hip).
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
constexpr uint64_t kXcdGroup = 64;           // consecutive tiles per XCD run (task copies)
// publish (block gather): runs of 256 tiles.  In publish + hydrate steps
// (each gather after a hydrate, as a serving engine and the benchmark run
// them) the 8 GiB batch gathers at 6672-6687 GB/s with runs of 256 against
// 6293-6406 with runs of 32 (two GPUs; 128: 6619-6662, 512: 6637-6645).
// Gathers back to back barely tell them apart (32: 6731-6749, 256:
// 6759-6768), and on distinct single requests runs of 256 are 1% slower.
constexpr uint64_t kXcdGroupGather = 256;
// hydrate: longer runs stream its contiguous reads better.  Runs of 128 /
// 512 / 2048 / 8192 tiles on the 8 GiB batch, one GPU: 6307 / 6372 / 6413 /
// 6399 GB/s; on distinct single requests 2048 is within 1% of 512.
constexpr uint64_t kXcdGroupScatter = 2048;
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

// Item whose tile range contains tile t: the last i in [0, n) with
// prefix[i] <= t, given prefix[0] <= t < prefix[n] (the cast and its inverse
// number their tiles by item).  Each round cuts the range into 64 steps and
// counts by ballot the step starts at or below t, so a wave needs
// ceil(log64 n) rounds.
__device__ inline int64_t find_item(const uint64_t* __restrict__ prefix, int64_t n, uint64_t t,
                                    int lane) {
  int64_t lo = 0, hi = n;
  while (hi - lo > 1) {
    const int64_t step = (hi - lo + kWaveLanes - 1) / kWaveLanes;
    const int64_t p = lo + (int64_t(lane) + 1) * step;
    const bool pred = lane < kWaveLanes - 1 && p < hi && prefix[p] <= t;
    lo += int64_t(__popcll(__ballot(pred))) * step;
    hi = min(hi, lo + step);
  }
  return lo;
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

// The 16 bytes that start r bytes (1..15) into the aligned vector a and run
// on into the next aligned vector b: bytes r .. r + 15 of a || b.  r is
// wave-uniform (one fragment per wave), so the word selection is a uniform
// branch, and each output word is one v_alignbyte_b32 of two neighbours.
__device__ __forceinline__ u32x4 realign(const u32x4 a, const u32x4 b, const uint32_t r) {
  const uint32_t sh = r & 3;
  uint32_t x0, x1, x2, x3, x4;
  switch (r >> 2) {
    case 0: x0 = a.x; x1 = a.y; x2 = a.z; x3 = a.w; x4 = b.x; break;
    case 1: x0 = a.y; x1 = a.z; x2 = a.w; x3 = b.x; x4 = b.y; break;
    case 2: x0 = a.z; x1 = a.w; x2 = b.x; x3 = b.y; x4 = b.z; break;
    default: x0 = a.w; x1 = b.x; x2 = b.y; x3 = b.z; x4 = b.w; break;
  }
  return u32x4{__builtin_amdgcn_alignbyte(x1, x0, sh), __builtin_amdgcn_alignbyte(x2, x1, sh),
               __builtin_amdgcn_alignbyte(x3, x2, sh), __builtin_amdgcn_alignbyte(x4, x3, sh)};
}

// One wave copies len bytes from s to d whatever their alignment: bytes up
// to d's 16-byte alignment, then 16-byte vectors, then a byte tail.  When s
// and d are congruent mod 16 each vector is one non-temporal load; otherwise
// it is assembled from the two aligned source vectors it straddles (lane i's
// second vector is lane i + 1's first, served by the cache).  Every aligned
// source vector read holds at least one byte of the range, so no read leaves
// the 16-byte granules the range touches.  store(p, v) writes one vector.
template <typename Store>
__device__ __forceinline__ void wave_copy_any(const uint8_t* s, uint8_t* d, uint64_t len, const int lane,
                                              Store store) {
  uint64_t head = (16 - (reinterpret_cast<uintptr_t>(d) & 15)) & 15;
  if (head > len) head = len;
  if (uint64_t(lane) < head) d[lane] = s[lane];
  s += head;
  d += head;
  len -= head;
  const uint64_t n16 = len >> 4;
  u32x4* dv = reinterpret_cast<u32x4*>(d);
  const uint32_t r = uint32_t(reinterpret_cast<uintptr_t>(s) & 15);
  if (r == 0) {
    const u32x4* sv = reinterpret_cast<const u32x4*>(s);
    for (uint64_t i = lane; i < n16; i += kWaveLanes) store(dv + i, ld_nt(sv + i));
  } else {
    const u32x4* sv = reinterpret_cast<const u32x4*>(s - r);
    for (uint64_t i = lane; i < n16; i += kWaveLanes) store(dv + i, realign(sv[i], sv[i + 1], r));
  }
  const uint64_t tail = len & 15;
  if (uint64_t(lane) < tail) d[(n16 << 4) + lane] = s[(n16 << 4) + lane];
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

// Largest grid used for one launch; bigger jobs loop (grid-stride).  A
// dispatch counts its work-items in 32 bits, so the cap times the largest
// workgroup here (512 threads) must stay below 2^32.
constexpr uint64_t kMaxGrid = uint64_t(1) << 22;
static_assert(kMaxGrid * 512 < (uint64_t(1) << 32), "grid work-items must fit 32 bits");

inline unsigned grid_for(uint64_t items) { return (unsigned)(items < kMaxGrid ? items : kMaxGrid); }

}  // namespace tc
