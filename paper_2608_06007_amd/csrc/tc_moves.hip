// Byte movers for gfx950: paged-KV block gather/scatter (publish / hydrate)
// and planned fragment copies (prefetch_many, materialization transfer).
//
// Design (measured on MI355X): the copies are HBM-bound, and the launch
// shape that streams best is a one-shot grid of small workgroups -- 256
// lanes, one 16-byte vector each, 4 KiB per workgroup -- with non-temporal
// loads and stores (the data is touched once) and a workgroup order that
// gives each XCD runs of consecutive tiles.  Workgroups are dealt to the 8
// XCDs round-robin by block index; without the regrouping every 32 KiB block
// would be split across all eight L2s and address translators.
#include "tc_internal.h"

namespace tc {
namespace {

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
    const uint64_t w = xcd_grouped(b, total_tiles, kGather ? kXcdGroup : kXcdGroupScatter);
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

// Byte-granular variant for pools whose bases, stride or block size are not
// 16-byte multiples.
template <bool kGather>
__global__ __launch_bounds__(kThreads) void k_blocks_bytes(const RegionTable tab, const int32_t R,
                                                          const int64_t B, const int64_t stride,
                                                          const int32_t* __restrict__ ids,
                                                          const uint64_t n_chunks,
                                                          uint8_t* __restrict__ buf) {
  for (uint64_t c = blockIdx.x; c < n_chunks; c += gridDim.x) {
    const uint64_t i = c / uint64_t(R);
    const int32_t r = (int32_t)(c - i * uint64_t(R));
    uint8_t* pool = reinterpret_cast<uint8_t*>(tab.base[r]) + int64_t(ids[i]) * stride;
    uint8_t* xfer = buf + c * uint64_t(B);
    const uint8_t* from = kGather ? pool : xfer;
    uint8_t* to = kGather ? xfer : pool;
    for (int64_t x = threadIdx.x; x < B; x += kThreads) to[x] = from[x];
  }
}

// ------------------------------------------------------------------------
// Fragment plan.  Fragment f becomes ceil((len + h) / piece) tasks, where
// h = dst_off & cut: with cut = 127 every task after a fragment's first starts
// on a 128-byte destination line (no line is split between two waves inside
// a fragment); cut = 0 gives plain multiples of the piece.  tstart[f] is its
// first task, tstart[n] the total.  Passes: per-block task and byte sums,
// an exclusive scan of the block sums (one workgroup), the per-fragment
// prefix, then (after the host has read the total) the task table.
// ------------------------------------------------------------------------
__device__ __forceinline__ uint64_t shfl_up_u64(uint64_t v, int delta) {
  const uint32_t lo = __shfl_up((uint32_t)v, delta, kWaveLanes);
  const uint32_t hi = __shfl_up((uint32_t)(v >> 32), delta, kWaveLanes);
  return (uint64_t(hi) << 32) | lo;
}

// Exclusive scan over a 256-thread block; *block_total receives the sum.
__device__ uint64_t block_exclusive_scan(uint64_t v, uint64_t* block_total) {
  __shared__ uint64_t wave_tot[kThreads / kWaveLanes];
  const int lane = threadIdx.x & (kWaveLanes - 1);
  const int w = threadIdx.x >> 6;
  uint64_t incl = v;
#pragma unroll
  for (int d = 1; d < kWaveLanes; d <<= 1) {
    const uint64_t o = shfl_up_u64(incl, d);
    if (lane >= d) incl += o;
  }
  if (lane == kWaveLanes - 1) wave_tot[w] = incl;
  __syncthreads();
  uint64_t before = 0, total = 0;
#pragma unroll
  for (int k = 0; k < kThreads / kWaveLanes; ++k) {
    if (k < w) before += wave_tot[k];
    total += wave_tot[k];
  }
  __syncthreads();  // wave_tot is reused by the next scan
  *block_total = total;
  return before + incl - v;
}

constexpr int kPlanPerThread = kPlanPerBlock / kThreads;  // 4

__device__ __forceinline__ uint64_t pieces_of(const tc_fragment& f, uint64_t piece, uint64_t cut) {
  return f.len ? (f.len + (f.dst_off & cut) + piece - 1) / piece : 0;
}

// Maximum over a 256-thread block (every thread gets it).
__device__ uint64_t block_max_u64(uint64_t v) {
  __shared__ uint64_t wave_max[kThreads / kWaveLanes];
#pragma unroll
  for (int d = kWaveLanes / 2; d >= 1; d >>= 1) {
    const uint64_t o = (uint64_t(uint32_t(__shfl_xor(uint32_t(v >> 32), d, kWaveLanes))) << 32) |
                       uint32_t(__shfl_xor(uint32_t(v), d, kWaveLanes));
    v = v > o ? v : o;
  }
  if ((threadIdx.x & (kWaveLanes - 1)) == 0) wave_max[threadIdx.x >> 6] = v;
  __syncthreads();
  uint64_t m = 0;
#pragma unroll
  for (int k = 0; k < kThreads / kWaveLanes; ++k) m = m > wave_max[k] ? m : wave_max[k];
  __syncthreads();
  return m;
}

// Per block: task and byte sums, whether some destination starts below its
// predecessor's (checked across the block's last boundary too), and the
// largest destination end.
__global__ __launch_bounds__(kThreads) void k_plan_count(const tc_fragment* __restrict__ frags,
                                                        const int64_t n, const uint64_t piece,
                                                        const uint64_t cut,
                                                        uint64_t* __restrict__ block_cnt,
                                                        uint64_t* __restrict__ block_len,
                                                        uint64_t* __restrict__ block_unord,
                                                        uint64_t* __restrict__ block_dend) {
  const int64_t f0 = int64_t(blockIdx.x) * kPlanPerBlock + int64_t(threadIdx.x) * kPlanPerThread;
  uint64_t c = 0, l = 0, dend = 0;
  int unord = 0;
#pragma unroll
  for (int j = 0; j < kPlanPerThread; ++j)
    if (f0 + j < n) {
      const tc_fragment f = frags[f0 + j];
      c += pieces_of(f, piece, cut);
      l += f.len;
      if (f.len && f.dst_off + f.len > dend) dend = f.dst_off + f.len;
      if (f0 + j + 1 < n && frags[f0 + j + 1].dst_off < f.dst_off) unord = 1;
    }
  uint64_t tc_, tl;
  block_exclusive_scan(c, &tc_);
  block_exclusive_scan(l, &tl);
  const int any_unord = __syncthreads_or(unord);
  const uint64_t bdend = block_max_u64(dend);
  if (threadIdx.x == 0) {
    block_cnt[blockIdx.x] = tc_;
    block_len[blockIdx.x] = tl;
    block_unord[blockIdx.x] = any_unord ? 1 : 0;
    block_dend[blockIdx.x] = bdend;
  }
}

// One workgroup: block_cnt becomes its exclusive prefix; the header gets
// the totals.
__global__ __launch_bounds__(kThreads) void k_plan_scan(uint64_t* __restrict__ block_cnt,
                                                       const uint64_t* __restrict__ block_len,
                                                       const uint64_t* __restrict__ block_unord,
                                                       const uint64_t* __restrict__ block_dend,
                                                       const int64_t nblocks, const uint64_t piece,
                                                       const uint64_t cut,
                                                       const int64_t n, const uint64_t capacity,
                                                       const uint64_t permuted,
                                                       PlanHeader* __restrict__ hdr,
                                                       uint64_t* __restrict__ tstart_end) {
  uint64_t carry = 0, bytes = 0, dend = 0;
  int unord = 0;
  for (int64_t base = 0; base < nblocks; base += kThreads) {
    const int64_t i = base + threadIdx.x;
    const uint64_t v = i < nblocks ? block_cnt[i] : 0;
    const uint64_t l = i < nblocks ? block_len[i] : 0;
    if (i < nblocks) {
      unord |= block_unord[i] ? 1 : 0;
      dend = dend > block_dend[i] ? dend : block_dend[i];
    }
    uint64_t total, ltot;
    const uint64_t ex = block_exclusive_scan(v, &total);
    block_exclusive_scan(l, &ltot);
    if (i < nblocks) block_cnt[i] = carry + ex;
    carry += total;
    bytes += ltot;
  }
  const int any_unord = __syncthreads_or(unord);
  dend = block_max_u64(dend);
  if (threadIdx.x == 0) {
    hdr->total_tasks = carry;
    hdr->piece = piece;
    hdr->payload = bytes;
    hdr->n = uint64_t(n);
    hdr->capacity = capacity;
    hdr->dst_unordered = any_unord ? 1 : 0;
    hdr->dst_end = dend;
    hdr->permuted = permuted;
    hdr->cut = cut;
    *tstart_end = carry;
  }
}

__global__ __launch_bounds__(kThreads) void k_plan_tstart(const tc_fragment* __restrict__ frags,
                                                         const int64_t n, const uint64_t piece,
                                                         const uint64_t cut,
                                                         const uint64_t* __restrict__ block_off,
                                                         uint64_t* __restrict__ tstart,
                                                         int64_t* __restrict__ windows,
                                                         const uint64_t capacity) {
  const int64_t f0 = int64_t(blockIdx.x) * kPlanPerBlock + int64_t(threadIdx.x) * kPlanPerThread;
  uint64_t c[kPlanPerThread];
  uint64_t s = 0;
#pragma unroll
  for (int j = 0; j < kPlanPerThread; ++j) {
    c[j] = f0 + j < n ? pieces_of(frags[f0 + j], piece, cut) : 0;
    s += c[j];
  }
  uint64_t block_total;
  uint64_t run = block_off[blockIdx.x] + block_exclusive_scan(s, &block_total);
  // the plan's total (written by k_plan_scan); the window table only has
  // room for a plan that fits the workspace
  const uint64_t total = tstart[n];
  const bool fits = total <= capacity;
  const uint64_t nwin = (total + kWindowTasks - 1) / kWindowTasks;
#pragma unroll
  for (int j = 0; j < kPlanPerThread; ++j) {
    if (f0 + j < n) {
      tstart[f0 + j] = run;
      // Every task lies in exactly one non-empty fragment, which is therefore
      // the first fragment of each window whose first task it holds and the
      // last fragment of each window whose last task it holds.
      if (fits && c[j]) {
        const uint64_t te = run + c[j];  // tasks [run, te)
        for (uint64_t w = (run + kWindowTasks - 1) / kWindowTasks; w * kWindowTasks < te; ++w)
          windows[2 * w] = f0 + j;
        for (uint64_t w = run / kWindowTasks; w < nwin; ++w) {
          const uint64_t last = min(w * kWindowTasks + kWindowTasks - 1, total - 1);
          if (last >= te) break;
          windows[2 * w + 1] = f0 + j;
        }
      }
    }
    run += c[j];
  }
}

__device__ __forceinline__ Task pack_task(uint64_t src, uint64_t dst, uint64_t len, bool first) {
  return Task{src | (dst << 48), (dst >> 16) | (len << 32) | (first ? kTaskFirst : 0)};
}

constexpr int kExpandPerBlock = int(kWindowTasks);  // tasks written by one workgroup

// Block j writes tasks [j * 1024, (j + 1) * 1024), whose first and last
// fragment k_plan_tstart recorded in windows[j].  If they span at most 1024
// fragments their tstart entries go to LDS and every task finds its fragment
// there, otherwise (long runs of empty fragments) each task searches
// globally.  A thread's four tasks are found first and their descriptors
// loaded together, so the loads overlap.
constexpr int kExpandPerThread = kExpandPerBlock / kThreads;
static_assert(kExpandPerThread * kThreads == kExpandPerBlock, "whole tasks per thread");

__global__ __launch_bounds__(kThreads) void k_plan_expand(const tc_fragment* __restrict__ frags,
                                                         const uint64_t* __restrict__ tstart,
                                                         const int64_t* __restrict__ windows,
                                                         const uint64_t total, const uint64_t piece,
                                                         const uint64_t cut,
                                                         Task* __restrict__ tasks) {
  __shared__ uint64_t win[kExpandPerBlock + 1];
  const uint64_t t0 = uint64_t(blockIdx.x) * kExpandPerBlock;
  const uint64_t t1 = min(total, t0 + kExpandPerBlock);
  const int64_t f0 = windows[2 * uint64_t(blockIdx.x)];
  const int64_t f1 = windows[2 * uint64_t(blockIdx.x) + 1];
  const int64_t span = f1 - f0 + 1;
  const bool local = span <= kExpandPerBlock;
  if (local)
    for (int64_t k = threadIdx.x; k <= span; k += kThreads) win[k] = tstart[f0 + k];
  __syncthreads();
  int64_t frag[kExpandPerThread];
  uint64_t start[kExpandPerThread];
#pragma unroll
  for (int j = 0; j < kExpandPerThread; ++j) {
    const uint64_t t = t0 + threadIdx.x + uint64_t(j) * kThreads;
    frag[j] = -1;
    start[j] = 0;
    if (t >= t1) continue;
    int64_t lo, hi;
    if (local) {  // win[lo] <= t < win[hi], indices relative to f0
      lo = 0;
      hi = span;
      while (hi - lo > 1) {
        const int64_t mid = (lo + hi) >> 1;
        if (win[mid] <= t)
          lo = mid;
        else
          hi = mid;
      }
      start[j] = win[lo];
      frag[j] = f0 + lo;
    } else {
      lo = f0;
      hi = f1 + 1;
      while (hi - lo > 1) {
        const int64_t mid = (lo + hi) >> 1;
        if (tstart[mid] <= t)
          lo = mid;
        else
          hi = mid;
      }
      start[j] = tstart[lo];
      frag[j] = lo;
    }
  }
  tc_fragment f[kExpandPerThread];
#pragma unroll
  for (int j = 0; j < kExpandPerThread; ++j)
    if (frag[j] >= 0) f[j] = frags[frag[j]];
#pragma unroll
  for (int j = 0; j < kExpandPerThread; ++j) {
    if (frag[j] < 0) continue;
    const uint64_t t = t0 + threadIdx.x + uint64_t(j) * kThreads;
    // task k covers [k * piece - h, (k + 1) * piece - h) of the fragment,
    // clipped to [0, len)
    const uint64_t k = t - start[j], h = f[j].dst_off & cut;
    const uint64_t off = k ? k * piece - h : 0;
    const uint64_t end = min(f[j].len, (k + 1) * piece - h);
    tasks[t] = pack_task(f[j].src_off + off, f[j].dst_off + off, end - off, k == 0);
  }
}

// ------------------------------------------------------------------------
// Planned copy: one task per wave, four consecutive tasks per workgroup
// (workgroups of one XCD run consecutive).
// ------------------------------------------------------------------------
constexpr int kTasksPerBlock = kThreads / kWaveLanes;

__global__ __launch_bounds__(kThreads) void k_copy_tasks(const uint8_t* __restrict__ src,
                                                        uint8_t* __restrict__ dst,
                                                        const PlanHeader* __restrict__ hdr,
                                                        const Task* __restrict__ tasks,
                                                        const uint64_t total,
                                                        const uint64_t nblocks) {
  const int lane = threadIdx.x & (kWaveLanes - 1);
  const uint64_t w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const bool reordered = hdr->permuted != 0;
  const uint64_t group = reordered ? kXcdGroupReordered : kXcdGroup;
  for (uint64_t b = blockIdx.x; b < nblocks; b += gridDim.x) {
    const uint64_t t = xcd_grouped(b, nblocks, group) * kTasksPerBlock + w;
    if (t >= total) continue;
    const Task tk = tasks[t];
    const uint8_t* s = src + task_src(tk);
    uint8_t* d = dst + task_dst(tk);
    uint64_t len = task_len(tk);
    const uintptr_t sa = reinterpret_cast<uintptr_t>(s), da = reinterpret_cast<uintptr_t>(d);
    if (((sa ^ da) & 15) == 0) {
      // byte head up to 16-byte alignment, 16-byte body, byte tail
      uint64_t head = (16 - (sa & 15)) & 15;
      if (head > len) head = len;
      if (uint64_t(lane) < head) d[lane] = s[lane];
      s += head;
      d += head;
      len -= head;
      const uint64_t n16 = len >> 4;
      const u32x4* sv = reinterpret_cast<const u32x4*>(s);
      u32x4* dv = reinterpret_cast<u32x4*>(d);
      if (reordered)
        for (uint64_t i = lane; i < n16; i += kWaveLanes) st_nt(dv + i, ld_nt(sv + i));
      else
        for (uint64_t i = lane; i < n16; i += kWaveLanes) st_sc1_nt(dv + i, ld_nt(sv + i));
      const uint64_t tail = len & 15;
      if (uint64_t(lane) < tail) d[(n16 << 4) + lane] = s[(n16 << 4) + lane];
    } else {
      for (uint64_t i = lane; i < len; i += kWaveLanes) d[i] = s[i];
    }
  }
}

// ------------------------------------------------------------------------
// Integrity digests (the verify stage of the materialization pipeline).
// A fragment's digest is S1 = sum b_i and S2 = sum (i + 1) b_i (mod 2^64)
// over its bytes.  The copy kernel, with the same launch shape as
// k_copy_tasks, also writes each task's partial sums into the task's digest
// slot: P1 = sum c_j and P2 = sum (a_j + 1) c_j over its own bytes c_j, where
// a_j is the byte's destination offset.  A fragment whose destination starts
// at D then has S1 = sum P1 and S2 = sum P2 - D * S1 over its tasks, however
// the plan cut it; k_digest_reduce adds the tasks of each fragment and
// subtracts D * S1 once.  No two tasks add into the same word during the
// copy, and the reduction adds at most a few words per window atomically.
// ------------------------------------------------------------------------
enum DigestMode { kCopyDigest = 0, kDigestSrc = 1, kDigestDst = 2 };

typedef uint64_t u64x2 __attribute__((ext_vector_type(2)));

// Bytes in every lane of the 16-byte vector v: sum and sum of m * c_m
// (m = 0..15, the byte's position within the vector).
__device__ __forceinline__ void vec_sums(const u32x4 v, uint32_t* sum, uint32_t* wsum) {
  const uint32_t ones = 0x01010101u;
  *sum = __builtin_amdgcn_udot4(v.x, ones,
                                __builtin_amdgcn_udot4(v.y, ones,
                                                       __builtin_amdgcn_udot4(v.z, ones,
                                                                              __builtin_amdgcn_udot4(v.w, ones, 0u, false),
                                                                              false),
                                                       false),
                                false);
  *wsum = __builtin_amdgcn_udot4(v.x, 0x03020100u,
                                 __builtin_amdgcn_udot4(v.y, 0x07060504u,
                                                        __builtin_amdgcn_udot4(v.z, 0x0B0A0908u,
                                                                               __builtin_amdgcn_udot4(v.w, 0x0F0E0D0Cu, 0u, false),
                                                                               false),
                                                        false),
                                 false);
}

// Sum of a 32-bit value over the 64 lanes of a wave (all lanes active):
// DPP adds within each row of 16 lanes (swap neighbours, swap pairs, mirror
// halves, mirror the row), then the four row sums read into scalars.
__device__ __forceinline__ uint32_t wave_sum32(uint32_t v) {
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false);   // quad_perm 1,0,3,2
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false);   // quad_perm 2,3,0,1
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false);  // row_half_mirror
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false);  // row_mirror
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 0) +
         (uint32_t)__builtin_amdgcn_readlane((int)v, 16) +
         (uint32_t)__builtin_amdgcn_readlane((int)v, 32) +
         (uint32_t)__builtin_amdgcn_readlane((int)v, 48);
}

// The same sum left in lane 63 only (other lanes hold partial sums): the row
// reduction, then row 0 added into row 1 and row 2 into row 3, then lane 31
// (rows 0 + 1) into rows 2 and 3.  No scalar work.
__device__ __forceinline__ uint32_t wave_sum32_lane63(uint32_t v) {
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false);   // quad_perm 1,0,3,2
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false);   // quad_perm 2,3,0,1
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false);  // row_half_mirror
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false);  // row_mirror
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false);  // row_bcast:15
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false);  // row_bcast:31
  return v;
}

// A task is summed in chunks of 256 vectors (4 KiB) of its 16-byte-aligned
// body: chunk 0 also takes the head bytes, the last chunk the tail bytes.
// Inside a chunk every weight is the byte's position relative to the chunk's
// base (0 for chunk 0, head + 4096 c after), below 4127, so the chunk's two
// sums are exact in 32 bits (sum of j * 255 over j < 4127 is below 2^32);
// the wave-uniform 64-bit totals add base * sum on top.
constexpr uint64_t kChunkVecs = 256;

// Sums of one task's bytes at s (copied to d in kCopyDigest mode), weighted
// by destination position (the task starts at destination offset dof); pre
// holds this lane's first body vector when the caller has loaded it already
// (tasks of one aligned vector per lane at most, no head).
template <int kMode>
__device__ __forceinline__ void task_sums(const uint8_t* s, uint8_t* d, const uint64_t len,
                                          const uint64_t dof, const int lane, const bool preloaded,
                                          const u32x4 pre, const bool plain, u64x2* slot) {
  uint64_t A = 0, W = 0;
  const uintptr_t sa = reinterpret_cast<uintptr_t>(s);
  const uintptr_t mis = kMode == kCopyDigest ? (sa ^ reinterpret_cast<uintptr_t>(d)) & 15 : 0;
  if (preloaded) {
    // len <= 64 vectors + tail, no head: one chunk
    const uint64_t n16 = len >> 4;
    uint32_t a = 0, ws = 0;
    if (uint64_t(lane) < n16) {
      if (kMode == kCopyDigest) st_task(reinterpret_cast<u32x4*>(d) + lane, pre, plain);
      uint32_t vs, vw;
      vec_sums(pre, &vs, &vw);
      a = vs;
      ws = uint32_t(lane << 4) * vs + vw;
    }
    const uint64_t body_end = n16 << 4;
    if (uint64_t(lane) < len - body_end) {
      const uint8_t x = s[body_end + lane];
      if (kMode == kCopyDigest) d[body_end + lane] = x;
      a += x;
      ws += uint32_t(body_end + lane) * x;
    }
    const uint32_t ta = wave_sum32_lane63(a), tw = wave_sum32_lane63(ws);
    if (lane == kWaveLanes - 1) *slot = u64x2{ta, uint64_t(tw) + (dof + 1) * ta};
    return;
  } else if (mis == 0) {
    uint64_t head = (16 - (sa & 15)) & 15;
    if (head > len) head = len;
    const uint64_t n16 = (len - head) >> 4;
    const uint64_t body_end = head + (n16 << 4);
    const uint64_t nchunks = n16 == 0 ? 1 : (n16 + kChunkVecs - 1) / kChunkVecs;
    const u32x4* sv = reinterpret_cast<const u32x4*>(s + head);
    u32x4* dv = kMode == kCopyDigest ? reinterpret_cast<u32x4*>(d + head) : nullptr;
    for (uint64_t c = 0; c < nchunks; ++c) {
      const uint64_t base = c == 0 ? 0 : head + (c << 12);
      uint32_t a = 0, ws = 0;
      if (c == 0 && uint64_t(lane) < head) {
        const uint8_t x = s[lane];
        if (kMode == kCopyDigest) d[lane] = x;
        a += x;
        ws += uint32_t(lane) * x;
      }
      const uint64_t i_end = min(n16, (c + 1) * kChunkVecs);
      for (uint64_t i = c * kChunkVecs + lane; i < i_end; i += kWaveLanes) {
        const u32x4 v = ld_nt(sv + i);
        if (kMode == kCopyDigest) st_task(dv + i, v, plain);
        uint32_t vs, vw;
        vec_sums(v, &vs, &vw);
        a += vs;
        ws += uint32_t(head + (i << 4) - base) * vs + vw;
      }
      if (c == nchunks - 1 && uint64_t(lane) < len - body_end) {
        const uint8_t x = s[body_end + lane];
        if (kMode == kCopyDigest) d[body_end + lane] = x;
        a += x;
        ws += uint32_t(body_end + lane - base) * x;
      }
      const uint64_t ca = wave_sum32(a), cw = wave_sum32(ws);
      A += ca;
      W += cw + base * ca;
    }
  } else {
    const uint64_t nchunks = len == 0 ? 0 : (len + 4095) >> 12;
    for (uint64_t c = 0; c < nchunks; ++c) {
      const uint64_t base = c << 12;
      const uint64_t i_end = min(len, base + 4096);
      uint32_t a = 0, ws = 0;
      for (uint64_t i = base + lane; i < i_end; i += kWaveLanes) {
        const uint8_t x = s[i];
        if (kMode == kCopyDigest) d[i] = x;
        a += x;
        ws += uint32_t(i - base) * x;
      }
      const uint64_t ca = wave_sum32(a), cw = wave_sum32(ws);
      A += ca;
      W += cw + base * ca;
    }
  }
  if (lane == 0) *slot = u64x2{A, W + (dof + 1) * A};
}

// kPerWave consecutive tasks per wave.  The first body vector of every task
// that fits one vector per lane is loaded before any of them is summed, so a
// wave keeps kPerWave KiB in flight instead of one.
template <int kMode, int kPerWave>
__global__ __launch_bounds__(kThreads) void k_copy_digest(const uint8_t* __restrict__ src,
                                                         uint8_t* __restrict__ dst,
                                                         const PlanHeader* __restrict__ hdr,
                                                         const Task* __restrict__ tasks,
                                                         u64x2* __restrict__ slots,
                                                         const uint64_t total,
                                                         const uint64_t nblocks,
                                                         uint64_t* __restrict__ digests,
                                                         const uint64_t words) {
  const bool plain = kMode == kCopyDigest && hdr->permuted != 0;
  const uint64_t group = plain ? kXcdGroupReordered : kXcdGroup;
  // clear the digests for the reduction that follows (it adds into them)
  for (uint64_t i = uint64_t(blockIdx.x) * kThreads + threadIdx.x; i < words;
       i += uint64_t(gridDim.x) * kThreads)
    digests[i] = 0;
  const int lane = threadIdx.x & (kWaveLanes - 1);
  const uint64_t w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  for (uint64_t b = blockIdx.x; b < nblocks; b += gridDim.x) {
    const uint64_t t0 = (xcd_grouped(b, nblocks, group) * kTasksPerBlock + w) * kPerWave;
    if (t0 >= total) continue;
    const uint8_t* s[kPerWave];
    uint8_t* d[kPerWave];
    uint64_t len[kPerWave];
    bool pre[kPerWave];
    u32x4 v[kPerWave];
    Task tk[kPerWave];
#pragma unroll
    for (int k = 0; k < kPerWave; ++k) tk[k] = tasks[min(t0 + k, total - 1)];  // one scalar load
#pragma unroll
    for (int k = 0; k < kPerWave; ++k) {
      const uint64_t so = task_src(tk[k]);
      const uint64_t dof = task_dst(tk[k]);
      s[k] = src + (kMode == kDigestDst ? dof : so);
      d[k] = kMode == kCopyDigest ? dst + dof : nullptr;
      len[k] = t0 + k < total ? task_len(tk[k]) : 0;
      const uintptr_t sa = reinterpret_cast<uintptr_t>(s[k]);
      const uintptr_t al = kMode == kCopyDigest ? (sa | reinterpret_cast<uintptr_t>(d[k])) & 15 : sa & 15;
      pre[k] = al == 0 && len[k] <= uint64_t(kWaveLanes) * 16 + 15;
      v[k] = u32x4{0, 0, 0, 0};
      if (pre[k] && uint64_t(lane) < (len[k] >> 4)) v[k] = ld_nt(reinterpret_cast<const u32x4*>(s[k]) + lane);
    }
    // The group is one run of a fragment when no task after the first starts
    // a fragment, every task is one aligned vector per lane and all but the
    // last are full 1 KiB pieces.  Its bytes then sit at positions below
    // kPerWave * 1024 <= 4096 from the first task's start, so the run's two
    // sums are exact in 32 bits and one wave reduction serves the group: the
    // first task's slot takes the run's sums and the others zeros, which the
    // reduction by fragment adds up to the same digest.
    bool run = t0 + kPerWave <= total;
#pragma unroll
    for (int k = 0; k < kPerWave; ++k) {
      run = run && pre[k] && (k == 0 || (tk[k].hi & kTaskFirst) == 0) &&
            (k == kPerWave - 1 || len[k] == uint64_t(kWaveLanes) * 16);
    }
    if (run) {
      uint32_t a = 0, ws = 0;
#pragma unroll
      for (int k = 0; k < kPerWave; ++k) {
        if (uint64_t(lane) < (len[k] >> 4)) {
          if (kMode == kCopyDigest) st_task(reinterpret_cast<u32x4*>(d[k]) + lane, v[k], plain);
          uint32_t vs, vw;
          vec_sums(v[k], &vs, &vw);
          a += vs;
          ws += uint32_t(k * kWaveLanes * 16 + lane * 16) * vs + vw;
        }
      }
      constexpr int kLast = kPerWave - 1;
      const uint64_t body_end = (len[kLast] >> 4) << 4;
      if (uint64_t(lane) < len[kLast] - body_end) {
        const uint8_t x = s[kLast][body_end + lane];
        if (kMode == kCopyDigest) d[kLast][body_end + lane] = x;
        a += x;
        ws += uint32_t(kLast * kWaveLanes * 16 + body_end + lane) * x;
      }
      const uint32_t ta = wave_sum32_lane63(a), tw = wave_sum32_lane63(ws);
      if (lane == kWaveLanes - 1)
        slots[t0] = u64x2{ta, uint64_t(tw) + (task_dst(tk[0]) + 1) * ta};
      else if (lane >= kWaveLanes - kPerWave)
        slots[t0 + (kWaveLanes - 1 - lane)] = u64x2{0, 0};
      continue;
    }
#pragma unroll
    for (int k = 0; k < kPerWave; ++k) {
      if (t0 + k >= total) break;
      task_sums<kMode>(s[k], d[k], len[k], task_dst(tk[k]), lane, pre[k], v[k], plain,
                       slots + t0 + k);
    }
  }
}

// digests[0 .. 2n) = 0 when there is no task to run (a fill kernel, so the
// sequence can be captured).
__global__ __launch_bounds__(kThreads) void k_fill_zero(uint64_t* __restrict__ p, const uint64_t n) {
  for (uint64_t i = uint64_t(blockIdx.x) * kThreads + threadIdx.x; i < n;
       i += uint64_t(gridDim.x) * kThreads)
    p[i] = 0;
}

// Reduce-by-fragment of the task slots.  Block j owns tasks
// [j * 1024, (j + 1) * 1024), whose first and last fragment the plan recorded
// in windows[j]; each thread takes four consecutive tasks, whose slots it
// loads first, and adds them per fragment in registers.  A fragment whose
// tasks all lie in the block is written with a plain store; one that crosses
// the block's edges (at most the first and the last) is added atomically into
// the zeroed digest.  Each partial sum subtracts D * S1 for its own S1, D
// being the fragment's destination offset (its first task's).
constexpr int kReducePerThread = kExpandPerBlock / kThreads;
static_assert(kReducePerThread * kThreads == kExpandPerBlock, "whole tasks per thread");

__global__ __launch_bounds__(kThreads) void k_digest_reduce(const uint64_t* __restrict__ tstart,
                                                           const uint64_t total,
                                                           const PlanHeader* __restrict__ hdr,
                                                           const uint64_t* __restrict__ perm,
                                                           const Task* __restrict__ tasks,
                                                           const u64x2* __restrict__ slots,
                                                           const int64_t* __restrict__ windows,
                                                           uint64_t* __restrict__ digests) {
  __shared__ uint64_t win[kExpandPerBlock + 1];
  __shared__ uint64_t acc[2 * kExpandPerBlock];
  const uint64_t t0 = uint64_t(blockIdx.x) * kExpandPerBlock;
  const uint64_t t1 = min(total, t0 + kExpandPerBlock);
  const uint64_t tb = t0 + uint64_t(threadIdx.x) * kReducePerThread;
  u64x2 p[kReducePerThread];
#pragma unroll
  for (int j = 0; j < kReducePerThread; ++j)
    p[j] = tb + j < t1 ? slots[tb + j] : u64x2{0, 0};
  const int64_t f0 = windows[2 * uint64_t(blockIdx.x)];
  const int64_t f1 = windows[2 * uint64_t(blockIdx.x) + 1];
  const int64_t span = f1 - f0 + 1;
  const bool local = span <= kExpandPerBlock;
  // digests are indexed by the caller's order; a reordered plan maps back
  const bool mapped = perm != nullptr && hdr->permuted != 0;
  if (local) {
    for (int64_t k = threadIdx.x; k <= span; k += kThreads) win[k] = tstart[f0 + k];
    for (int64_t k = threadIdx.x; k < 2 * span; k += kThreads) acc[k] = 0;
  }
  __syncthreads();
  if (local) {
    // destination offsets of the fragments this thread writes out below
    uint64_t dbase[kReducePerThread];
#pragma unroll
    for (int j = 0; j < kReducePerThread; ++j) {
      const int64_t k = threadIdx.x + int64_t(j) * kThreads;
      dbase[j] = k < span && win[k] < win[k + 1] ? task_dst(tasks[win[k]]) : 0;
    }
    if (tb < t1) {
      // fragment of the first task: win[lo] <= tb < win[hi], relative to f0
      int64_t lo = 0, hi = span;
      while (hi - lo > 1) {
        const int64_t mid = (lo + hi) >> 1;
        if (win[mid] <= tb)
          lo = mid;
        else
          hi = mid;
      }
      uint64_t s1 = 0, s2 = 0;
#pragma unroll
      for (int j = 0; j < kReducePerThread; ++j) {
        const uint64_t t = tb + j;
        if (t >= t1) break;
        // win[span] > t1 - 1 >= t, so lo stays below span
        while (win[lo + 1] <= t) {
          if (s1 | s2) {
            atomicAdd(reinterpret_cast<unsigned long long*>(&acc[2 * lo]), (unsigned long long)s1);
            atomicAdd(reinterpret_cast<unsigned long long*>(&acc[2 * lo + 1]), (unsigned long long)s2);
          }
          s1 = s2 = 0;
          ++lo;
        }
        s1 += p[j].x;
        s2 += p[j].y;
      }
      if (s1 | s2) {
        atomicAdd(reinterpret_cast<unsigned long long*>(&acc[2 * lo]), (unsigned long long)s1);
        atomicAdd(reinterpret_cast<unsigned long long*>(&acc[2 * lo + 1]), (unsigned long long)s2);
      }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kReducePerThread; ++j) {
      const int64_t k = threadIdx.x + int64_t(j) * kThreads;
      if (k >= span) break;
      uint64_t* out = digests + 2 * (mapped ? perm[f0 + k] : uint64_t(f0 + k));
      const uint64_t a = acc[2 * k], b = acc[2 * k + 1] - dbase[j] * acc[2 * k];
      if (win[k] >= t0 && win[k + 1] <= t1) {
        out[0] = a;
        out[1] = b;
      } else {
        atomicAdd(reinterpret_cast<unsigned long long*>(out), (unsigned long long)a);
        atomicAdd(reinterpret_cast<unsigned long long*>(out + 1), (unsigned long long)b);
      }
    }
  } else {
    // long runs of empty fragments: each task searches the global table
#pragma unroll
    for (int j = 0; j < kReducePerThread; ++j) {
      const uint64_t t = tb + j;
      if (t >= t1) break;
      int64_t lo = f0, hi = f1 + 1;
      while (hi - lo > 1) {
        const int64_t mid = (lo + hi) >> 1;
        if (tstart[mid] <= t)
          lo = mid;
        else
          hi = mid;
      }
      const uint64_t s2 = p[j].y - task_dst(tasks[tstart[lo]]) * p[j].x;
      const uint64_t o = mapped ? perm[lo] : uint64_t(lo);
      atomicAdd(reinterpret_cast<unsigned long long*>(&digests[2 * o]), (unsigned long long)p[j].x);
      atomicAdd(reinterpret_cast<unsigned long long*>(&digests[2 * o + 1]), (unsigned long long)s2);
    }
  }
}

// ------------------------------------------------------------------------
// Destination-ordered plans: a counting sort of the fragments by
// dst_off >> shift (buckets of 2^shift bytes).  The tasks then write the
// destination in address order -- measured +12.6% on a million fragments
// scattered over 16 GiB (gathers, which read scattered blocks and write in
// order, are the fastest block pattern on this GPU).  Inside a bucket the
// order is whatever the atomics give; a copy does not depend on it.
// ------------------------------------------------------------------------
__device__ __forceinline__ uint64_t bucket_of(uint64_t dst_off, int shift, uint64_t nbk) {
  const uint64_t b = dst_off >> shift;  // empty fragments may lie past the end: clamp
  return b < nbk ? b : nbk - 1;
}

// Bucket sizes; each fragment keeps the count it found as its rank inside
// its bucket (in no particular order), so the scatter needs no atomics.
__global__ __launch_bounds__(kThreads) void k_bucket_hist(const tc_fragment* __restrict__ frags,
                                                         const int64_t n, const int shift,
                                                         const uint64_t nbk,
                                                         uint64_t* __restrict__ cnt,
                                                         uint64_t* __restrict__ rank) {
  for (int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * kThreads)
    rank[i] = atomicAdd(
        reinterpret_cast<unsigned long long*>(&cnt[bucket_of(frags[i].dst_off, shift, nbk)]), 1ull);
}

// Exclusive scan of v[0 .. m) in place, in three passes: sums of 1024
// entries, a scan of those sums (one workgroup), then each 1024-entry block.
__global__ __launch_bounds__(kThreads) void k_scan_sums(const uint64_t* __restrict__ v,
                                                       const uint64_t m,
                                                       uint64_t* __restrict__ sums) {
  const uint64_t i0 = uint64_t(blockIdx.x) * kPlanPerBlock + uint64_t(threadIdx.x) * kPlanPerThread;
  uint64_t t = 0;
#pragma unroll
  for (int j = 0; j < kPlanPerThread; ++j)
    if (i0 + j < m) t += v[i0 + j];
  uint64_t total;
  block_exclusive_scan(t, &total);
  if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

__global__ __launch_bounds__(kThreads) void k_scan_one(uint64_t* __restrict__ v, const uint64_t m) {
  uint64_t carry = 0;
  for (uint64_t base = 0; base < m; base += kThreads) {
    const uint64_t i = base + threadIdx.x;
    uint64_t total;
    const uint64_t ex = block_exclusive_scan(i < m ? v[i] : 0, &total);
    if (i < m) v[i] = carry + ex;
    carry += total;
  }
}

__global__ __launch_bounds__(kThreads) void k_scan_apply(uint64_t* __restrict__ v, const uint64_t m,
                                                        const uint64_t* __restrict__ sums) {
  const uint64_t i0 = uint64_t(blockIdx.x) * kPlanPerBlock + uint64_t(threadIdx.x) * kPlanPerThread;
  uint64_t c[kPlanPerThread];
  uint64_t t = 0;
#pragma unroll
  for (int j = 0; j < kPlanPerThread; ++j) {
    c[j] = i0 + j < m ? v[i0 + j] : 0;
    t += c[j];
  }
  uint64_t total;
  uint64_t run = sums[blockIdx.x] + block_exclusive_scan(t, &total);
#pragma unroll
  for (int j = 0; j < kPlanPerThread; ++j) {
    if (i0 + j < m) v[i0 + j] = run;
    run += c[j];
  }
}

// Fragment i goes to its bucket's start plus its rank.
__global__ __launch_bounds__(kThreads) void k_bucket_scatter(const tc_fragment* __restrict__ frags,
                                                            const int64_t n, const int shift,
                                                            const uint64_t nbk,
                                                            const uint64_t* __restrict__ off,
                                                            const uint64_t* __restrict__ rank,
                                                            tc_fragment* __restrict__ sorted,
                                                            uint64_t* __restrict__ perm) {
  for (int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * kThreads) {
    const tc_fragment f = frags[i];
    const uint64_t pos = off[bucket_of(f.dst_off, shift, nbk)] + rank[i];
    sorted[pos] = f;
    perm[pos] = uint64_t(i);
  }
}

// Largest grid used for one launch; bigger jobs loop (grid-stride).
constexpr uint64_t kMaxGrid = uint64_t(1) << 24;

unsigned grid_for(uint64_t items) { return (unsigned)(items < kMaxGrid ? items : kMaxGrid); }

}  // namespace

// ------------------------------------------------------------------------
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

static int64_t plan_blocks(int64_t n) { return (n + kPlanPerBlock - 1) / kPlanPerBlock; }

static size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Buckets for reordering a list of n fragments (0: lists this short keep
// their order): a quarter of n rounded up to a power of two, at most 2^18.
static uint64_t plan_buckets(int64_t n) {
  if (n < kReorderMin) return 0;
  uint64_t p = 1;
  while (p < uint64_t(n)) p <<= 1;
  p /= 4;
  return p < (uint64_t(1) << 18) ? p : (uint64_t(1) << 18);
}

static size_t plan_tail_bytes(int64_t n) {
  size_t t = align256(8 * size_t(n + 1)) + align256(4 * 8 * size_t(plan_blocks(n)));
  const uint64_t nbk = plan_buckets(n);
  if (nbk)
    t += align256(sizeof(tc_fragment) * size_t(n)) + align256(8 * size_t(n)) + align256(8 * nbk) +
         align256(8 * ((nbk + kPlanPerBlock - 1) / kPlanPerBlock));
  return t;
}

// Bytes of the task table, digest slots and window entries for cap tasks.
static size_t task_area_bytes(size_t cap) {
  return kTaskBytes * cap + kWindowBytes * ((cap + kWindowTasks - 1) / kWindowTasks);
}

PlanLayout plan_layout(int64_t n, size_t ws_bytes) {
  PlanLayout L;
  const size_t tail = plan_tail_bytes(n);
  const size_t start = ws_bytes > tail ? ((ws_bytes - tail) & ~size_t(255)) : 0;
  L.tstart = start;
  L.blocks = start + align256(8 * size_t(n + 1));
  L.nbuckets = plan_buckets(n);
  L.sorted = L.blocks + align256(4 * 8 * size_t(plan_blocks(n)));
  L.perm = L.sorted + align256(sizeof(tc_fragment) * size_t(n));
  L.buckets = L.perm + align256(8 * size_t(n));
  L.bucket_sums = L.buckets + align256(8 * L.nbuckets);
  // every task has a 16-byte digest slot after the task table, and every
  // 1024 tasks a window entry after the slots
  const size_t avail = start > kTasksOffset ? start - kTasksOffset : 0;
  size_t cap = avail / (kTaskBytes * kWindowTasks + kWindowBytes) * kWindowTasks;
  while (task_area_bytes(cap + 1) <= avail) ++cap;
  L.capacity = cap;
  L.slots = kTasksOffset + cap * sizeof(Task);
  L.windows = kTasksOffset + cap * kTaskBytes;
  return L;
}

// Room for 4n + 2^23 tasks: pieces stay at 1 KiB while the payload is below
// ~2 KiB per fragment plus 8 GiB (a fragment's line offset can add a task).
size_t frag_workspace_bytes(int64_t n) {
  return kTasksOffset + task_area_bytes(4 * size_t(n) + (size_t(1) << 23)) + plan_tail_bytes(n) +
         256;
}

size_t frag_workspace_min_bytes(int64_t n) {
  return kTasksOffset + task_area_bytes(size_t(n) + 1) + plan_tail_bytes(n) + 256;
}

hipError_t launch_plan_count(const tc_fragment* frags, int64_t n, uint64_t piece, uint64_t cut, void* ws,
                             const PlanLayout& L, bool permuted, hipStream_t s) {
  uint8_t* base = static_cast<uint8_t*>(ws);
  PlanHeader* hdr = reinterpret_cast<PlanHeader*>(base);
  uint64_t* tstart = reinterpret_cast<uint64_t*>(base + L.tstart);
  const int64_t nb = plan_blocks(n);
  uint64_t* bcnt = reinterpret_cast<uint64_t*>(base + L.blocks);
  uint64_t* blen = bcnt + nb;
  uint64_t* bunord = blen + nb;
  uint64_t* bdend = bunord + nb;
  hipLaunchKernelGGL(k_plan_count, dim3((unsigned)nb), dim3(kThreads), 0, s, frags, n, piece, cut, bcnt,
                     blen, bunord, bdend);
  hipLaunchKernelGGL(k_plan_scan, dim3(1), dim3(kThreads), 0, s, bcnt, (const uint64_t*)blen,
                     (const uint64_t*)bunord, (const uint64_t*)bdend, nb, piece, cut, n,
                     uint64_t(L.capacity), uint64_t(permuted ? 1 : 0), hdr, tstart + n);
  hipLaunchKernelGGL(k_plan_tstart, dim3((unsigned)nb), dim3(kThreads), 0, s, frags, n, piece, cut,
                     (const uint64_t*)bcnt, tstart, reinterpret_cast<int64_t*>(base + L.windows),
                     uint64_t(L.capacity));
  return hipGetLastError();
}

hipError_t launch_plan_reorder(const tc_fragment* frags, int64_t n, int shift, void* ws,
                               const PlanLayout& L, hipStream_t s) {
  if (n == 0 || L.nbuckets == 0) return hipSuccess;
  uint8_t* base = static_cast<uint8_t*>(ws);
  uint64_t* cnt = reinterpret_cast<uint64_t*>(base + L.buckets);
  uint64_t* sums = reinterpret_cast<uint64_t*>(base + L.bucket_sums);
  tc_fragment* sorted = reinterpret_cast<tc_fragment*>(base + L.sorted);
  uint64_t* perm = reinterpret_cast<uint64_t*>(base + L.perm);
  // ranks live in tstart's room, which the recount after the reorder rewrites
  uint64_t* rank = reinterpret_cast<uint64_t*>(base + L.tstart);
  const uint64_t nbk = L.nbuckets;
  const uint64_t sblocks = (nbk + kPlanPerBlock - 1) / kPlanPerBlock;
  const unsigned fgrid = grid_for((uint64_t(n) + kThreads - 1) / kThreads);
  hipLaunchKernelGGL(k_fill_zero, dim3(grid_for((nbk + kThreads - 1) / kThreads)), dim3(kThreads),
                     0, s, cnt, nbk);
  hipLaunchKernelGGL(k_bucket_hist, dim3(fgrid), dim3(kThreads), 0, s, frags, n, shift, nbk, cnt,
                     rank);
  hipLaunchKernelGGL(k_scan_sums, dim3((unsigned)sblocks), dim3(kThreads), 0, s,
                     (const uint64_t*)cnt, nbk, sums);
  hipLaunchKernelGGL(k_scan_one, dim3(1), dim3(kThreads), 0, s, sums, sblocks);
  hipLaunchKernelGGL(k_scan_apply, dim3((unsigned)sblocks), dim3(kThreads), 0, s, cnt, nbk,
                     (const uint64_t*)sums);
  hipLaunchKernelGGL(k_bucket_scatter, dim3(fgrid), dim3(kThreads), 0, s, frags, n, shift, nbk,
                     (const uint64_t*)cnt, (const uint64_t*)rank, sorted, perm);
  return hipGetLastError();
}

hipError_t launch_plan_expand(const tc_fragment* frags, uint64_t total, uint64_t piece, uint64_t cut,
                              void* ws, const PlanLayout& L, hipStream_t s) {
  if (total == 0) return hipSuccess;
  uint8_t* base = static_cast<uint8_t*>(ws);
  const uint64_t* tstart = reinterpret_cast<const uint64_t*>(base + L.tstart);
  Task* tasks = reinterpret_cast<Task*>(base + kTasksOffset);
  const uint64_t grid = (total + kExpandPerBlock - 1) / kExpandPerBlock;
  const int64_t* windows = reinterpret_cast<const int64_t*>(base + L.windows);
  hipLaunchKernelGGL(k_plan_expand, dim3((unsigned)grid), dim3(kThreads), 0, s, frags, tstart,
                     windows, total, piece, cut, tasks);
  return hipGetLastError();
}

hipError_t launch_copy_tasks(const uint8_t* src, uint8_t* dst, const void* ws, uint64_t total,
                             hipStream_t s) {
  if (total == 0) return hipSuccess;
  const Task* tasks = reinterpret_cast<const Task*>(static_cast<const uint8_t*>(ws) + kTasksOffset);
  const uint64_t nblocks = (total + kTasksPerBlock - 1) / kTasksPerBlock;
  hipLaunchKernelGGL(k_copy_tasks, dim3(grid_for(nblocks)), dim3(kThreads), 0, s, src, dst,
                     static_cast<const PlanHeader*>(ws), tasks, total, nblocks);
  return hipGetLastError();
}

}  // namespace tc

namespace tc {

hipError_t launch_copy_digest(const uint8_t* src, uint8_t* dst, void* ws, const PlanLayout& L,
                              int64_t n, uint64_t total, int mode, uint64_t* digests,
                              hipStream_t s) {
  if (n == 0) return hipSuccess;
  const uint64_t words = 2 * uint64_t(n);
  if (total == 0) {
    const uint64_t zgrid = (words + kThreads - 1) / kThreads;
    hipLaunchKernelGGL(k_fill_zero, dim3(grid_for(zgrid)), dim3(kThreads), 0, s, digests, words);
    return hipGetLastError();
  }
  uint8_t* base = static_cast<uint8_t*>(ws);
  const Task* tasks = reinterpret_cast<const Task*>(base + kTasksOffset);
  u64x2* slots = reinterpret_cast<u64x2*>(base + L.slots);
  const PlanHeader* hdr = reinterpret_cast<const PlanHeader*>(base);
  // Tasks per wave: two for the copy (measured 6.1 vs 5.9 TB/s with one on a
  // TP=8 shard of 1 KiB pieces), four when only reading (4.9 vs 4.75; eight
  // gives no more).
  const uint64_t per_block = uint64_t(kTasksPerBlock) * (mode == kCopyDigest ? 2 : 4);
  const uint64_t nblocks = (total + per_block - 1) / per_block;
  const dim3 grid(grid_for(nblocks)), block(kThreads);
  if (mode == kCopyDigest)
    hipLaunchKernelGGL((k_copy_digest<kCopyDigest, 2>), grid, block, 0, s, src, dst, hdr, tasks, slots,
                       total, nblocks, digests, words);
  else if (mode == kDigestSrc)
    hipLaunchKernelGGL((k_copy_digest<kDigestSrc, 4>), grid, block, 0, s, src, nullptr, hdr, tasks,
                       slots, total, nblocks, digests, words);
  else
    hipLaunchKernelGGL((k_copy_digest<kDigestDst, 4>), grid, block, 0, s, src, nullptr, hdr, tasks,
                       slots, total, nblocks, digests, words);
  const uint64_t rgrid = (total + kExpandPerBlock - 1) / kExpandPerBlock;
  hipLaunchKernelGGL(k_digest_reduce, dim3((unsigned)rgrid), dim3(kThreads), 0, s,
                     reinterpret_cast<const uint64_t*>(base + L.tstart), total,
                     reinterpret_cast<const PlanHeader*>(base),
                     L.nbuckets ? reinterpret_cast<const uint64_t*>(base + L.perm) : nullptr,
                     tasks, (const u64x2*)slots, reinterpret_cast<const int64_t*>(base + L.windows),
                     digests);
  return hipGetLastError();
}

}  // namespace tc
