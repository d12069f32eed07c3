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
// Vector stores with the SC1 scope bit, alone (gather's contiguous output) or
// with NT (hydrate's scattered blocks, planned task copies): measured +1-4%
// over plain non-temporal stores on those streams.  (For a storm of small
// random fragments plain NT stores are ~10% faster; the shard and expert
// copies, which matter more, prefer SC1 NT.)
__device__ __forceinline__ void st_sc1(u32x4* p, u32x4 v) {
  asm volatile("global_store_dwordx4 %0, %1, off sc1" ::"v"(p), "v"(v) : "memory");
}
__device__ __forceinline__ void st_sc1_nt(u32x4* p, u32x4 v) {
  asm volatile("global_store_dwordx4 %0, %1, off sc1 nt" ::"v"(p), "v"(v) : "memory");
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
        st_sc1(reinterpret_cast<u32x4*>(xfer + off), ld_nt(reinterpret_cast<const u32x4*>(pool + off)));
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
// Fragment plan.  Fragment f becomes ceil(len / piece) tasks; tstart[f] is
// its first task, tstart[n] the total.  Passes: per-block task and byte sums,
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

__device__ __forceinline__ uint64_t pieces_of(uint64_t len, uint64_t piece) {
  return (len + piece - 1) / piece;
}

__global__ __launch_bounds__(kThreads) void k_plan_count(const tc_fragment* __restrict__ frags,
                                                        const int64_t n, const uint64_t piece,
                                                        uint64_t* __restrict__ block_cnt,
                                                        uint64_t* __restrict__ block_len) {
  const int64_t f0 = int64_t(blockIdx.x) * kPlanPerBlock + int64_t(threadIdx.x) * kPlanPerThread;
  uint64_t c = 0, l = 0;
#pragma unroll
  for (int j = 0; j < kPlanPerThread; ++j)
    if (f0 + j < n) {
      const uint64_t len = frags[f0 + j].len;
      c += pieces_of(len, piece);
      l += len;
    }
  uint64_t tc_, tl;
  block_exclusive_scan(c, &tc_);
  block_exclusive_scan(l, &tl);
  if (threadIdx.x == 0) {
    block_cnt[blockIdx.x] = tc_;
    block_len[blockIdx.x] = tl;
  }
}

// One workgroup: block_cnt becomes its exclusive prefix; the header gets
// the totals.
__global__ __launch_bounds__(kThreads) void k_plan_scan(uint64_t* __restrict__ block_cnt,
                                                       const uint64_t* __restrict__ block_len,
                                                       const int64_t nblocks, const uint64_t piece,
                                                       const int64_t n, const uint64_t capacity,
                                                       PlanHeader* __restrict__ hdr,
                                                       uint64_t* __restrict__ tstart_end) {
  uint64_t carry = 0, bytes = 0;
  for (int64_t base = 0; base < nblocks; base += kThreads) {
    const int64_t i = base + threadIdx.x;
    const uint64_t v = i < nblocks ? block_cnt[i] : 0;
    const uint64_t l = i < nblocks ? block_len[i] : 0;
    uint64_t total, ltot;
    const uint64_t ex = block_exclusive_scan(v, &total);
    block_exclusive_scan(l, &ltot);
    if (i < nblocks) block_cnt[i] = carry + ex;
    carry += total;
    bytes += ltot;
  }
  if (threadIdx.x == 0) {
    hdr->total_tasks = carry;
    hdr->piece = piece;
    hdr->payload = bytes;
    hdr->n = uint64_t(n);
    hdr->capacity = capacity;
    *tstart_end = carry;
  }
}

__global__ __launch_bounds__(kThreads) void k_plan_tstart(const tc_fragment* __restrict__ frags,
                                                         const int64_t n, const uint64_t piece,
                                                         const uint64_t* __restrict__ block_off,
                                                         uint64_t* __restrict__ tstart) {
  const int64_t f0 = int64_t(blockIdx.x) * kPlanPerBlock + int64_t(threadIdx.x) * kPlanPerThread;
  uint64_t c[kPlanPerThread];
  uint64_t s = 0;
#pragma unroll
  for (int j = 0; j < kPlanPerThread; ++j) {
    c[j] = f0 + j < n ? pieces_of(frags[f0 + j].len, piece) : 0;
    s += c[j];
  }
  uint64_t total;
  uint64_t run = block_off[blockIdx.x] + block_exclusive_scan(s, &total);
#pragma unroll
  for (int j = 0; j < kPlanPerThread; ++j) {
    if (f0 + j < n) tstart[f0 + j] = run;
    run += c[j];
  }
}

// Last f in [lo, hi) with tstart[f] <= t, given tstart[lo] <= t < tstart[hi]
// (64-way search by one wave).
__device__ int64_t wave_find(const uint64_t* __restrict__ tstart, int64_t lo, int64_t hi,
                             uint64_t t, int lane) {
  while (hi - lo > 1) {
    const int64_t step = (hi - lo + kWaveLanes - 1) / kWaveLanes;
    const int64_t p = lo + (int64_t(lane) + 1) * step;
    const bool pred = lane < kWaveLanes - 1 && p < hi && tstart[p] <= t;
    lo += int64_t(__popcll(__ballot(pred))) * step;
    hi = min(hi, lo + step);
  }
  return lo;
}

__device__ __forceinline__ Task pack_task(uint64_t src, uint64_t dst, uint64_t len) {
  return Task{src | (dst << 48), (dst >> 16) | (len << 32)};
}

constexpr int kExpandPerBlock = 1024;  // tasks written by one workgroup

// Block j writes tasks [j * 1024, (j + 1) * 1024).  Wave 0 finds the first
// and last task's fragments; if they span at most 1024 fragments their
// tstart entries go to LDS and every task finds its fragment there,
// otherwise (long runs of empty fragments) each task searches globally.
__global__ __launch_bounds__(kThreads) void k_plan_expand(const tc_fragment* __restrict__ frags,
                                                         const int64_t n,
                                                         const uint64_t* __restrict__ tstart,
                                                         const uint64_t total, const uint64_t piece,
                                                         Task* __restrict__ tasks) {
  __shared__ uint64_t win[kExpandPerBlock + 1];
  __shared__ int64_t range[2];
  const int lane = threadIdx.x & (kWaveLanes - 1);
  const uint64_t t0 = uint64_t(blockIdx.x) * kExpandPerBlock;
  const uint64_t t1 = min(total, t0 + kExpandPerBlock);
  if (threadIdx.x < kWaveLanes) {
    const int64_t f0 = wave_find(tstart, 0, n, t0, lane);
    const int64_t f1 = wave_find(tstart, f0, n, t1 - 1, lane);
    if (lane == 0) {
      range[0] = f0;
      range[1] = f1;
    }
  }
  __syncthreads();
  const int64_t f0 = range[0], f1 = range[1];
  const int64_t span = f1 - f0 + 1;
  const bool local = span <= kExpandPerBlock;
  if (local)
    for (int64_t k = threadIdx.x; k <= span; k += kThreads) win[k] = tstart[f0 + k];
  __syncthreads();
  for (uint64_t t = t0 + threadIdx.x; t < t1; t += kThreads) {
    int64_t lo, hi;
    uint64_t start;
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
      start = win[lo];
      lo += f0;
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
      start = tstart[lo];
    }
    const tc_fragment f = frags[lo];
    const uint64_t off = (t - start) * piece;
    const uint64_t rem = f.len - off;
    tasks[t] = pack_task(f.src_off + off, f.dst_off + off, rem < piece ? rem : piece);
  }
}

// ------------------------------------------------------------------------
// Planned copy: one task per wave, four consecutive tasks per workgroup
// (workgroups of one XCD run consecutive).
// ------------------------------------------------------------------------
constexpr int kTasksPerBlock = kThreads / kWaveLanes;

__global__ __launch_bounds__(kThreads) void k_copy_tasks(const uint8_t* __restrict__ src,
                                                        uint8_t* __restrict__ dst,
                                                        const Task* __restrict__ tasks,
                                                        const uint64_t total,
                                                        const uint64_t nblocks) {
  const int lane = threadIdx.x & (kWaveLanes - 1);
  const uint64_t w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  for (uint64_t b = blockIdx.x; b < nblocks; b += gridDim.x) {
    const uint64_t t = xcd_grouped(b, nblocks, kXcdGroup) * kTasksPerBlock + w;
    if (t >= total) continue;
    const Task tk = tasks[t];
    const uint8_t* s = src + (tk.lo & (kOffsetLimit - 1));
    uint8_t* d = dst + ((tk.lo >> 48) | ((tk.hi & 0xFFFFFFFFu) << 16));
    uint64_t len = tk.hi >> 32;
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
      for (uint64_t i = lane; i < n16; i += kWaveLanes) st_sc1_nt(dv + i, ld_nt(sv + i));
      const uint64_t tail = len & 15;
      if (uint64_t(lane) < tail) d[(n16 << 4) + lane] = s[(n16 << 4) + lane];
    } else {
      for (uint64_t i = lane; i < len; i += kWaveLanes) d[i] = s[i];
    }
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

static size_t plan_tail_bytes(int64_t n) {
  return align256(8 * size_t(n + 1)) + align256(2 * 8 * size_t(plan_blocks(n)));
}

PlanLayout plan_layout(int64_t n, size_t ws_bytes) {
  PlanLayout L;
  const size_t tail = plan_tail_bytes(n);
  const size_t start = ws_bytes > tail ? ((ws_bytes - tail) & ~size_t(255)) : 0;
  L.tstart = start;
  L.blocks = start + align256(8 * size_t(n + 1));
  L.capacity = start > kTasksOffset ? (start - kTasksOffset) / sizeof(Task) : 0;
  return L;
}

// Room for 4n + 2^23 tasks: pieces stay at 1 KiB while the payload is below
// ~3 KiB per fragment plus 8 GiB.
size_t frag_workspace_bytes(int64_t n) {
  return kTasksOffset + sizeof(Task) * (4 * size_t(n) + (size_t(1) << 23)) + plan_tail_bytes(n) +
         256;
}

size_t frag_workspace_min_bytes(int64_t n) {
  return kTasksOffset + sizeof(Task) * (size_t(n) + 1) + plan_tail_bytes(n) + 256;
}

hipError_t launch_plan_count(const tc_fragment* frags, int64_t n, uint64_t piece, void* ws,
                             const PlanLayout& L, hipStream_t s) {
  uint8_t* base = static_cast<uint8_t*>(ws);
  PlanHeader* hdr = reinterpret_cast<PlanHeader*>(base);
  uint64_t* tstart = reinterpret_cast<uint64_t*>(base + L.tstart);
  const int64_t nb = plan_blocks(n);
  uint64_t* bcnt = reinterpret_cast<uint64_t*>(base + L.blocks);
  uint64_t* blen = bcnt + nb;
  hipLaunchKernelGGL(k_plan_count, dim3((unsigned)nb), dim3(kThreads), 0, s, frags, n, piece, bcnt,
                     blen);
  hipLaunchKernelGGL(k_plan_scan, dim3(1), dim3(kThreads), 0, s, bcnt, (const uint64_t*)blen, nb,
                     piece, n, uint64_t(L.capacity), hdr, tstart + n);
  hipLaunchKernelGGL(k_plan_tstart, dim3((unsigned)nb), dim3(kThreads), 0, s, frags, n, piece,
                     (const uint64_t*)bcnt, tstart);
  return hipGetLastError();
}

hipError_t launch_plan_expand(const tc_fragment* frags, int64_t n, uint64_t total, uint64_t piece,
                              void* ws, const PlanLayout& L, hipStream_t s) {
  if (total == 0) return hipSuccess;
  uint8_t* base = static_cast<uint8_t*>(ws);
  const uint64_t* tstart = reinterpret_cast<const uint64_t*>(base + L.tstart);
  Task* tasks = reinterpret_cast<Task*>(base + kTasksOffset);
  const uint64_t grid = (total + kExpandPerBlock - 1) / kExpandPerBlock;
  hipLaunchKernelGGL(k_plan_expand, dim3((unsigned)grid), dim3(kThreads), 0, s, frags, n, tstart,
                     total, piece, tasks);
  return hipGetLastError();
}

hipError_t launch_copy_tasks(const uint8_t* src, uint8_t* dst, const void* ws, uint64_t total,
                             hipStream_t s) {
  if (total == 0) return hipSuccess;
  const Task* tasks = reinterpret_cast<const Task*>(static_cast<const uint8_t*>(ws) + kTasksOffset);
  const uint64_t nblocks = (total + kTasksPerBlock - 1) / kTasksPerBlock;
  hipLaunchKernelGGL(k_copy_tasks, dim3(grid_for(nblocks)), dim3(kThreads), 0, s, src, dst, tasks,
                     total, nblocks);
  return hipGetLastError();
}

}  // namespace tc
