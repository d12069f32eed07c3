// Fragment plans for gfx950: a descriptor list cut into tasks of at most
// one piece, one task per wave of the copy, in destination order for long
// unordered lists; and the plan's workspace layout.
#include "tc_device.h"

namespace tc {
namespace {

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
// predecessor's (checked across the block's last boundary too), the largest
// destination end, and whether some fragment ends past the 48-bit offsets of
// a task (flag bit 0: unordered, bit 1: out of range).
__global__ __launch_bounds__(kThreads) void k_plan_count(const tc_fragment* __restrict__ frags,
                                                        const int64_t n, const uint64_t piece,
                                                        const uint64_t cut,
                                                        uint64_t* __restrict__ block_cnt,
                                                        uint64_t* __restrict__ block_len,
                                                        uint64_t* __restrict__ block_unord,
                                                        uint64_t* __restrict__ block_dend) {
  const int64_t f0 = int64_t(blockIdx.x) * kPlanPerBlock + int64_t(threadIdx.x) * kPlanPerThread;
  uint64_t c = 0, l = 0, dend = 0;
  int unord = 0, bad = 0;
#pragma unroll
  for (int j = 0; j < kPlanPerThread; ++j)
    if (f0 + j < n) {
      const tc_fragment f = frags[f0 + j];
      c += pieces_of(f, piece, cut);
      l += f.len;
      if (f.len && f.dst_off + f.len > dend) dend = f.dst_off + f.len;
      if (f.len && (f.len > kOffsetLimit || f.src_off > kOffsetLimit - f.len ||
                    f.dst_off > kOffsetLimit - f.len))
        bad = 1;
      if (f0 + j + 1 < n && frags[f0 + j + 1].dst_off < f.dst_off) unord = 1;
    }
  uint64_t tc_, tl;
  block_exclusive_scan(c, &tc_);
  block_exclusive_scan(l, &tl);
  const int any_unord = __syncthreads_or(unord);
  const int any_bad = __syncthreads_or(bad);
  const uint64_t bdend = block_max_u64(dend);
  if (threadIdx.x == 0) {
    block_cnt[blockIdx.x] = tc_;
    block_len[blockIdx.x] = tl;
    block_unord[blockIdx.x] = (any_unord ? 1u : 0u) | (any_bad ? 2u : 0u);
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
  int unord = 0, bad = 0;
  for (int64_t base = 0; base < nblocks; base += kThreads) {
    const int64_t i = base + threadIdx.x;
    const uint64_t v = i < nblocks ? block_cnt[i] : 0;
    const uint64_t l = i < nblocks ? block_len[i] : 0;
    if (i < nblocks) {
      unord |= (block_unord[i] & 1u) ? 1 : 0;
      bad |= (block_unord[i] & 2u) ? 1 : 0;
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
  const int any_bad = __syncthreads_or(bad);
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
    hdr->out_of_range = any_bad ? 1 : 0;
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

}  // namespace

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

}  // namespace tc
