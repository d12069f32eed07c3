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
// first task, tstart[n] the total.
//
// Every pass runs on the device and takes its decisions from the plan header,
// so a plan is enqueued without waiting for the host:
//   count (1 KiB pieces, line cut; clears the reordering's counters)
//   -> decide: totals, status, piece, reordering (one workgroup)
//   [reorder: bucket histogram, bucket scan, scatter -- lists of >= 4096]
//   count again -- only for a reordered list or a larger piece
//   tstart + windows (each workgroup sums the block counts before it)
//   -> expansion into the task table.
// A pass the header does not ask for returns at once.  Every launch costs a
// few microseconds even then, so the passes are as few as the decisions
// allow: 5 launches for short lists, 8 for long ones (9 past 16M fragments).
// ------------------------------------------------------------------------
// v of lane l (l the same in every lane).
__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int l) {
  return (uint64_t(uint32_t(__builtin_amdgcn_readlane(int(uint32_t(v >> 32)), l))) << 32) |
         uint32_t(__builtin_amdgcn_readlane(int(uint32_t(v)), l));
}

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
// Window entries a lane writes for its fragment by itself; a fragment with
// more goes to its whole wave.  With 8, the 256 experts of a MoE permutation
// (28 entries each, all in the first wave of one workgroup) took 40 us in 256
// wave rounds; alone, one 4 GiB fragment (8192 entries) took 437 us.
constexpr uint64_t kWideFragmentWindows = 64;

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
// a task (flag bit 0: unordered, bit 1: out of range).  First pass: the given
// list with 1 KiB pieces and the line cut.  Second pass (again != 0): only if
// the header asks for it, over the list the header names (the reordered one
// or the given one) with the header's piece and cut; only the task sums.
// The first pass also clears the reordering's bucket counters (clear[0 ..
// nclear)), which the histogram adds into if the list is reordered.
__global__ __launch_bounds__(kThreads) void k_plan_count(const tc_fragment* __restrict__ given,
                                                        const tc_fragment* __restrict__ sorted,
                                                        const int64_t n, const int again,
                                                        const PlanHeader* __restrict__ hdr,
                                                        uint64_t* __restrict__ block_cnt,
                                                        uint64_t* __restrict__ block_len,
                                                        uint64_t* __restrict__ block_unord,
                                                        uint64_t* __restrict__ block_dend,
                                                        uint64_t* __restrict__ clear,
                                                        const uint64_t nclear) {
  const tc_fragment* frags = given;
  uint64_t piece = kMinPiece, cut = 127;
  if (!again) {
    for (uint64_t i = uint64_t(blockIdx.x) * kThreads + threadIdx.x; i < nclear;
         i += uint64_t(gridDim.x) * kThreads)
      clear[i] = 0;
  } else {
    if (hdr->status != TC_OK || !(hdr->recount || hdr->permuted)) return;
    if (hdr->permuted) frags = sorted;
    piece = hdr->piece;
    cut = hdr->cut;
  }
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
    if (!again) {
      block_len[blockIdx.x] = tl;
      block_unord[blockIdx.x] = (any_unord ? 1u : 0u) | (any_bad ? 2u : 0u);
      block_dend[blockIdx.x] = bdend;
    }
  }
}

__device__ __forceinline__ uint64_t pow2_at_least(uint64_t x) {
  uint64_t p = 1;
  while (p < x) p <<= 1;
  return p;
}

// One workgroup: the totals of the first count and the plan's decisions.
//   status: TC_ERR_OUT_OF_RANGE if a fragment ends past 2^48, else TC_OK;
//   piece: 1 KiB with the line cut while the tasks fit the workspace;
//     otherwise the smallest power of two >= payload / (capacity - n) (at most
//     2^30), without the cut, and the list is counted again (recount);
//   permuted: a list of >= 4096 fragments (nbuckets > 0) whose destinations
//     are not in ascending order is reordered by destination, with buckets of
//     2^shift bytes covering the largest destination end.
// The task count is final here unless the list is counted again; tstart
// then sets it, with TC_ERR_WORKSPACE if it still does not fit.
__global__ __launch_bounds__(kThreads) void k_plan_scan(const uint64_t* __restrict__ block_cnt,
                                                       const uint64_t* __restrict__ block_len,
                                                       const uint64_t* __restrict__ block_unord,
                                                       const uint64_t* __restrict__ block_dend,
                                                       const int64_t nblocks, const int64_t n,
                                                       const uint64_t capacity,
                                                       const uint64_t nbuckets,
                                                       PlanHeader* __restrict__ hdr) {
  uint64_t carry = 0, bytes = 0, dend = 0;
  int unord = 0, bad = 0;
  for (int64_t i = threadIdx.x; i < nblocks; i += kThreads) {
    carry += block_cnt[i];
    bytes += block_len[i];
    unord |= (block_unord[i] & 1u) ? 1 : 0;
    bad |= (block_unord[i] & 2u) ? 1 : 0;
    dend = dend > block_dend[i] ? dend : block_dend[i];
  }
  block_exclusive_scan(carry, &carry);
  block_exclusive_scan(bytes, &bytes);
  const int any_unord = __syncthreads_or(unord);
  const int any_bad = __syncthreads_or(bad);
  dend = block_max_u64(dend);
  if (threadIdx.x == 0) {
    uint64_t st = any_bad ? TC_ERR_OUT_OF_RANGE : TC_OK;
    uint64_t piece = kMinPiece, cut = 127, recount = 0;
    if (st == TC_OK && carry > capacity) {
      // Too many 1 KiB pieces for the workspace: larger pieces bound the
      // count by n + payload / piece <= capacity (a task's length has 31 bits).
      const uint64_t room = capacity - uint64_t(n);
      piece = pow2_at_least(max(kMinPiece, (bytes + room - 1) / room));
      piece = min(piece, kMaxPiece);
      cut = 0;
      recount = 1;
    }
    if (st == TC_OK && !recount && carry > (uint64_t(1) << 33)) st = TC_ERR_INVALID_ARGUMENT;
    const uint64_t permuted = (st == TC_OK && any_unord && nbuckets) ? 1 : 0;
    uint64_t shift = 12;
    while (shift < 62 && (dend >> shift) >= nbuckets) ++shift;
    hdr->piece = piece;
    hdr->payload = bytes;
    hdr->n = uint64_t(n);
    hdr->capacity = capacity;
    hdr->dst_unordered = any_unord ? 1 : 0;
    hdr->dst_end = dend;
    hdr->permuted = permuted;
    hdr->cut = cut;
    hdr->out_of_range = any_bad ? 1 : 0;
    hdr->recount = recount;
    hdr->shift = shift;
    hdr->status = st;
    // final unless counted again
    hdr->total_tasks = (st == TC_OK && !recount) ? carry : 0;
  }
}

// Long lists only (more than kPrefixBlocks count blocks): the block counts'
// exclusive prefix into block_off in one workgroup, and, for a list counted
// again, its task count and status.
constexpr int64_t kPrefixBlocks = 16384;

__global__ __launch_bounds__(kThreads) void k_plan_offsets(const uint64_t* __restrict__ block_cnt,
                                                          uint64_t* __restrict__ block_off,
                                                          const int64_t nblocks,
                                                          const uint64_t capacity,
                                                          PlanHeader* __restrict__ hdr) {
  if (hdr->status != TC_OK) return;
  uint64_t carry = 0;
  for (int64_t base = 0; base < nblocks; base += kThreads) {
    const int64_t i = base + threadIdx.x;
    uint64_t total;
    const uint64_t ex = block_exclusive_scan(i < nblocks ? block_cnt[i] : 0, &total);
    if (i < nblocks) block_off[i] = carry + ex;
    carry += total;
  }
  if (threadIdx.x == 0 && (hdr->recount || hdr->permuted)) {
    uint64_t st = TC_OK;
    if (carry > capacity) st = TC_ERR_WORKSPACE;
    else if (carry > (uint64_t(1) << 33)) st = TC_ERR_INVALID_ARGUMENT;
    hdr->status = st;
    hdr->total_tasks = st == TC_OK ? carry : 0;
  }
}

// Per-fragment first task and the window table, for the list the header
// names, with its piece and cut.  Each workgroup takes its offset from the
// block counts: it sums those before it itself (block_off == nullptr), or
// reads k_plan_offsets' prefix for long lists.  A list counted again gets its
// task count and status here (every workgroup finds the same total; the
// first writes it).  Nothing for a failed plan.
__global__ __launch_bounds__(kThreads) void k_plan_tstart(const tc_fragment* __restrict__ given,
                                                         const tc_fragment* __restrict__ sorted,
                                                         const int64_t n, const int64_t nblocks,
                                                         PlanHeader* __restrict__ hdr,
                                                         const uint64_t* __restrict__ block_cnt,
                                                         const uint64_t* __restrict__ block_off,
                                                         const uint64_t capacity,
                                                         uint64_t* __restrict__ tstart,
                                                         int64_t* __restrict__ windows) {
  if (hdr->status != TC_OK) return;
  const bool counted_again = hdr->recount || hdr->permuted;
  uint64_t before, total;
  if (block_off) {
    before = block_off[blockIdx.x];
    total = hdr->total_tasks;
  } else {
    uint64_t b = 0, a = 0;
    for (int64_t j = threadIdx.x; j < nblocks; j += kThreads) {
      const uint64_t c = block_cnt[j];
      a += c;
      if (j < int64_t(blockIdx.x)) b += c;
    }
    block_exclusive_scan(b, &before);
    block_exclusive_scan(a, &total);
    if (counted_again) {
      uint64_t st = TC_OK;
      if (total > capacity) st = TC_ERR_WORKSPACE;
      else if (total > (uint64_t(1) << 33)) st = TC_ERR_INVALID_ARGUMENT;
      if (st != TC_OK) {
        if (blockIdx.x == 0 && threadIdx.x == 0) {
          hdr->status = st;
          hdr->total_tasks = 0;
        }
        return;
      }
      if (blockIdx.x == 0 && threadIdx.x == 0) hdr->total_tasks = total;
    }
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) tstart[n] = total;
  const tc_fragment* frags = hdr->permuted ? sorted : given;
  const uint64_t piece = hdr->piece, cut = hdr->cut;
  const int64_t f0 = int64_t(blockIdx.x) * kPlanPerBlock + int64_t(threadIdx.x) * kPlanPerThread;
  uint64_t c[kPlanPerThread];
  uint64_t s = 0;
#pragma unroll
  for (int j = 0; j < kPlanPerThread; ++j) {
    c[j] = f0 + j < n ? pieces_of(frags[f0 + j], piece, cut) : 0;
    s += c[j];
  }
  uint64_t block_total;
  uint64_t run = before + block_exclusive_scan(s, &block_total);
  const uint64_t nwin = (total + kWindowTasks - 1) / kWindowTasks;
  const int lane = threadIdx.x & (kWaveLanes - 1);
#pragma unroll
  for (int j = 0; j < kPlanPerThread; ++j) {
    const int64_t f = f0 + j;
    if (f < n) tstart[f] = run;
    // Every task lies in exactly one non-empty fragment.  The one holding
    // tasks [run, te) is therefore the first fragment of the windows whose
    // first task it holds, [ceil(run/W), ceil(te/W)), and the last fragment of
    // those whose last task (w*W + W-1, total-1 for the last window) it holds,
    // [run/W, te/W), or up to the last window when te is the total.
    uint64_t a0 = 0, a1 = 0, b0 = 0, b1 = 0;
    if (f < n && c[j]) {
      const uint64_t te = run + c[j];
      a0 = (run + kWindowTasks - 1) / kWindowTasks;
      a1 = (te + kWindowTasks - 1) / kWindowTasks;
      b0 = run / kWindowTasks;
      b1 = te == total ? nwin : te / kWindowTasks;
    }
    // A fragment spanning many windows (a large tensor) is written by its
    // whole wave, one such fragment after another.
    const bool wide = (a1 - a0) + (b1 - b0) > kWideFragmentWindows;
    if (!wide) {
      for (uint64_t w = a0; w < a1; ++w) windows[2 * w] = f;
      for (uint64_t w = b0; w < b1; ++w) windows[2 * w + 1] = f;
    }
    for (uint64_t m = __ballot(wide); m; m &= m - 1) {
      const int l = __ffsll((unsigned long long)m) - 1;
      const int64_t fl = int64_t(readlane_u64(uint64_t(f), l));
      const uint64_t la1 = readlane_u64(a1, l), lb1 = readlane_u64(b1, l);
      for (uint64_t w = readlane_u64(a0, l) + lane; w < la1; w += kWaveLanes) windows[2 * w] = fl;
      for (uint64_t w = readlane_u64(b0, l) + lane; w < lb1; w += kWaveLanes) windows[2 * w + 1] = fl;
    }
    run += c[j];
  }
}

__device__ __forceinline__ Task pack_task(uint64_t src, uint64_t dst, uint64_t len, bool first) {
  return Task{src | (dst << 48), (dst >> 16) | (len << 32) | (first ? kTaskFirst : 0)};
}


// Window j's workgroup writes tasks [j * 1024, (j + 1) * 1024), whose first
// and last fragment k_plan_tstart recorded in windows[j].  If they span at
// most 1024 fragments their tstart entries go to LDS and every task finds its
// fragment there, otherwise (long runs of empty fragments) each task searches
// globally.  A thread's four tasks are found first and their descriptors
// loaded together, so the loads overlap.  The grid is bounded by the
// workspace's capacity (the task count is only known on the device) and
// strides over the windows; workgroups past the plan's last window return.
constexpr int kExpandPerThread = kExpandPerBlock / kThreads;
static_assert(kExpandPerThread * kThreads == kExpandPerBlock, "whole tasks per thread");

__global__ __launch_bounds__(kThreads) void k_plan_expand(const tc_fragment* __restrict__ given,
                                                         const tc_fragment* __restrict__ sorted,
                                                         const uint64_t* __restrict__ tstart,
                                                         const int64_t* __restrict__ windows,
                                                         const PlanHeader* __restrict__ hdr,
                                                         Task* __restrict__ tasks) {
  __shared__ uint64_t win[kExpandPerBlock + 1];
  if (hdr->status != TC_OK) return;
  const uint64_t total = hdr->total_tasks, piece = hdr->piece, cut = hdr->cut;
  const tc_fragment* frags = hdr->permuted ? sorted : given;
  const uint64_t nwin = (total + kExpandPerBlock - 1) / kExpandPerBlock;
  for (uint64_t wj = blockIdx.x; wj < nwin; wj += gridDim.x) {
    const uint64_t t0 = wj * kExpandPerBlock;
    const uint64_t t1 = min(total, t0 + kExpandPerBlock);
    const int64_t f0 = windows[2 * wj];
    const int64_t f1 = windows[2 * wj + 1];
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
    __syncthreads();  // win is refilled by the next window
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

// The reordering passes run only when the header asks for it (permuted);
// the bucket size comes from the header too.  The counters are cleared by
// the first count.
// Bucket sizes; each fragment keeps the count it found as its rank inside
// its bucket (in no particular order), so the scatter needs no atomics.
__global__ __launch_bounds__(kThreads) void k_bucket_hist(const tc_fragment* __restrict__ frags,
                                                         const int64_t n,
                                                         const PlanHeader* __restrict__ hdr,
                                                         const uint64_t nbk,
                                                         uint64_t* __restrict__ cnt,
                                                         uint64_t* __restrict__ rank) {
  if (!hdr->permuted) return;
  const int shift = int(hdr->shift);
  for (int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * kThreads)
    rank[i] = atomicAdd(
        reinterpret_cast<unsigned long long*>(&cnt[bucket_of(frags[i].dst_off, shift, nbk)]), 1ull);
}

// Bucket offsets in two levels: each workgroup scans 1024 bucket counts in
// place (exclusive, within its block) and records the block's total; the
// scatter adds the totals of the blocks before (at most 256 of them).
__global__ __launch_bounds__(kThreads) void k_bucket_scan(const PlanHeader* __restrict__ hdr,
                                                         uint64_t* __restrict__ v, const uint64_t m,
                                                         uint64_t* __restrict__ sums) {
  if (!hdr->permuted) return;
  const uint64_t i0 = uint64_t(blockIdx.x) * kPlanPerBlock + uint64_t(threadIdx.x) * kPlanPerThread;
  uint64_t c[kPlanPerThread];
  uint64_t t = 0;
#pragma unroll
  for (int j = 0; j < kPlanPerThread; ++j) {
    c[j] = i0 + j < m ? v[i0 + j] : 0;
    t += c[j];
  }
  uint64_t total;
  uint64_t run = block_exclusive_scan(t, &total);
#pragma unroll
  for (int j = 0; j < kPlanPerThread; ++j) {
    if (i0 + j < m) v[i0 + j] = run;
    run += c[j];
  }
  if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

// Fragment i goes to its bucket's start plus its rank: the bucket's offset
// inside its block of 1024 buckets, plus the totals of the blocks before it
// (scanned here into LDS; nbk <= 2^18, so at most 256 blocks).
constexpr uint64_t kMaxBucketBlocks = kThreads;

__global__ __launch_bounds__(kThreads) void k_bucket_scatter(const tc_fragment* __restrict__ frags,
                                                            const int64_t n,
                                                            const PlanHeader* __restrict__ hdr,
                                                            const uint64_t nbk,
                                                            const uint64_t* __restrict__ off,
                                                            const uint64_t* __restrict__ sums,
                                                            const uint64_t* __restrict__ rank,
                                                            tc_fragment* __restrict__ sorted,
                                                            uint64_t* __restrict__ perm) {
  __shared__ uint64_t base[kMaxBucketBlocks];
  if (!hdr->permuted) return;
  const int shift = int(hdr->shift);
  const uint64_t nsb = (nbk + kPlanPerBlock - 1) / kPlanPerBlock;
  uint64_t total;
  const uint64_t ex = block_exclusive_scan(threadIdx.x < nsb ? sums[threadIdx.x] : 0, &total);
  if (threadIdx.x < nsb) base[threadIdx.x] = ex;
  __syncthreads();
  for (int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * kThreads) {
    const tc_fragment f = frags[i];
    const uint64_t b = bucket_of(f.dst_off, shift, nbk);
    const uint64_t pos = base[b / kPlanPerBlock] + off[b] + rank[i];
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

// Workgroups of the expansion: one per window of a plan that fills the
// workspace, at most this many (the rest stride).  Surplus workgroups read
// the header and return.
constexpr uint64_t kExpandGridCap = 16384;

hipError_t launch_plan(const tc_fragment* frags, int64_t n, void* ws, const PlanLayout& L,
                       hipStream_t s) {
  uint8_t* base = static_cast<uint8_t*>(ws);
  PlanHeader* hdr = reinterpret_cast<PlanHeader*>(base);
  uint64_t* tstart = reinterpret_cast<uint64_t*>(base + L.tstart);
  const int64_t nb = plan_blocks(n);
  uint64_t* bcnt = reinterpret_cast<uint64_t*>(base + L.blocks);
  uint64_t* blen = bcnt + nb;
  uint64_t* bunord = blen + nb;
  uint64_t* bdend = bunord + nb;
  int64_t* windows = reinterpret_cast<int64_t*>(base + L.windows);
  // the reordered list (only in layouts with buckets)
  const tc_fragment* sorted = L.nbuckets ? reinterpret_cast<const tc_fragment*>(base + L.sorted) : frags;
  uint64_t* cnt = L.nbuckets ? reinterpret_cast<uint64_t*>(base + L.buckets) : nullptr;
  const uint64_t nbk = L.nbuckets;
  const uint64_t cap = uint64_t(L.capacity);
  const PlanHeader* ch = hdr;
  // 1. count with 1 KiB pieces and the line cut (and clear the bucket
  //    counters); totals and decisions
  hipLaunchKernelGGL(k_plan_count, dim3((unsigned)nb), dim3(kThreads), 0, s, frags, sorted, n, 0, ch,
                     bcnt, blen, bunord, bdend, cnt, nbk);
  hipLaunchKernelGGL(k_plan_scan, dim3(1), dim3(kThreads), 0, s, (const uint64_t*)bcnt,
                     (const uint64_t*)blen, (const uint64_t*)bunord, (const uint64_t*)bdend, nb, n, cap,
                     nbk, hdr);
  // 2. destination order for long unordered lists (each pass checks the header)
  if (nbk) {
    static_assert((uint64_t(1) << 18) <= kMaxBucketBlocks * kPlanPerBlock, "bucket blocks fit the scatter's LDS");
    uint64_t* sums = reinterpret_cast<uint64_t*>(base + L.bucket_sums);
    tc_fragment* sorted_w = reinterpret_cast<tc_fragment*>(base + L.sorted);
    uint64_t* perm = reinterpret_cast<uint64_t*>(base + L.perm);
    // ranks live in tstart's room, which tstart rewrites after the reorder
    uint64_t* rank = tstart;
    const uint64_t sblocks = (nbk + kPlanPerBlock - 1) / kPlanPerBlock;
    const unsigned fgrid = grid_for((uint64_t(n) + kThreads - 1) / kThreads);
    hipLaunchKernelGGL(k_bucket_hist, dim3(fgrid), dim3(kThreads), 0, s, frags, n, ch, nbk, cnt, rank);
    hipLaunchKernelGGL(k_bucket_scan, dim3((unsigned)sblocks), dim3(kThreads), 0, s, ch, cnt, nbk, sums);
    hipLaunchKernelGGL(k_bucket_scatter, dim3(fgrid), dim3(kThreads), 0, s, frags, n, ch, nbk,
                       (const uint64_t*)cnt, (const uint64_t*)sums, (const uint64_t*)rank, sorted_w, perm);
  }
  // 3. count again (a reordered list, or a larger piece), only if the header asks
  hipLaunchKernelGGL(k_plan_count, dim3((unsigned)nb), dim3(kThreads), 0, s, frags, sorted, n, 1, ch,
                     bcnt, blen, bunord, bdend, (uint64_t*)nullptr, uint64_t(0));
  // 4. per-fragment first tasks and windows (long lists read a prefix of the
  //    block counts; blen is free by then), then the task table
  uint64_t* boff = nullptr;
  if (nb > kPrefixBlocks) {
    boff = blen;
    hipLaunchKernelGGL(k_plan_offsets, dim3(1), dim3(kThreads), 0, s, (const uint64_t*)bcnt, boff, nb,
                       cap, hdr);
  }
  hipLaunchKernelGGL(k_plan_tstart, dim3((unsigned)nb), dim3(kThreads), 0, s, frags, sorted, n, nb, hdr,
                     (const uint64_t*)bcnt, (const uint64_t*)boff, cap, tstart, windows);
  const uint64_t wins = (cap + kExpandPerBlock - 1) / kExpandPerBlock;
  const uint64_t egrid = wins < kExpandGridCap ? wins : kExpandGridCap;
  hipLaunchKernelGGL(k_plan_expand, dim3((unsigned)(egrid ? egrid : 1)), dim3(kThreads), 0, s, frags,
                     sorted, (const uint64_t*)tstart, (const int64_t*)windows, ch,
                     reinterpret_cast<Task*>(base + kTasksOffset));
  return hipGetLastError();
}

}  // namespace tc
