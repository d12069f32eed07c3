// Planned copies for gfx950: the fragment copy of a plan's tasks, and the
// same copy (or a read alone) with per-fragment integrity digests.
#include "tc_device.h"

namespace tc {
namespace {

// ------------------------------------------------------------------------
// Planned copy: one task per wave, four consecutive tasks per workgroup
// (workgroups of one XCD run consecutive).
// ------------------------------------------------------------------------
constexpr int kTasksPerBlock = kThreads / kWaveLanes;

// total == kTasksFromPlan: the count is read from the plan's header (a plan
// enqueued without the host knowing its size) and the grid, bounded by the
// workspace, strides over the tasks.  The grid is then a multiple of 8 XCD
// runs, so each pass over it still gives every XCD runs of consecutive tasks.
__global__ __launch_bounds__(kThreads) void k_copy_tasks(const uint8_t* __restrict__ src,
                                                        uint8_t* __restrict__ dst,
                                                        const PlanHeader* __restrict__ hdr,
                                                        const Task* __restrict__ tasks,
                                                        uint64_t total, uint64_t nblocks) {
  if (total == kTasksFromPlan) {
    total = hdr->total_tasks;
    nblocks = (total + kTasksPerBlock - 1) / kTasksPerBlock;
  }
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
    if (((sa | da | len) & 15) == 0 && len <= uint64_t(kWaveLanes) * 16) {
      // The common task: both ends 16-byte aligned, at most one vector per
      // lane, no head or tail bytes (C3 planned copy -0.4%, the storm -0.8%,
      // its one-call copy -1.6% against the general path alone).
      if (uint64_t(lane) * 16 < len) {
        const u32x4 v = ld_nt(reinterpret_cast<const u32x4*>(s) + lane);
        if (reordered)
          st_nt(reinterpret_cast<u32x4*>(d) + lane, v);
        else
          st_sc1_nt(reinterpret_cast<u32x4*>(d) + lane, v);
      }
    } else if (((sa ^ da) & 15) == 0) {
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
      // source and destination differ mod 16: realigned 16-byte vectors
      // (two stateless store functors: a lambda capturing the flag was kept
      // per lane in LDS by the compiler)
      if (reordered)
        wave_copy_any(s, d, len, lane, [](u32x4* p, u32x4 v) { st_nt(p, v); });
      else
        wave_copy_any(s, d, len, lane, [](u32x4* p, u32x4 v) { st_sc1_nt(p, v); });
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
  } else {
    // Vectors aligned on the destination when copying (on the source when
    // only reading); a copy whose source and destination differ mod 16
    // assembles each vector from the two source vectors it straddles.
    const uintptr_t anchor = kMode == kCopyDigest ? reinterpret_cast<uintptr_t>(d) : sa;
    uint64_t head = (16 - (anchor & 15)) & 15;
    if (head > len) head = len;
    const uint64_t n16 = (len - head) >> 4;
    const uint64_t body_end = head + (n16 << 4);
    const uint64_t nchunks = n16 == 0 ? 1 : (n16 + kChunkVecs - 1) / kChunkVecs;
    const uint32_t r = mis ? uint32_t((sa + head) & 15) : 0;
    const u32x4* sv = reinterpret_cast<const u32x4*>(s + head - r);
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
        const u32x4 v = r ? realign(sv[i], sv[i + 1], r) : ld_nt(sv + i);
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

}  // namespace

// Workgroups of a copy whose task count is only known on the device (a
// multiple of 8 XCD runs of the longest group, 8 x 256).  Measured on copies
// of 1.8M, 3.7M and 9.8M tasks: each further pass of a grid-stride loop costs
// a few percent against a grid of exactly one workgroup per four tasks, and
// each surplus workgroup (it reads the count and returns) about 0.2 ns;
// 2^19 workgroups came within 2%, 2% and 6% of the exact grid.  Plans in a
// smaller workspace get the grid their capacity bounds.
constexpr uint64_t kDeviceCountGrid = uint64_t(1) << 19;
static_assert(kDeviceCountGrid % (kXcds * kXcdGroupReordered) == 0, "whole XCD rounds");

hipError_t launch_copy_tasks(const uint8_t* src, uint8_t* dst, const void* ws, uint64_t total,
                             uint64_t cap_tasks, hipStream_t s) {
  if (total == 0) return hipSuccess;
  const Task* tasks = reinterpret_cast<const Task*>(static_cast<const uint8_t*>(ws) + kTasksOffset);
  uint64_t nblocks, grid;
  if (total == kTasksFromPlan) {
    nblocks = 0;  // read on the device
    const uint64_t bound = (cap_tasks + kTasksPerBlock - 1) / kTasksPerBlock;
    grid = bound < kDeviceCountGrid ? bound : kDeviceCountGrid;
    if (grid == 0) return hipSuccess;
  } else {
    nblocks = (total + kTasksPerBlock - 1) / kTasksPerBlock;
    grid = grid_for(nblocks);
  }
  hipLaunchKernelGGL(k_copy_tasks, dim3((unsigned)grid), dim3(kThreads), 0, s, src, dst,
                     static_cast<const PlanHeader*>(ws), tasks, total, nblocks);
  return hipGetLastError();
}

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
