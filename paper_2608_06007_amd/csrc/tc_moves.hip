// Byte movers for gfx950: paged-KV block gather/scatter (publish / hydrate)
// and planned fragment copies (prefetch_many, materialization transfer).
//
// All of it is HBM-bound streaming.  Every lane moves 16-byte vectors, a
// wave keeps several of them in flight before it stores, and work is cut
// so that every workgroup / wave moves a similar number of bytes.
#include "tc_internal.h"

namespace tc {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;      // 4 waves of 64 lanes
constexpr int kWaveLanes = 64;

__device__ __forceinline__ int wave_id_in_block() {
  return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
}

// ------------------------------------------------------------------------
// Block gather / scatter.  One workgroup tile = 256 lanes x 16 B x U of one
// (id, region) chunk; a chunk of block_bytes is covered by tiles_per_chunk
// tiles.  Workgroup w handles tile w (grid-stride if the grid is capped).
// ------------------------------------------------------------------------
template <int U, bool kGather>
__global__ __launch_bounds__(kThreads) void k_blocks_vec(const RegionTable tab, const int32_t R,
                                                        const int64_t B, const int64_t stride,
                                                        const int32_t* __restrict__ ids,
                                                        const int64_t total_tiles,
                                                        const int64_t tiles_per_chunk,
                                                        uint8_t* __restrict__ buf) {
  constexpr int64_t kTileBytes = int64_t(kThreads) * 16 * U;
  for (int64_t w = blockIdx.x; w < total_tiles; w += gridDim.x) {
    const int64_t c = w / tiles_per_chunk;  // chunk index = i * R + r
    const int64_t k = w - c * tiles_per_chunk;
    const int64_t i = c / R;
    const int32_t r = (int32_t)(c - i * R);
    const int64_t id = ids[i];
    uint8_t* pool = reinterpret_cast<uint8_t*>(tab.base[r]) + id * stride;
    uint8_t* xfer = buf + c * B;
    const uint8_t* from = kGather ? pool : xfer;
    uint8_t* to = kGather ? xfer : pool;
    const int64_t off0 = k * kTileBytes + int64_t(threadIdx.x) * 16;
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t off = off0 + int64_t(u) * kThreads * 16;
      if (off < B) v[u] = *reinterpret_cast<const u32x4*>(from + off);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t off = off0 + int64_t(u) * kThreads * 16;
      if (off < B) *reinterpret_cast<u32x4*>(to + off) = v[u];
    }
  }
}

// Byte-granular variant for pools whose bases, stride or block size are not
// 16-byte multiples.
template <bool kGather>
__global__ __launch_bounds__(kThreads) void k_blocks_bytes(const RegionTable tab, const int32_t R,
                                                          const int64_t B, const int64_t stride,
                                                          const int32_t* __restrict__ ids,
                                                          const int64_t n_chunks,
                                                          uint8_t* __restrict__ buf) {
  for (int64_t c = blockIdx.x; c < n_chunks; c += gridDim.x) {
    const int64_t i = c / R;
    const int32_t r = (int32_t)(c - i * R);
    uint8_t* pool = reinterpret_cast<uint8_t*>(tab.base[r]) + int64_t(ids[i]) * stride;
    uint8_t* xfer = buf + c * B;
    const uint8_t* from = kGather ? pool : xfer;
    uint8_t* to = kGather ? xfer : pool;
    for (int64_t b = threadIdx.x; b < B; b += kThreads) to[b] = from[b];
  }
}

constexpr int kBlockUnroll = 4;  // 16 KiB per workgroup tile

// ------------------------------------------------------------------------
// Fragment plan.  Fragment f is cut into ceil(len / kPieceBytes) pieces
// ("tasks"); tstart[f] is the index of its first task and tstart[n] the
// total.  Three small passes: per-block task sums, an exclusive scan of the
// block sums (one workgroup), and the per-fragment prefix.
// ------------------------------------------------------------------------
__device__ __forceinline__ uint64_t pieces_of(uint64_t len) {
  return (len + kPieceBytes - 1) / kPieceBytes;
}

__device__ __forceinline__ uint64_t shfl_up_u64(uint64_t v, int delta) {
  const uint32_t lo = __shfl_up((uint32_t)v, delta, kWaveLanes);
  const uint32_t hi = __shfl_up((uint32_t)(v >> 32), delta, kWaveLanes);
  return (uint64_t(hi) << 32) | lo;
}

// Inclusive scan within a wave.
__device__ __forceinline__ uint64_t wave_inclusive_scan(uint64_t v, int lane) {
#pragma unroll
  for (int d = 1; d < kWaveLanes; d <<= 1) {
    const uint64_t o = shfl_up_u64(v, d);
    if (lane >= d) v += o;
  }
  return v;
}

// Exclusive scan over a 256-thread block; *block_total receives the sum.
__device__ uint64_t block_exclusive_scan(uint64_t v, uint64_t* block_total) {
  __shared__ uint64_t wave_tot[kThreads / kWaveLanes];
  const int lane = threadIdx.x & (kWaveLanes - 1);
  const int w = threadIdx.x >> 6;
  const uint64_t incl = wave_inclusive_scan(v, lane);
  if (lane == kWaveLanes - 1) wave_tot[w] = incl;
  __syncthreads();
  uint64_t before = 0, total = 0;
#pragma unroll
  for (int k = 0; k < kThreads / kWaveLanes; ++k) {
    if (k < w) before += wave_tot[k];
    total += wave_tot[k];
  }
  __syncthreads();  // wave_tot may be reused by the caller's next scan
  *block_total = total;
  return before + incl - v;
}

constexpr int kPlanPerThread = kPlanPerBlock / kThreads;  // 4

__global__ __launch_bounds__(kThreads) void k_plan_count(const tc_fragment* __restrict__ frags,
                                                        const int64_t n,
                                                        uint64_t* __restrict__ block_sum) {
  const int64_t f0 = int64_t(blockIdx.x) * kPlanPerBlock + int64_t(threadIdx.x) * kPlanPerThread;
  uint64_t s = 0;
#pragma unroll
  for (int j = 0; j < kPlanPerThread; ++j)
    if (f0 + j < n) s += pieces_of(frags[f0 + j].len);
  uint64_t total;
  block_exclusive_scan(s, &total);
  if (threadIdx.x == 0) block_sum[blockIdx.x] = total;
}

// One workgroup: block_sum[0..nblocks) becomes its exclusive prefix, and
// *grand_total the sum of all of it.
__global__ __launch_bounds__(kThreads) void k_plan_scan(uint64_t* __restrict__ block_sum,
                                                       const int64_t nblocks,
                                                       uint64_t* __restrict__ grand_total) {
  uint64_t carry = 0;
  for (int64_t base = 0; base < nblocks; base += kThreads) {
    const int64_t i = base + threadIdx.x;
    const uint64_t v = i < nblocks ? block_sum[i] : 0;
    uint64_t total;
    const uint64_t ex = block_exclusive_scan(v, &total);
    if (i < nblocks) block_sum[i] = carry + ex;
    carry += total;
  }
  if (threadIdx.x == 0) *grand_total = carry;
}

__global__ __launch_bounds__(kThreads) void k_plan_write(const tc_fragment* __restrict__ frags,
                                                        const int64_t n,
                                                        const uint64_t* __restrict__ block_off,
                                                        uint64_t* __restrict__ tstart) {
  const int64_t f0 = int64_t(blockIdx.x) * kPlanPerBlock + int64_t(threadIdx.x) * kPlanPerThread;
  uint64_t c[kPlanPerThread];
  uint64_t s = 0;
#pragma unroll
  for (int j = 0; j < kPlanPerThread; ++j) {
    c[j] = f0 + j < n ? pieces_of(frags[f0 + j].len) : 0;
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

// ------------------------------------------------------------------------
// Planned copy.  A persistent grid of waves walks the task list in chunks
// of kTasksPerChunk consecutive tasks (chunk c goes to wave c mod #waves);
// the chunk's first fragment is found with a 64-way search of tstart.
// ------------------------------------------------------------------------

// Last f in [0, n) with tstart[f] <= t, given tstart[0] <= t < tstart[n].
__device__ int64_t find_fragment(const uint64_t* __restrict__ tstart, int64_t n, uint64_t t,
                                 int lane) {
  int64_t lo = 0, hi = n;
  while (hi - lo > 1) {
    const int64_t step = (hi - lo + kWaveLanes - 1) / kWaveLanes;
    const int64_t p = lo + (int64_t(lane) + 1) * step;
    const bool pred = lane < kWaveLanes - 1 && p < hi && tstart[p] <= t;
    const int64_t cnt = __popcll(__ballot(pred));
    lo += cnt * step;
    hi = min(hi, lo + step);
  }
  return lo;
}

// Copy len bytes with one wave.  Source and destination with the same
// address residue mod 16 take the vector path (byte head and tail around
// 16-byte vectors, U vectors in flight per lane); others go byte by byte.
template <int U>
__device__ __forceinline__ void wave_copy(const uint8_t* s, uint8_t* d, uint64_t len, int lane) {
  const uintptr_t sa = reinterpret_cast<uintptr_t>(s);
  const uintptr_t da = reinterpret_cast<uintptr_t>(d);
  if (((sa ^ da) & 15) == 0) {
    uint64_t head = (16 - (sa & 15)) & 15;
    if (head > len) head = len;
    if (uint64_t(lane) < head) d[lane] = s[lane];
    s += head;
    d += head;
    len -= head;
    const uint64_t n16 = len >> 4;
    const u32x4* sv = reinterpret_cast<const u32x4*>(s);
    u32x4* dv = reinterpret_cast<u32x4*>(d);
    uint64_t i = lane;
    for (; i + uint64_t(kWaveLanes) * (U - 1) < n16; i += uint64_t(kWaveLanes) * U) {
      u32x4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) v[u] = sv[i + u * kWaveLanes];
#pragma unroll
      for (int u = 0; u < U; ++u) dv[i + u * kWaveLanes] = v[u];
    }
    for (; i < n16; i += kWaveLanes) dv[i] = sv[i];
    const uint64_t tail = len & 15;
    if (uint64_t(lane) < tail) d[(n16 << 4) + lane] = s[(n16 << 4) + lane];
  } else {
    for (uint64_t i = lane; i < len; i += kWaveLanes) d[i] = s[i];
  }
}

constexpr int kCopyUnroll = 8;

__global__ __launch_bounds__(kThreads) void k_copy_planned(const uint8_t* __restrict__ src,
                                                          uint8_t* __restrict__ dst,
                                                          const tc_fragment* __restrict__ frags,
                                                          const int64_t n,
                                                          const uint64_t* __restrict__ tstart) {
  const int lane = threadIdx.x & (kWaveLanes - 1);
  const int64_t nwaves = int64_t(gridDim.x) * (kThreads / kWaveLanes);
  const int64_t wave = int64_t(blockIdx.x) * (kThreads / kWaveLanes) + wave_id_in_block();
  const uint64_t total = tstart[n];
  const uint64_t nchunks = (total + kTasksPerChunk - 1) / kTasksPerChunk;
  for (uint64_t ch = wave; ch < nchunks; ch += nwaves) {
    const uint64_t t0 = ch * kTasksPerChunk;
    const uint64_t t1 = min(t0 + kTasksPerChunk, total);
    int64_t f = find_fragment(tstart, n, t0, lane);
    for (uint64_t t = t0; t < t1; ++t) {
      while (tstart[f + 1] <= t) ++f;  // stops at f = n-1 at the latest
      const uint64_t off = (t - tstart[f]) * kPieceBytes;
      const uint64_t flen = frags[f].len;
      const uint64_t len = min(kPieceBytes, flen - off);
      wave_copy<kCopyUnroll>(src + frags[f].src_off + off, dst + frags[f].dst_off + off, len,
                             lane);
    }
  }
}

int g_copy_blocks_per_cu = 0;

}  // namespace

// ------------------------------------------------------------------------
hipError_t launch_blocks(const RegionTable& tab, int32_t R, int64_t B, int64_t stride,
                         const int32_t* ids, int64_t n, uint8_t* buf, bool gather, bool aligned,
                         hipStream_t s) {
  const int64_t chunks = n * R;
  const int64_t cap = int64_t(1) << 30;
  if (aligned) {
    constexpr int64_t kTile = int64_t(kThreads) * 16 * kBlockUnroll;
    const int64_t tpc = (B + kTile - 1) / kTile;
    const int64_t total = chunks * tpc;
    const unsigned grid = (unsigned)(total < cap ? total : cap);
    if (gather)
      hipLaunchKernelGGL((k_blocks_vec<kBlockUnroll, true>), dim3(grid), dim3(kThreads), 0, s, tab,
                         R, B, stride, ids, total, tpc, buf);
    else
      hipLaunchKernelGGL((k_blocks_vec<kBlockUnroll, false>), dim3(grid), dim3(kThreads), 0, s,
                         tab, R, B, stride, ids, total, tpc, buf);
  } else {
    const unsigned grid = (unsigned)(chunks < cap ? chunks : cap);
    if (gather)
      hipLaunchKernelGGL((k_blocks_bytes<true>), dim3(grid), dim3(kThreads), 0, s, tab, R, B,
                         stride, ids, chunks, buf);
    else
      hipLaunchKernelGGL((k_blocks_bytes<false>), dim3(grid), dim3(kThreads), 0, s, tab, R, B,
                         stride, ids, chunks, buf);
  }
  return hipGetLastError();
}

static int64_t plan_blocks(int64_t n) { return (n + kPlanPerBlock - 1) / kPlanPerBlock; }

size_t frag_workspace_bytes(int64_t n) {
  return size_t(8) * size_t(n + 1) + size_t(8) * size_t(plan_blocks(n)) + 256;
}

static uint64_t* ws_tstart(void* ws) { return reinterpret_cast<uint64_t*>(ws); }
static uint64_t* ws_blocks(void* ws, int64_t n) { return reinterpret_cast<uint64_t*>(ws) + (n + 1); }

hipError_t launch_plan_fragments(const tc_fragment* frags, int64_t n, void* ws, hipStream_t s) {
  const int64_t nb = plan_blocks(n);
  uint64_t* tstart = ws_tstart(ws);
  uint64_t* bsum = ws_blocks(ws, n);
  hipLaunchKernelGGL(k_plan_count, dim3((unsigned)nb), dim3(kThreads), 0, s, frags, n, bsum);
  hipLaunchKernelGGL(k_plan_scan, dim3(1), dim3(kThreads), 0, s, bsum, nb, tstart + n);
  hipLaunchKernelGGL(k_plan_write, dim3((unsigned)nb), dim3(kThreads), 0, s, frags, n,
                     (const uint64_t*)bsum, tstart);
  return hipGetLastError();
}

hipError_t launch_copy_planned(const uint8_t* src, uint8_t* dst, const tc_fragment* frags,
                               int64_t n, const void* ws, const DeviceInfo& di, hipStream_t s) {
  if (g_copy_blocks_per_cu == 0) {
    int per_cu = 0;
    hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_copy_planned, kThreads, 0);
    if (e != hipSuccess) return e;
    g_copy_blocks_per_cu = per_cu > 0 ? per_cu : 1;
  }
  const unsigned grid = (unsigned)(di.cus * g_copy_blocks_per_cu);
  hipLaunchKernelGGL(k_copy_planned, dim3(grid), dim3(kThreads), 0, s, src, dst, frags, n,
                     (const uint64_t*)ws);
  return hipGetLastError();
}

}  // namespace tc
