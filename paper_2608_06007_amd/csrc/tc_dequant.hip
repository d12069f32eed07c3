// The inverse of the block-scaled cast for gfx950: E4M3 codes with one fp32
// scale per 128x128 tile back to bf16, y = RN_bf16(RN_f32(value(q) * s)).
//
// Layout mirrors the cast: full tiles of aligned items with 16 lanes x 8
// codes per 128-byte code row (8 bf16 = 16 B stored per lane and row),
// non-temporal loads and stores, XCD groups of 4 tiles -- a quarter tile per
// 256-thread workgroup when a per-tile table gives each tile's addresses,
// else the whole tile per 512-thread workgroup after an item search; partial
// tiles and unaligned items go to an element-wise kernel.  Decoding uses v_cvt_pk_f32_fp8, which is exact for
// every finite E4M3 code and gives NaN for S.1111.111; the bf16 rounding is
// done on the integer bits (nearest, ties to even; NaN -> 0x7FC0).
#include "tc_device.h"

namespace tc {
namespace {

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// bf16 stores are st_sc1_nt: SC1 NT measured 5809 against 5709 GB/s with
// plain NT stores on the 70B shard.

constexpr int kTile = 128;
constexpr int kDequantThreads = 512;
constexpr int kRowsPerPass = kDequantThreads / 16;
constexpr int kPasses = kTile / kRowsPerPass;
constexpr uint64_t kDequantXcdGroup = 4;  // consecutive tiles per XCD run

// bf16 bits of a binary32 value: nearest, ties to even; NaN -> 0x7FC0.
__device__ __forceinline__ uint32_t bf16_bits(float v) {
  const uint32_t u = __float_as_uint(v);
  const uint32_t r = (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
  return (u & 0x7FFFFFFFu) > 0x7F800000u ? 0x7FC0u : r;
}

// Four codes (one 32-bit word) -> four bf16 (two 32-bit words).
__device__ __forceinline__ u32x2 dequant4(uint32_t w, float s) {
  const f32x2 a = __builtin_amdgcn_cvt_pk_f32_fp8((int)w, false);
  const f32x2 b = __builtin_amdgcn_cvt_pk_f32_fp8((int)w, true);
  return u32x2{bf16_bits(a.x * s) | (bf16_bits(a.y * s) << 16),
               bf16_bits(b.x * s) | (bf16_bits(b.y * s) << 16)};
}

// One full tile by one workgroup: qs and ys point at the tile's first code
// and first bf16 element, src_ld and dst_ld are the row pitches, s the scale.
__device__ __forceinline__ void dequant_tile(const uint8_t* __restrict__ qs, uint16_t* __restrict__ ys,
                                             const int64_t src_ld, const int64_t dst_ld, const float s) {
  const int seg = threadIdx.x & 15;  // 8 codes per lane, 16 lanes per 128-byte row
  const int prow = threadIdx.x >> 4;
  u32x2 v[kPasses];
#pragma unroll
  for (int p = 0; p < kPasses; ++p)
    v[p] = __builtin_nontemporal_load(
        reinterpret_cast<const u32x2*>(qs + int64_t(p * kRowsPerPass + prow) * src_ld + seg * 8));
#pragma unroll
  for (int p = 0; p < kPasses; ++p) {
    const u32x2 lo = dequant4(v[p].x, s), hi = dequant4(v[p].y, s);
    st_sc1_nt(reinterpret_cast<u32x4*>(ys + int64_t(p * kRowsPerPass + prow) * dst_ld + seg * 8),
              u32x4{lo.x, lo.y, hi.x, hi.y});
  }
}

__global__ __launch_bounds__(kDequantThreads) void k_dequant_full(const uint8_t* __restrict__ codes,
                                                          const float* __restrict__ scales,
                                                          uint16_t* __restrict__ dst,
                                                          const tc_dequant_item* __restrict__ items,
                                                          const uint64_t* __restrict__ prefix,
                                                          const int64_t n_items, const uint64_t t0,
                                                          const uint64_t count) {
  const int lane = threadIdx.x & (kWaveLanes - 1);
  const uint64_t t = t0 + xcd_grouped(blockIdx.x, count, kDequantXcdGroup);
  const int64_t it = find_item(prefix, n_items, t, lane);
  const tc_dequant_item item = items[it];
  const int64_t full_c = item.cols / kTile;
  const int64_t local = int64_t(t - prefix[it]);
  const int64_t ti = local / full_c, tj = local - ti * full_c;
  dequant_tile(codes + item.src_off + ti * kTile * item.src_ld + tj * kTile,
               dst + item.dst_off + ti * kTile * item.dst_ld + tj * kTile, item.src_ld, item.dst_ld,
               scales[item.scale_off + ti * item.scale_ld + tj]);
}

// The tiles of a per-tile table, a quarter tile per workgroup: 256 threads
// take 32 rows (two passes of 16 rows, one 8-byte code load and one 16-byte
// store per lane and pass).  With the table a workgroup finds its tile in one
// load, so the dependent chain the whole-tile unit amortized (item search,
// item, scale) is gone; the slabs of a tile share its entry and scale.
// Measured on the 70B TP=8 shard, interleaved in one process: 6260-6274 GB/s
// against 5932-5951 for the whole tile per 512-thread workgroup from the same
// table (16-row slabs of 128 threads: 6264-6274; 64 rows of 512 threads:
// 6100-6113; XCD runs of 2 or 8 tiles: 5984-5994, 6188-6213).
constexpr int kSlabs = 4;
constexpr int kSlabThreads = 256;
constexpr int kSlabRows = kTile / kSlabs;
constexpr int kSlabRowsPerPass = kSlabThreads / 16;
constexpr int kSlabPasses = kSlabRows / kSlabRowsPerPass;
static_assert(kSlabPasses * kSlabRowsPerPass == kSlabRows, "whole passes per slab");
constexpr uint64_t kSlabTilesPerLaunch = kMaxGrid / kSlabs;

__global__ __launch_bounds__(kSlabThreads) void k_dequant_slab_tab(const uint8_t* __restrict__ codes,
                                                                  const float* __restrict__ scales,
                                                                  uint16_t* __restrict__ dst,
                                                                  const TileEntry* __restrict__ tab,
                                                                  const uint64_t t0, const uint64_t count) {
  const uint64_t u = xcd_grouped(blockIdx.x, count * kSlabs, kDequantXcdGroup * kSlabs);
  const TileEntry e = tab[t0 + u / kSlabs];
  const int64_t r0 = int64_t(u % kSlabs) * kSlabRows;
  const int64_t src_ld = int64_t(uint32_t(e.lds)), dst_ld = int64_t(e.lds >> 32);
  const uint8_t* qs = codes + e.in_off + r0 * src_ld;
  uint16_t* ys = dst + e.out_off + r0 * dst_ld;
  const int seg = threadIdx.x & 15;
  const int prow = threadIdx.x >> 4;
  u32x2 v[kSlabPasses];
#pragma unroll
  for (int p = 0; p < kSlabPasses; ++p)
    v[p] = __builtin_nontemporal_load(
        reinterpret_cast<const u32x2*>(qs + int64_t(p * kSlabRowsPerPass + prow) * src_ld + seg * 8));
  const float s = scales[e.scale_idx];
#pragma unroll
  for (int p = 0; p < kSlabPasses; ++p) {
    const u32x2 lo = dequant4(v[p].x, s), hi = dequant4(v[p].y, s);
    st_sc1_nt(reinterpret_cast<u32x4*>(ys + int64_t(p * kSlabRowsPerPass + prow) * dst_ld + seg * 8),
              u32x4{lo.x, lo.y, hi.x, hi.y});
  }
}

// Partial tiles and unaligned items, element by element; numbered within an
// item like the cast's edge tiles.
__global__ __launch_bounds__(kDequantThreads) void k_dequant_edge(const uint8_t* __restrict__ codes,
                                                          const float* __restrict__ scales,
                                                          uint16_t* __restrict__ dst,
                                                          const tc_dequant_item* __restrict__ items,
                                                          const uint64_t* __restrict__ prefix,
                                                          const uint8_t* __restrict__ aligned,
                                                          const int64_t n_items, const uint64_t t0) {
  const int lane = threadIdx.x & (kWaveLanes - 1);
  const uint64_t t = t0 + blockIdx.x;
  const int64_t it = find_item(prefix, n_items, t, lane);
  const tc_dequant_item item = items[it];
  const int64_t tr = (item.rows + kTile - 1) / kTile, tcn = (item.cols + kTile - 1) / kTile;
  const int64_t fr = aligned[it] ? item.rows / kTile : 0;
  const int64_t fc = aligned[it] ? item.cols / kTile : 0;
  const int64_t e = int64_t(t - prefix[it]);
  int64_t ti, tj;
  if (e < (tr - fr) * tcn) {
    ti = fr + e / tcn;
    tj = e % tcn;
  } else {
    const int64_t e2 = e - (tr - fr) * tcn;
    ti = e2 / (tcn - fc);
    tj = fc + e2 % (tcn - fc);
  }
  const int64_t r0 = ti * kTile, c0 = tj * kTile;
  const int64_t h = min<int64_t>(kTile, item.rows - r0);
  const int64_t wd = min<int64_t>(kTile, item.cols - c0);
  const uint8_t* qs = codes + item.src_off + r0 * item.src_ld + c0;
  uint16_t* ys = dst + item.dst_off + r0 * item.dst_ld + c0;
  const float s = scales[item.scale_off + ti * item.scale_ld + tj];
  for (int64_t k = threadIdx.x; k < h * wd; k += kDequantThreads) {
    const int64_t rr = k / wd, cc = k - rr * wd;
    const f32x2 v = __builtin_amdgcn_cvt_pk_f32_fp8((int)qs[rr * item.src_ld + cc], false);
    ys[rr * item.dst_ld + cc] = (uint16_t)bf16_bits(v.x * s);
  }
}

}  // namespace

hipError_t launch_dequant_blockscaled(const uint8_t* codes, const float* scales, uint16_t* dst,
                                      const void* ws, int64_t n_items, uint64_t full_tiles,
                                      uint64_t edge_tiles, bool tiled, hipStream_t s) {
  const CastLayout L = cast_layout(n_items);
  const uint8_t* base = static_cast<const uint8_t*>(ws);
  const tc_dequant_item* items = reinterpret_cast<const tc_dequant_item*>(base + L.items);
  const uint64_t* fp = reinterpret_cast<const uint64_t*>(base + L.full_prefix);
  const uint64_t* ep = reinterpret_cast<const uint64_t*>(base + L.edge_prefix);
  const uint8_t* al = base + L.aligned;
  const TileEntry* tab = reinterpret_cast<const TileEntry*>(base + L.bytes);
  if (tiled) {
    for (uint64_t t0 = 0; t0 < full_tiles; t0 += kSlabTilesPerLaunch) {
      const uint64_t cnt = full_tiles - t0 < kSlabTilesPerLaunch ? full_tiles - t0 : kSlabTilesPerLaunch;
      hipLaunchKernelGGL(k_dequant_slab_tab, dim3((unsigned)(cnt * kSlabs)), dim3(kSlabThreads), 0, s, codes,
                         scales, dst, tab, t0, cnt);
    }
  } else {
    for (uint64_t t0 = 0; t0 < full_tiles; t0 += kMaxGrid) {
      const uint64_t cnt = full_tiles - t0 < kMaxGrid ? full_tiles - t0 : kMaxGrid;
      hipLaunchKernelGGL(k_dequant_full, dim3((unsigned)cnt), dim3(kDequantThreads), 0, s, codes, scales,
                         dst, items, fp, n_items, t0, cnt);
    }
  }
  for (uint64_t t0 = 0; t0 < edge_tiles; t0 += kMaxGrid) {
    const uint64_t cnt = edge_tiles - t0 < kMaxGrid ? edge_tiles - t0 : kMaxGrid;
    hipLaunchKernelGGL(k_dequant_edge, dim3((unsigned)cnt), dim3(kDequantThreads), 0, s, codes, scales, dst,
                       items, ep, al, n_items, t0);
  }
  return hipGetLastError();
}

}  // namespace tc
