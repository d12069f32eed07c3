// bf16 -> fp8 E4M3 cast with one fp32 scale per 128x128 tile (a
// transform_into rule for weight synchronization), for gfx950.
//
// Per tile: amax from the bf16 bit patterns (|x| as a 15-bit integer, so
// Inf/NaN are caught by the same max), s = amax / 448 (correctly rounded),
// then q = E4M3(RN(x / s)).
//
// Quotient without a division per element: with r = RN(1/s) (normal s),
// q0 = RN(x * r) differs from RN(x / s) by at most ~1.5 * 2^-23 relative.
// lo = RN(q0 * (1 - 2^-20)) and hi = RN(q0 * (1 + 2^-20)) bracket RN(x / s),
// and the E4M3 rounding is monotonic, so when lo and hi convert to the same
// code that code is E4M3(RN(x / s)).  Otherwise (within ~2^-20 of a rounding
// midpoint, about one element in 65536) the element is redone with a true
// division.  Subnormal scales (tiny amax) use the division throughout.
//
// Conversion: v_cvt_pk_fp8_f32 rounds to nearest even into the OCP E4M3
// format.  For |v| < 464 it equals the saturating E4M3 rounding; the
// quotients of a finite tile stay below 449 (|x| <= amax and s is amax/448
// rounded to nearest, worst case a subnormal s with 8 significant bits), and
// lo/hi stay below 450, so no clamp is needed on this path.
#include "tc_device.h"

namespace tc {
namespace {

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));

constexpr int kTile = 128;

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Two E4M3 codes packed into bits [15:0] (word 0) or [31:16] (word 1) of old.
template <bool kHiWord>
__device__ __forceinline__ uint32_t cvt2(float a, float b, uint32_t old) {
  return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(a, b, (int)old, kHiWord);
}

// Max of |bf16| over the two halves of w, as 15-bit integers (packed u16 max).
__device__ __forceinline__ uint32_t absmax2(uint32_t acc, uint32_t w) {
  const u16x2 a = __builtin_bit_cast(u16x2, acc);
  const u16x2 b = __builtin_bit_cast(u16x2, w & 0x7FFF7FFFu);
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(a, b));
}

// Four codes of RN(x/s) for the bf16 pairs in words w0 (elements 0,1) and
// w1 (elements 2,3), division-free unless near a rounding midpoint.
__device__ __forceinline__ uint32_t codes4_fast(uint32_t w0, uint32_t w1, float r, float s) {
  const float x0 = bf16_lo(w0), x1 = bf16_hi(w0), x2 = bf16_lo(w1), x3 = bf16_hi(w1);
  const float q0 = x0 * r, q1 = x1 * r, q2 = x2 * r, q3 = x3 * r;
  constexpr float kDown = 1.0f - 0x1.0p-20f;
  constexpr float kUp = 1.0f + 0x1.0p-20f;
  uint32_t lo = cvt2<false>(q0 * kDown, q1 * kDown, 0);
  lo = cvt2<true>(q2 * kDown, q3 * kDown, lo);
  uint32_t hi = cvt2<false>(q0 * kUp, q1 * kUp, 0);
  hi = cvt2<true>(q2 * kUp, q3 * kUp, hi);
  if (lo != hi) {
    // Near a rounding midpoint: use the correctly rounded quotient.
    lo = cvt2<false>(x0 / s, x1 / s, 0);
    lo = cvt2<true>(x2 / s, x3 / s, lo);
  }
  return lo;
}

// Four codes of RN(x/s) with a true division per element.
__device__ __forceinline__ uint32_t codes4_div(uint32_t w0, uint32_t w1, float s) {
  uint32_t c = cvt2<false>(bf16_lo(w0) / s, bf16_hi(w0) / s, 0);
  return cvt2<true>(bf16_lo(w1) / s, bf16_hi(w1) / s, c);
}

// Codes when the tile's amax is 0: only the sign bits survive.
__device__ __forceinline__ uint32_t codes4_zero(uint32_t w0, uint32_t w1) {
  return ((w0 >> 8) & 0x80u) | ((w0 >> 16) & 0x8000u) | ((w1 << 8) & 0x800000u) |
         (w1 & 0x80000000u);
}

// Single-element code for the generic path (same rules as the tile path).
__device__ __forceinline__ uint8_t code1(uint16_t bits, int mode, float s) {
  // mode 0: finite tile, 1: zero tile, 2: non-finite tile
  if (mode == 2) return 0x7F;
  if (mode == 1) return (bits & 0x8000u) ? 0x80 : 0x00;
  const float q = __uint_as_float(uint32_t(bits) << 16) / s;
  return (uint8_t)(cvt2<false>(q, q, 0) & 0xFFu);
}

// One 128x128 tile per workgroup of 512 threads: 32 elements (4 x 16 B) per
// thread, 16 threads per 256-byte row, 32 rows per pass, 4 passes.
constexpr int kCastThreads = 512;
constexpr int kCastWaves = kCastThreads / kWaveLanes;
constexpr int kRowsPerPass = kCastThreads / 16;
constexpr int kPasses = kTile / kRowsPerPass;
constexpr uint64_t kCastXcdGroup = 4;  // consecutive tiles per XCD run

// Code stores carry the SC1 scope bit with NT, as the copies' stores do
// (measured on the 70B shard: 5867 against 5841 GB/s with plain NT).
__device__ __forceinline__ void st_codes(u32x2* p, u32x2 v) {
  asm volatile("global_store_dwordx2 %0, %1, off sc1 nt" ::"v"(p), "v"(v) : "memory");
}

// Maximum of v over the 64 lanes of a wave (all lanes active): DPP maxima
// within each row of 16 lanes (swap neighbours, swap pairs, mirror halves,
// mirror the row), then the four row maxima read into scalars.  A butterfly
// of __shfl_xor compiled to six dependent ds_bpermute round trips; this
// measured +1.3% on the C4 shard cast (one GPU, the two builds interleaved).
__device__ __forceinline__ uint32_t wave_max32(uint32_t v) {
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false));  // row_half_mirror
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false));  // row_mirror
  return max(max((uint32_t)__builtin_amdgcn_readlane((int)v, 0), (uint32_t)__builtin_amdgcn_readlane((int)v, 16)),
             max((uint32_t)__builtin_amdgcn_readlane((int)v, 32), (uint32_t)__builtin_amdgcn_readlane((int)v, 48)));
}

// Reduce a per-thread 15-bit amax over the workgroup (one tile per
// workgroup, so red is written once).
__device__ __forceinline__ uint32_t block_amax(uint32_t m, uint32_t* red) {
  m = wave_max32(m);
  if ((threadIdx.x & (kWaveLanes - 1)) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  uint32_t r = 0;
#pragma unroll
  for (int k = 0; k < kCastWaves; ++k) r = max(r, red[k]);
  return r;
}

// One full 128x128 tile by one workgroup: xs and qs point at the tile's
// first source element and first code, src_ld and dst_ld are the row
// pitches, *scale receives the tile's scale.
__device__ __forceinline__ void cast_tile(const uint16_t* __restrict__ xs, uint8_t* __restrict__ qs,
                                          const int64_t src_ld, const int64_t dst_ld,
                                          float* __restrict__ scale, uint32_t* red) {
  const int seg = threadIdx.x & 15;  // 16 lanes per 256-byte row (8 bf16 = 16 B each)
  const int prow = threadIdx.x >> 4;
  u32x4 v[kPasses];
#pragma unroll
  for (int p = 0; p < kPasses; ++p)
    v[p] = ld_nt(reinterpret_cast<const u32x4*>(xs + int64_t(p * kRowsPerPass + prow) * src_ld + seg * 8));
  uint32_t m2 = 0;
#pragma unroll
  for (int p = 0; p < kPasses; ++p) {
    m2 = absmax2(m2, v[p].x);
    m2 = absmax2(m2, v[p].y);
    m2 = absmax2(m2, v[p].z);
    m2 = absmax2(m2, v[p].w);
  }
  const uint32_t amax_bits = block_amax(max(m2 & 0xFFFFu, m2 >> 16), red);
  float s;
  u32x2 o[kPasses];
  if (amax_bits >= 0x7F80u) {  // Inf or NaN in the tile
    s = __uint_as_float(0x7FC00000u);
#pragma unroll
    for (int p = 0; p < kPasses; ++p) o[p] = u32x2{0x7F7F7F7Fu, 0x7F7F7F7Fu};
  } else if (amax_bits == 0) {
    s = 0.0f;
#pragma unroll
    for (int p = 0; p < kPasses; ++p) o[p] = u32x2{codes4_zero(v[p].x, v[p].y), codes4_zero(v[p].z, v[p].w)};
  } else {
    s = __uint_as_float(amax_bits << 16) / 448.0f;
    if (s >= 0x1.0p-126f) {
      const float r = 1.0f / s;
#pragma unroll
      for (int p = 0; p < kPasses; ++p)
        o[p] = u32x2{codes4_fast(v[p].x, v[p].y, r, s), codes4_fast(v[p].z, v[p].w, r, s)};
    } else {
#pragma unroll
      for (int p = 0; p < kPasses; ++p)
        o[p] = u32x2{codes4_div(v[p].x, v[p].y, s), codes4_div(v[p].z, v[p].w, s)};
    }
  }
#pragma unroll
  for (int p = 0; p < kPasses; ++p)
    st_codes(reinterpret_cast<u32x2*>(qs + int64_t(p * kRowsPerPass + prow) * dst_ld + seg * 8), o[p]);
  if (threadIdx.x == 0) *scale = s;
}

// Full tiles of items whose rows are 16-byte aligned (source) and 8-byte
// aligned (codes): one workgroup per tile, tile t0 + (XCD-grouped block).
// prefix counts each item's full tiles (rows/128 x cols/128, or 0).
__global__ __launch_bounds__(kCastThreads) void k_cast_full(const uint16_t* __restrict__ src,
                                                           uint8_t* __restrict__ dst,
                                                           float* __restrict__ scales,
                                                           const tc_cast_item* __restrict__ items,
                                                           const uint64_t* __restrict__ prefix,
                                                           const int64_t n_items,
                                                           const uint64_t t0, const uint64_t count) {
  __shared__ uint32_t red[kCastWaves];
  const int lane = threadIdx.x & (kWaveLanes - 1);
  const uint64_t t = t0 + xcd_grouped(blockIdx.x, count, kCastXcdGroup);
  const int64_t it = find_item(prefix, n_items, t, lane);
  const tc_cast_item item = items[it];
  const int64_t full_c = item.cols / kTile;
  const int64_t local = int64_t(t - prefix[it]);
  const int64_t ti = local / full_c, tj = local - ti * full_c;
  cast_tile(src + item.src_off + ti * kTile * item.src_ld + tj * kTile,
            dst + item.dst_off + ti * kTile * item.dst_ld + tj * kTile, item.src_ld, item.dst_ld,
            scales + item.scale_off + ti * item.scale_ld + tj, red);
}

// The same with the tile's addresses read from the per-tile table: one
// load before the data loads instead of the item search, the item's record
// and a division (measured +4.5% on the 70B TP=8 shard).
__global__ __launch_bounds__(kCastThreads) void k_cast_full_tab(const uint16_t* __restrict__ src,
                                                               uint8_t* __restrict__ dst,
                                                               float* __restrict__ scales,
                                                               const TileEntry* __restrict__ tab,
                                                               const uint64_t t0, const uint64_t count) {
  __shared__ uint32_t red[kCastWaves];
  const uint64_t t = t0 + xcd_grouped(blockIdx.x, count, kCastXcdGroup);
  const TileEntry e = tab[t];
  cast_tile(src + e.in_off, dst + e.out_off, int64_t(uint32_t(e.lds)), int64_t(e.lds >> 32),
            scales + e.scale_idx, red);
}

// The per-tile table of the full tiles, one thread per tile: the tile's item
// by binary search of the full-tile prefix, then its row and column of
// tiles.  Cast and inverse-cast items share the record layout.
__global__ __launch_bounds__(kThreads) void k_tile_expand(const tc_cast_item* __restrict__ items,
                                                         const uint64_t* __restrict__ prefix,
                                                         const int64_t n_items, const uint64_t full_tiles,
                                                         TileEntry* __restrict__ tab) {
  for (uint64_t t = uint64_t(blockIdx.x) * kThreads + threadIdx.x; t < full_tiles;
       t += uint64_t(gridDim.x) * kThreads) {
    int64_t lo = 0, hi = n_items;  // the last item with prefix <= t
    while (hi - lo > 1) {
      const int64_t mid = lo + (hi - lo) / 2;
      if (prefix[mid] <= t)
        lo = mid;
      else
        hi = mid;
    }
    const tc_cast_item item = items[lo];
    const int64_t full_c = item.cols / kTile;
    const int64_t local = int64_t(t - prefix[lo]);
    const int64_t ti = local / full_c, tj = local - ti * full_c;
    TileEntry e;
    e.in_off = item.src_off + uint64_t(ti * kTile * item.src_ld + tj * kTile);
    e.out_off = item.dst_off + uint64_t(ti * kTile * item.dst_ld + tj * kTile);
    e.scale_idx = item.scale_off + uint64_t(ti * item.scale_ld + tj);
    e.lds = uint64_t(item.src_ld) | (uint64_t(item.dst_ld) << 32);
    tab[t] = e;
  }
}

// The remaining tiles: partial tiles at the bottom and right edges, and every
// tile of items that are not aligned for the vector path.  Element by
// element; prefix counts each item's remaining tiles.  Within an item they
// are numbered row of tiles by row of tiles: first the tile rows from fr
// (all tile columns), then the tile columns from fc of the first fr rows,
// where fr x fc is the item's full-tile grid (0 x 0 for unaligned items).
__global__ __launch_bounds__(kCastThreads) void k_cast_edge(const uint16_t* __restrict__ src,
                                                           uint8_t* __restrict__ dst,
                                                           float* __restrict__ scales,
                                                           const tc_cast_item* __restrict__ items,
                                                           const uint64_t* __restrict__ prefix,
                                                           const uint8_t* __restrict__ aligned,
                                                           const int64_t n_items,
                                                           const uint64_t t0) {
  __shared__ uint32_t red[kCastWaves];
  const int lane = threadIdx.x & (kWaveLanes - 1);
  const uint64_t t = t0 + blockIdx.x;
  const int64_t it = find_item(prefix, n_items, t, lane);
  const tc_cast_item item = items[it];
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
  const uint16_t* xs = src + item.src_off + r0 * item.src_ld + c0;
  uint8_t* qs = dst + item.dst_off + r0 * item.dst_ld + c0;
  const int64_t cnt = h * wd;
  uint32_t m = 0;
  for (int64_t k = threadIdx.x; k < cnt; k += kCastThreads) {
    const int64_t rr = k / wd, cc = k - rr * wd;
    m = max(m, uint32_t(xs[rr * item.src_ld + cc]) & 0x7FFFu);
  }
  const uint32_t amax_bits = block_amax(m, red);
  int mode;
  float s;
  if (amax_bits >= 0x7F80u) {
    mode = 2;
    s = __uint_as_float(0x7FC00000u);
  } else if (amax_bits == 0) {
    mode = 1;
    s = 0.0f;
  } else {
    mode = 0;
    s = __uint_as_float(amax_bits << 16) / 448.0f;
  }
  for (int64_t k = threadIdx.x; k < cnt; k += kCastThreads) {
    const int64_t rr = k / wd, cc = k - rr * wd;
    qs[rr * item.dst_ld + cc] = code1(xs[rr * item.src_ld + cc], mode, s);
  }
  if (threadIdx.x == 0) scales[item.scale_off + ti * item.scale_ld + tj] = s;
}

// Elementwise cast with one given scale: 8 elements per thread.
__global__ __launch_bounds__(kThreads) void k_cast_scaled(const uint16_t* __restrict__ src,
                                                         const int64_t n, const float s,
                                                         uint8_t* __restrict__ dst,
                                                         const int vec_ok) {
  const int64_t stride = int64_t(gridDim.x) * kThreads;
  for (int64_t g = int64_t(blockIdx.x) * kThreads + threadIdx.x; g * 8 < n; g += stride) {
    const int64_t i0 = g * 8;
    uint16_t x[8];
    if (vec_ok && i0 + 8 <= n) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(src + i0);
      x[0] = v.x & 0xFFFF; x[1] = v.x >> 16; x[2] = v.y & 0xFFFF; x[3] = v.y >> 16;
      x[4] = v.z & 0xFFFF; x[5] = v.z >> 16; x[6] = v.w & 0xFFFF; x[7] = v.w >> 16;
    } else {
#pragma unroll
      for (int k = 0; k < 8; ++k) x[k] = i0 + k < n ? src[i0 + k] : 0;
    }
    uint8_t c[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const float q = __uint_as_float(uint32_t(x[k]) << 16) / s;
      const uint32_t a = __float_as_uint(q) & 0x7FFFFFFFu;
      if (a > 0x7F800000u)
        c[k] = 0x7F;  // NaN, whatever its sign
      else if (a >= 0x43E00000u)  // |q| >= 448 (and Inf): saturate
        c[k] = (uint8_t)(((__float_as_uint(q) >> 24) & 0x80u) | 0x7Eu);
      else
        c[k] = (uint8_t)(cvt2<false>(q, q, 0) & 0xFFu);
    }
    if (vec_ok && i0 + 8 <= n) {
      const u32x2 o = {uint32_t(c[0]) | uint32_t(c[1]) << 8 | uint32_t(c[2]) << 16 | uint32_t(c[3]) << 24,
                       uint32_t(c[4]) | uint32_t(c[5]) << 8 | uint32_t(c[6]) << 16 | uint32_t(c[7]) << 24};
      *reinterpret_cast<u32x2*>(dst + i0) = o;
    } else {
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if (i0 + k < n) dst[i0 + k] = c[k];
    }
  }
}

// Writes one chunk of the tile table into the workspace: the items (64-byte
// records, cast or inverse-cast items alike), their tile prefixes and their
// vector-path flags, and after the last chunk the two totals.  The chunk
// travels in the kernel arguments, so the host table needs no staging buffer
// and may be reused once the launch call returns; a graph that captures the
// launch keeps its own copy of the chunk.
__global__ __launch_bounds__(kThreads) void k_tile_table(const TableChunk c, uint8_t* __restrict__ ws,
                                                        const uint64_t items_off,
                                                        const uint64_t full_off,
                                                        const uint64_t edge_off,
                                                        const uint64_t aligned_off) {
  static_assert(sizeof(tc_cast_item) == 8 * kItemWords, "items are 8 words");
  uint64_t* items = reinterpret_cast<uint64_t*>(ws + items_off) + c.first * kItemWords;
  for (uint32_t k = threadIdx.x; k < c.count * kItemWords; k += kThreads) items[k] = c.words[k];
  uint64_t* fp = reinterpret_cast<uint64_t*>(ws + full_off);
  uint64_t* ep = reinterpret_cast<uint64_t*>(ws + edge_off);
  for (uint32_t k = threadIdx.x; k < c.count; k += kThreads) {
    fp[c.first + k] = c.fprefix[k];
    ep[c.first + k] = c.eprefix[k];
    ws[aligned_off + c.first + k] = c.aligned[k];
  }
  if (c.last && threadIdx.x == 0) {
    fp[c.first + c.count] = c.ftotal;
    ep[c.first + c.count] = c.etotal;
  }
}

}  // namespace

static size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

hipError_t launch_tile_chunk(const TableChunk& c, int64_t n_items, void* ws, hipStream_t s) {
  const CastLayout L = cast_layout(n_items);
  hipLaunchKernelGGL(k_tile_table, dim3(1), dim3(kThreads), 0, s, c, static_cast<uint8_t*>(ws),
                     uint64_t(L.items), uint64_t(L.full_prefix), uint64_t(L.edge_prefix),
                     uint64_t(L.aligned));
  return hipGetLastError();
}

CastLayout cast_layout(int64_t n_items) {
  CastLayout L;
  L.items = 0;
  L.full_prefix = align256(sizeof(tc_cast_item) * size_t(n_items));
  L.edge_prefix = L.full_prefix + align256(8 * size_t(n_items + 1));
  L.aligned = L.edge_prefix + align256(8 * size_t(n_items + 1));
  L.bytes = L.aligned + align256(size_t(n_items));
  return L;
}

size_t cast_workspace_bytes(int64_t n_items) { return cast_layout(n_items).bytes; }

hipError_t launch_tile_expand(void* ws, int64_t n_items, uint64_t full_tiles, hipStream_t s) {
  if (full_tiles == 0) return hipSuccess;
  const CastLayout L = cast_layout(n_items);
  uint8_t* base = static_cast<uint8_t*>(ws);
  hipLaunchKernelGGL(k_tile_expand, dim3(grid_for((full_tiles + kThreads - 1) / kThreads)), dim3(kThreads),
                     0, s, reinterpret_cast<const tc_cast_item*>(base + L.items),
                     reinterpret_cast<const uint64_t*>(base + L.full_prefix), n_items, full_tiles,
                     reinterpret_cast<TileEntry*>(base + L.bytes));
  return hipGetLastError();
}

hipError_t launch_cast_blockscaled(const uint16_t* src, uint8_t* dst, float* scales,
                                   const void* ws, int64_t n_items, uint64_t full_tiles,
                                   uint64_t edge_tiles, bool tiled, hipStream_t s) {
  const CastLayout L = cast_layout(n_items);
  const uint8_t* base = static_cast<const uint8_t*>(ws);
  const tc_cast_item* items = reinterpret_cast<const tc_cast_item*>(base + L.items);
  const uint64_t* fp = reinterpret_cast<const uint64_t*>(base + L.full_prefix);
  const uint64_t* ep = reinterpret_cast<const uint64_t*>(base + L.edge_prefix);
  const uint8_t* al = base + L.aligned;
  const TileEntry* tab = reinterpret_cast<const TileEntry*>(base + L.bytes);
  for (uint64_t t0 = 0; t0 < full_tiles; t0 += kMaxGrid) {
    const uint64_t cnt = full_tiles - t0 < kMaxGrid ? full_tiles - t0 : kMaxGrid;
    if (tiled)
      hipLaunchKernelGGL(k_cast_full_tab, dim3((unsigned)cnt), dim3(kCastThreads), 0, s, src, dst, scales,
                         tab, t0, cnt);
    else
      hipLaunchKernelGGL(k_cast_full, dim3((unsigned)cnt), dim3(kCastThreads), 0, s, src, dst, scales,
                         items, fp, n_items, t0, cnt);
  }
  for (uint64_t t0 = 0; t0 < edge_tiles; t0 += kMaxGrid) {
    const uint64_t cnt = edge_tiles - t0 < kMaxGrid ? edge_tiles - t0 : kMaxGrid;
    hipLaunchKernelGGL(k_cast_edge, dim3((unsigned)cnt), dim3(kCastThreads), 0, s, src, dst, scales,
                       items, ep, al, n_items, t0);
  }
  return hipGetLastError();
}

hipError_t launch_cast_scaled(const uint16_t* src, int64_t n, float scale, uint8_t* dst,
                              hipStream_t s) {
  const int vec_ok = ((reinterpret_cast<uintptr_t>(src) & 15) == 0 &&
                      (reinterpret_cast<uintptr_t>(dst) & 7) == 0);
  const int64_t groups = (n + 7) / 8;
  int64_t blocks = (groups + kThreads - 1) / kThreads;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(k_cast_scaled, dim3((unsigned)blocks), dim3(kThreads), 0, s, src, n, scale,
                     dst, vec_ok);
  return hipGetLastError();
}

}  // namespace tc
