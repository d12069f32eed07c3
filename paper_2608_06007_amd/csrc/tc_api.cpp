// C ABI of the data path: argument checks, optional validation, launches.
// Host-only code; the kernels live in tc_blocks.hip, tc_plan.hip, tc_copy.hip,
// tc_cast.hip and tc_dequant.hip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "tc_internal.h"

namespace {

thread_local int g_last_hip_error = 0;
std::atomic<int> g_validate{-1};  // -1: not yet read from the environment

bool validating() {
  int v = g_validate.load(std::memory_order_relaxed);
  if (v < 0) {
    const char* e = std::getenv("TC_VALIDATE");
    int expected = -1;
    // tc_set_validate may have run meanwhile: only an unset flag takes the environment
    g_validate.compare_exchange_strong(expected, (e && e[0] && e[0] != '0') ? 1 : 0,
                                       std::memory_order_relaxed);
    v = g_validate.load(std::memory_order_relaxed);
  }
  return v == 1;
}

tc_status hip_fail(hipError_t e) {
  g_last_hip_error = (int)e;
  return TC_ERR_HIP;
}

tc_status check(hipError_t e) { return e == hipSuccess ? TC_OK : hip_fail(e); }

// Copy a device array to the host after the stream has produced it.
template <typename T>
tc_status fetch(const T* dev, int64_t n, std::vector<T>* out, hipStream_t s) {
  out->resize((size_t)n);
  if (n == 0) return TC_OK;
  hipError_t e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e);
  e = hipMemcpy(out->data(), dev, sizeof(T) * (size_t)n, hipMemcpyDeviceToHost);
  return check(e);
}

struct Range {
  uint64_t lo, hi;  // [lo, hi)
};

// True if any two non-empty ranges overlap.
bool any_overlap(std::vector<Range> r) {
  r.erase(std::remove_if(r.begin(), r.end(), [](const Range& x) { return x.hi == x.lo; }), r.end());
  std::sort(r.begin(), r.end(), [](const Range& a, const Range& b) { return a.lo < b.lo; });
  for (size_t i = 1; i < r.size(); ++i)
    if (r[i].lo < r[i - 1].hi) return true;
  return false;
}

// True if a range of a overlaps a range of b.
bool cross_overlap(std::vector<Range> a, std::vector<Range> b) {
  auto by_lo = [](const Range& x, const Range& y) { return x.lo < y.lo; };
  auto empty = [](const Range& x) { return x.hi == x.lo; };
  a.erase(std::remove_if(a.begin(), a.end(), empty), a.end());
  b.erase(std::remove_if(b.begin(), b.end(), empty), b.end());
  std::sort(a.begin(), a.end(), by_lo);
  std::sort(b.begin(), b.end(), by_lo);
  // sweep: keep the furthest end seen in each list
  size_t i = 0, j = 0;
  uint64_t end_a = 0, end_b = 0;
  while (i < a.size() || j < b.size()) {
    if (j == b.size() || (i < a.size() && a[i].lo <= b[j].lo)) {
      if (a[i].lo < end_b) return true;
      end_a = std::max(end_a, a[i].hi);
      ++i;
    } else {
      if (b[j].lo < end_a) return true;
      end_b = std::max(end_b, b[j].hi);
      ++j;
    }
  }
  return false;
}

tc_status blocks_common(const tc_block_pool* pool, const int32_t* ids, int64_t n, void* buf,
                        bool gather, hipStream_t s) {
  if (n < 0 || !tc::pool_valid(pool)) return TC_ERR_INVALID_ARGUMENT;
  if (n == 0) return TC_OK;
  if (!ids || !buf) return TC_ERR_INVALID_ARGUMENT;
  const int32_t R = pool->num_regions;
  const int64_t B = pool->block_bytes, stride = pool->block_stride;
  // so does the transfer buffer's, n * R * B bytes
  if (n > INT64_MAX / R / B) return TC_ERR_INVALID_ARGUMENT;
  if (validating()) {
    std::vector<int32_t> h;
    tc_status st = fetch(ids, n, &h, s);
    if (st != TC_OK) return st;
    std::vector<uint8_t> seen((size_t)pool->num_blocks, 0);
    for (int32_t id : h) {
      if (id < 0 || id >= pool->num_blocks) return TC_ERR_OUT_OF_RANGE;
      if (!gather && seen[(size_t)id]) return TC_ERR_ALIAS;
      seen[(size_t)id] = 1;
    }
    // transfer buffer against the blocks it is exchanged with
    std::vector<Range> pool_r, buf_r;
    buf_r.push_back({(uint64_t)(uintptr_t)buf, (uint64_t)(uintptr_t)buf + uint64_t(n * R * B)});
    for (int r = 0; r < R; ++r) {
      const uint64_t base = pool->region_base[r];
      const uint64_t span = uint64_t(pool->num_blocks - 1) * uint64_t(stride) + uint64_t(B);
      pool_r.push_back({base, base + span});
    }
    if (cross_overlap(pool_r, buf_r)) return TC_ERR_ALIAS;
    if (!gather) {
      // the blocks written must not overlap one another (regions may share memory)
      std::vector<Range> w;
      w.reserve(h.size() * (size_t)R);
      for (int32_t id : h)
        for (int r = 0; r < R; ++r) {
          const uint64_t a = pool->region_base[r] + uint64_t(id) * uint64_t(stride);
          w.push_back({a, a + uint64_t(B)});
        }
      if (any_overlap(w)) return TC_ERR_ALIAS;
    }
  }
  tc::RegionTable tab;
  bool aligned = (B % 16) == 0 && (stride % 16) == 0 && ((uintptr_t)buf % 16) == 0;
  for (int r = 0; r < R; ++r) {
    tab.base[r] = pool->region_base[r];
    aligned = aligned && (tab.base[r] % 16) == 0;
  }
  for (int r = R; r < TC_MAX_REGIONS; ++r) tab.base[r] = 0;
  return check(tc::launch_blocks(tab, R, B, stride, ids, n, static_cast<uint8_t*>(buf), gather,
                                 aligned, s));
}

bool view_ok(const tc_tp_view& v, int32_t tp, int32_t rank) {
  if (tp < 1 || rank < 0 || rank >= tp) return false;
  if (v.rows < 0 || v.cols < 0 || v.src_ld < v.cols || v.dst_ld < 0) return false;
  if (!(v.elem_bytes == 1 || v.elem_bytes == 2 || v.elem_bytes == 4 || v.elem_bytes == 8))
    return false;
  if (v.split == TC_SPLIT_ROWS) {
    if (v.rows % tp) return false;
    if (v.dst_ld < v.cols) return false;
  } else if (v.split == TC_SPLIT_COLS) {
    if (v.cols % tp) return false;
    if (v.dst_ld < v.cols / tp) return false;
  } else if (v.split == TC_SPLIT_NONE) {
    if (v.dst_ld < v.cols) return false;
  } else {
    return false;
  }
  return true;
}

// The rank's sub-matrix of a view: first source element, shape.
struct Slice {
  uint64_t src_elem;  // element offset from the matrix origin
  int64_t rows, cols;
};

Slice slice_of(const tc_tp_view& v, int32_t tp, int32_t rank) {
  if (v.split == TC_SPLIT_ROWS) {
    const int64_t k = v.rows / tp;
    return {uint64_t(rank) * uint64_t(k) * uint64_t(v.src_ld), k, v.cols};
  }
  if (v.split == TC_SPLIT_COLS) {
    const int64_t k = v.cols / tp;
    return {uint64_t(rank) * uint64_t(k), v.rows, k};
  }
  return {0, v.rows, v.cols};
}

// Fragments of one view: one per row, or one for the whole slice when the
// rows are contiguous in both source and destination.
template <typename Emit>
void view_fragments(const tc_tp_view& v, int32_t tp, int32_t rank, Emit emit) {
  const Slice sl = slice_of(v, tp, rank);
  if (sl.rows == 0 || sl.cols == 0) return;
  const uint64_t eb = uint64_t(v.elem_bytes);
  const uint64_t row_bytes = uint64_t(sl.cols) * eb;
  const uint64_t src0 = v.src_off + sl.src_elem * eb;
  const bool contiguous = (sl.rows == 1) || (v.src_ld == sl.cols && v.dst_ld == sl.cols);
  if (contiguous) {
    emit(tc_fragment{src0, v.dst_off, row_bytes * uint64_t(sl.rows)});
    return;
  }
  for (int64_t r = 0; r < sl.rows; ++r)
    emit(tc_fragment{src0 + uint64_t(r) * uint64_t(v.src_ld) * eb,
                     v.dst_off + uint64_t(r) * uint64_t(v.dst_ld) * eb, row_bytes});
}


bool elem_ok(int32_t eb) { return eb == 1 || eb == 2 || eb == 4 || eb == 8; }

bool reshard_ok(const tc_reshard_view& v, int32_t dst_tp, int32_t dst_rank) {
  if (!v.src_off || v.src_tp < 1 || dst_tp < 1 || dst_rank < 0 || dst_rank >= dst_tp) return false;
  if (v.rows < 0 || v.cols < 0 || !elem_ok(v.elem_bytes)) return false;
  if (v.split == TC_SPLIT_ROWS) return v.rows % v.src_tp == 0 && v.rows % dst_tp == 0;
  if (v.split == TC_SPLIT_COLS) return v.cols % v.src_tp == 0 && v.cols % dst_tp == 0;
  return v.split == TC_SPLIT_NONE;
}

// Fragments that fill the destination rank's slice from the overlapping
// source slices, in ascending destination order (so a plan keeps the list's
// order and the copy writes the slice front to back).
template <typename Emit>
void reshard_fragments(const tc_reshard_view& v, int32_t dst_tp, int32_t d, Emit emit) {
  if (v.rows == 0 || v.cols == 0) return;
  const uint64_t eb = uint64_t(v.elem_bytes);
  if (v.split == TC_SPLIT_NONE) {
    emit(tc_fragment{v.src_off[0], v.dst_off, uint64_t(v.rows) * uint64_t(v.cols) * eb});
    return;
  }
  const bool by_rows = v.split == TC_SPLIT_ROWS;
  const int64_t extent = by_rows ? v.rows : v.cols;
  const int64_t ns = extent / v.src_tp, nd = extent / dst_tp;  // slice widths
  const int64_t d0 = int64_t(d) * nd, d1 = d0 + nd;
  const int64_t s0 = d0 / ns, s1 = (d1 - 1) / ns;  // overlapping source slices
  if (by_rows) {
    const uint64_t row = uint64_t(v.cols) * eb;
    for (int64_t s = s0; s <= s1; ++s) {
      const int64_t a = std::max(d0, s * ns), b = std::min(d1, (s + 1) * ns);
      emit(tc_fragment{v.src_off[s] + uint64_t(a - s * ns) * row, v.dst_off + uint64_t(a - d0) * row,
                       uint64_t(b - a) * row});
    }
  } else if (ns == nd) {
    // identical column blocks: the whole slice is one contiguous run
    emit(tc_fragment{v.src_off[s0], v.dst_off, uint64_t(v.rows) * uint64_t(ns) * eb});
  } else {
    // row by row; within a row, the source slices left to right
    for (int64_t r = 0; r < v.rows; ++r)
      for (int64_t s = s0; s <= s1; ++s) {
        const int64_t a = std::max(d0, s * ns), b = std::min(d1, (s + 1) * ns);
        emit(tc_fragment{v.src_off[s] + (uint64_t(r) * uint64_t(ns) + uint64_t(a - s * ns)) * eb,
                         v.dst_off + (uint64_t(r) * uint64_t(nd) + uint64_t(a - d0)) * eb,
                         uint64_t(b - a) * eb});
      }
  }
}

// Cast items that fill the destination rank's fp8 slice from the
// overlapping bf16 source slices, one item per source slice; each writes its
// part of the slice's scale grid.  A boundary between two source slices must
// fall on a 128-element tile edge of the destination slice (a tile cannot
// take its amax from two sources); returns false otherwise, and for views
// that are not bf16.
template <typename Emit>
bool reshard_cast_items(const tc_reshard_view& v, uint64_t scale_off, int32_t dst_tp, int32_t d,
                        Emit emit) {
  if (v.elem_bytes != 2) return false;
  const int32_t nsrc = v.split == TC_SPLIT_NONE ? 1 : v.src_tp;
  for (int32_t s = 0; s < nsrc; ++s)
    if (v.src_off[s] % 2) return false;
  if (v.rows == 0 || v.cols == 0) return true;
  if (v.split == TC_SPLIT_NONE) {
    emit(tc_cast_item{v.src_off[0] / 2, v.rows, v.cols, v.cols, v.dst_off, v.cols, scale_off,
                      (v.cols + 127) / 128});
    return true;
  }
  const bool by_rows = v.split == TC_SPLIT_ROWS;
  const int64_t extent = by_rows ? v.rows : v.cols;
  const int64_t ns = extent / v.src_tp, nd = extent / dst_tp;
  const int64_t d0 = int64_t(d) * nd, d1 = d0 + nd;
  const int64_t dcols = by_rows ? v.cols : nd;  // destination slice width
  const int64_t sld = (dcols + 127) / 128;
  for (int64_t s = d0 / ns; s <= (d1 - 1) / ns; ++s) {
    const int64_t a = std::max(d0, s * ns), b = std::min(d1, (s + 1) * ns);
    if ((a - d0) % 128) return false;
    if (by_rows)
      emit(tc_cast_item{v.src_off[s] / 2 + uint64_t(a - s * ns) * uint64_t(v.cols), b - a, v.cols,
                        v.cols, v.dst_off + uint64_t(a - d0) * uint64_t(v.cols), v.cols,
                        scale_off + uint64_t((a - d0) / 128) * uint64_t(sld), sld});
    else
      emit(tc_cast_item{v.src_off[s] / 2 + uint64_t(a - s * ns), v.rows, b - a, ns,
                        v.dst_off + uint64_t(a - d0), nd, scale_off + uint64_t((a - d0) / 128), sld});
  }
  return true;
}

// Item counts above this are refused (the cast grids grow with them).
constexpr int64_t kMaxItems = int64_t(1) << 33;

static_assert(sizeof(tc_dequant_item) == sizeof(tc_cast_item), "shared workspace layout");
static_assert(sizeof(tc_cast_item) == 8 * tc::kItemWords, "items are copied as 8 words");
static_assert(sizeof(tc_dequant_item) == 8 * tc::kItemWords, "items are copied as 8 words");

// Tile ranges of an item list, on the host: full tiles of vector-aligned
// items go to the streaming kernel, every other tile to the element-wise one.
// Cast items read 16-byte-aligned bf16 rows and write 8-byte-aligned code
// rows; inverse items read 8-byte-aligned code rows and write 16-byte-aligned
// bf16 rows.  False for an invalid item.
template <typename Item>
bool item_tiles(const Item& it, uint64_t in_base, uint64_t out_base, bool cast, uint8_t* aligned,
                uint64_t* full, uint64_t* all) {
  if (it.rows < 0 || it.cols < 0 || it.src_ld < it.cols || it.dst_ld < it.cols) return false;
  const uint64_t tr = uint64_t((it.rows + 127) / 128), tcn = uint64_t((it.cols + 127) / 128);
  if (it.rows > 0 && it.cols > 0 && it.scale_ld < int64_t(tcn)) return false;
  bool al;
  if (cast) {  // bf16 in (elements), codes out (bytes)
    const uint64_t x = in_base + 2 * it.src_off, q = out_base + it.dst_off;
    al = x % 16 == 0 && (2 * uint64_t(it.src_ld)) % 16 == 0 && q % 8 == 0 && uint64_t(it.dst_ld) % 8 == 0;
  } else {     // codes in (bytes), bf16 out (elements)
    const uint64_t q = in_base + it.src_off, y = out_base + 2 * it.dst_off;
    al = q % 8 == 0 && uint64_t(it.src_ld) % 8 == 0 && y % 16 == 0 && (2 * uint64_t(it.dst_ld)) % 16 == 0;
  }
  *aligned = al ? 1 : 0;
  *all = (it.rows > 0 && it.cols > 0) ? tr * tcn : 0;
  *full = al ? uint64_t(it.rows / 128) * uint64_t(it.cols / 128) : 0;
  return true;
}

// Validate every item and total its tiles (no table is kept).
template <typename Item>
tc_status tile_totals(const Item* items, int64_t n_items, uint64_t in_base, uint64_t out_base,
                      bool cast, uint64_t* full, uint64_t* edge) {
  *full = *edge = 0;
  for (int64_t i = 0; i < n_items; ++i) {
    uint8_t al;
    uint64_t f, all;
    if (!item_tiles(items[i], in_base, out_base, cast, &al, &f, &all)) return TC_ERR_INVALID_ARGUMENT;
    *full += f;
    *edge += all - f;
  }
  return TC_OK;
}

// Enqueue the table's writes chunk by chunk, each chunk built on the stack
// and carried in its launch's arguments: no host or device memory is taken.
template <typename Item>
hipError_t upload_tile_table(const Item* items, int64_t n_items, uint64_t in_base, uint64_t out_base,
                             bool cast, uint64_t full, uint64_t edge, void* ws, hipStream_t s) {
  tc::TableChunk c;
  uint64_t fsum = 0, esum = 0;
  for (int64_t i0 = 0; i0 < n_items; i0 += tc::kTableChunkItems) {
    const int64_t cnt = std::min<int64_t>(n_items - i0, tc::kTableChunkItems);
    c.first = uint64_t(i0);
    c.count = uint32_t(cnt);
    c.last = i0 + cnt == n_items ? 1u : 0u;
    c.ftotal = full;
    c.etotal = edge;
    for (int64_t k = 0; k < cnt; ++k) {
      const Item& it = items[i0 + k];
      std::memcpy(&c.words[k * tc::kItemWords], &it, sizeof(Item));
      uint64_t f, all;
      item_tiles(it, in_base, out_base, cast, &c.aligned[k], &f, &all);
      c.fprefix[k] = fsum;
      c.eprefix[k] = esum;
      fsum += f;
      esum += all - f;
    }
    hipError_t e = tc::launch_tile_chunk(c, n_items, ws, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// Debug checks of a cast's item list: codes and scale grids of different
// items must not overlap one another or the bf16 source.
static tc_status check_cast_ranges(const void* src_base, const void* dst_base, const void* scale_base,
                                   const tc_cast_item* items, int64_t n_items) {
  std::vector<Range> q, sc, srcr;
  const uint64_t db = (uint64_t)(uintptr_t)dst_base, sb = (uint64_t)(uintptr_t)scale_base;
  const uint64_t xb = (uint64_t)(uintptr_t)src_base;
  for (int64_t i = 0; i < n_items; ++i) {
    const tc_cast_item& it = items[i];
    if (it.rows == 0 || it.cols == 0) continue;
    const int64_t tcn = (it.cols + 127) / 128, tr = (it.rows + 127) / 128;
    for (int64_t r = 0; r < it.rows; ++r) {
      const uint64_t a = db + it.dst_off + uint64_t(r) * uint64_t(it.dst_ld);
      q.push_back({a, a + uint64_t(it.cols)});
      const uint64_t x = xb + 2 * (it.src_off + uint64_t(r) * uint64_t(it.src_ld));
      srcr.push_back({x, x + 2 * uint64_t(it.cols)});
    }
    for (int64_t r = 0; r < tr; ++r) {
      const uint64_t a = sb + 4 * (it.scale_off + uint64_t(r) * uint64_t(it.scale_ld));
      sc.push_back({a, a + 4 * uint64_t(tcn)});
    }
  }
  std::vector<Range> outs = q;
  outs.insert(outs.end(), sc.begin(), sc.end());
  if (any_overlap(outs)) return TC_ERR_ALIAS;
  if (cross_overlap(outs, srcr)) return TC_ERR_ALIAS;
  return TC_OK;
}

// The same for the inverse: bf16 outputs disjoint, and apart from the codes
// and scales they read.
static tc_status check_dequant_ranges(const void* codes_base, const void* scale_base,
                                      const void* dst_base, const tc_dequant_item* items,
                                      int64_t n_items) {
  std::vector<Range> outs, srcs;
  const uint64_t db = (uint64_t)(uintptr_t)dst_base, qb = (uint64_t)(uintptr_t)codes_base;
  const uint64_t sb = (uint64_t)(uintptr_t)scale_base;
  for (int64_t i = 0; i < n_items; ++i) {
    const tc_dequant_item& it = items[i];
    if (it.rows == 0 || it.cols == 0) continue;
    const int64_t tcn = (it.cols + 127) / 128, tr = (it.rows + 127) / 128;
    for (int64_t r = 0; r < it.rows; ++r) {
      const uint64_t a = db + 2 * (it.dst_off + uint64_t(r) * uint64_t(it.dst_ld));
      outs.push_back({a, a + 2 * uint64_t(it.cols)});
      const uint64_t x = qb + it.src_off + uint64_t(r) * uint64_t(it.src_ld);
      srcs.push_back({x, x + uint64_t(it.cols)});
    }
    for (int64_t r = 0; r < tr; ++r) {
      const uint64_t a = sb + 4 * (it.scale_off + uint64_t(r) * uint64_t(it.scale_ld));
      srcs.push_back({a, a + 4 * uint64_t(tcn)});
    }
  }
  if (any_overlap(outs)) return TC_ERR_ALIAS;
  if (cross_overlap(outs, srcs)) return TC_ERR_ALIAS;
  return TC_OK;
}

// prepare: checks, the host tile table, and its enqueued upload into the
// workspace (by value, in the launches' arguments).  cast selects the item
// kind; in_base/out_base are the bases whose alignment the table assumes.
template <typename Item>
static tc_status prepare_tiles(const void* in_base, const void* out_base, const Item* items,
                               int64_t n_items, int32_t tile, void* workspace, size_t workspace_bytes,
                               bool cast, tc_tile_plan* plan, hipStream_t stream) {
  if (!plan) return TC_ERR_INVALID_ARGUMENT;
  *plan = tc_tile_plan{0, 0, 0, 0, 0, 0, 0};
  if (n_items < 0 || n_items > kMaxItems || tile != 128) return TC_ERR_INVALID_ARGUMENT;
  if (n_items == 0) return TC_OK;
  if (!in_base || !out_base || !items || !workspace) return TC_ERR_INVALID_ARGUMENT;
  if (workspace_bytes < tc::cast_workspace_bytes(n_items)) return TC_ERR_WORKSPACE;
  if ((uintptr_t)workspace % 256) return TC_ERR_INVALID_ARGUMENT;
  // bf16 bases hold 2-byte elements
  if ((cast ? (uintptr_t)in_base : (uintptr_t)out_base) % 2) return TC_ERR_INVALID_ARGUMENT;
  const uint64_t ib = (uint64_t)(uintptr_t)in_base, ob = (uint64_t)(uintptr_t)out_base;
  uint64_t full, edge;
  tc_status st = tile_totals(items, n_items, ib, ob, cast, &full, &edge);
  if (st != TC_OK) return st;
  st = check(upload_tile_table(items, n_items, ib, ob, cast, full, edge, workspace, stream));
  if (st != TC_OK) return st;
  // The per-tile table, when the workspace has room for it and every row
  // pitch fits its 32-bit fields.
  bool tiled = full > 0 && full < (uint64_t(1) << 50) &&
               workspace_bytes - tc::cast_workspace_bytes(n_items) >= full * tc::kTileEntryBytes;
  for (int64_t i = 0; tiled && i < n_items; ++i)
    tiled = uint64_t(items[i].src_ld) >> 32 == 0 && uint64_t(items[i].dst_ld) >> 32 == 0;
  if (tiled) {
    st = check(tc::launch_tile_expand(workspace, n_items, full, stream));
    if (st != TC_OK) return st;
  }
  *plan = tc_tile_plan{n_items, full, edge, uint32_t(ib % 16), uint32_t(ob % 16), tiled ? 1u : 0u, 0};
  return TC_OK;
}

// Workspace for n_items items and the per-tile table of all their full
// tiles (counted as if every item were aligned; 0 for an invalid item).
template <typename Item>
static size_t workspace_with_tiles(const Item* items, int64_t n_items) {
  if (n_items < 0 || n_items > kMaxItems || (n_items > 0 && !items)) return 0;
  uint64_t tiles = 0;
  for (int64_t i = 0; i < n_items; ++i) {
    const Item& it = items[i];
    if (it.rows < 0 || it.cols < 0) return 0;
    tiles += uint64_t(it.rows / 128) * uint64_t(it.cols / 128);
    if (tiles > (uint64_t(1) << 40)) return 0;
  }
  return tc::cast_workspace_bytes(n_items) + ((tiles * tc::kTileEntryBytes + 255) & ~uint64_t(255));
}

// Checks of a planned launch: the table's size, and bases with the
// alignment the table was made for.
static tc_status planned_args(const void* in_base, const void* out_base, const float* scale_base,
                              const void* workspace, size_t workspace_bytes,
                              const tc_tile_plan* plan) {
  if (!plan || plan->n_items < 0 || plan->n_items > kMaxItems) return TC_ERR_INVALID_ARGUMENT;
  if (plan->full_tiles + plan->edge_tiles == 0) return TC_OK;
  if (!in_base || !out_base || !scale_base || !workspace || (uintptr_t)workspace % 256 ||
      (uintptr_t)scale_base % 4)
    return TC_ERR_INVALID_ARGUMENT;
  if (workspace_bytes < tc::cast_workspace_bytes(plan->n_items)) return TC_ERR_WORKSPACE;
  if (plan->tiled > 1) return TC_ERR_INVALID_ARGUMENT;
  if (plan->tiled && (workspace_bytes - tc::cast_workspace_bytes(plan->n_items)) / tc::kTileEntryBytes <
                         plan->full_tiles)
    return TC_ERR_WORKSPACE;
  if ((uintptr_t)in_base % 16 != plan->in_align || (uintptr_t)out_base % 16 != plan->out_align)
    return TC_ERR_INVALID_ARGUMENT;
  return TC_OK;
}

}  // namespace

namespace tc {
tc_status hip_status(hipError_t e) { return check(e); }

bool pool_valid(const tc_block_pool* p) {
  if (!p || !p->region_base) return false;
  if (p->num_regions < 1 || p->num_regions > TC_MAX_REGIONS) return false;
  if (p->num_blocks < 1 || p->block_bytes < 1 || p->block_stride < p->block_bytes) return false;
  if (p->num_blocks > INT64_MAX / p->block_stride) return false;
  if (p->block_bytes > INT64_MAX / p->num_regions) return false;
  for (int r = 0; r < p->num_regions; ++r)
    if (p->region_base[r] == 0) return false;
  return true;
}
}  // namespace tc

extern "C" {

tc_status tc_gather_blocks(const tc_block_pool* pool, const int32_t* ids, int64_t n, void* out,
                           hipStream_t stream) {
  try {
    return blocks_common(pool, ids, n, out, true, stream);
  } catch (...) {
    return TC_ERR_HOST_RESOURCES;  // host memory or threads
  }
}

tc_status tc_scatter_blocks(const tc_block_pool* pool, const int32_t* ids, int64_t n,
                            const void* in, hipStream_t stream) {
  try {
    return blocks_common(pool, ids, n, const_cast<void*>(in), false, stream);
  } catch (...) {
    return TC_ERR_HOST_RESOURCES;  // host memory or threads
  }
}

// Fragment, item and task counts above this are refused.  The plan and
// reduce kernels launch one 256-thread workgroup per 1024 fragments or tasks
// without striding, and a dispatch counts its work-items in 32 bits; 2^33
// descriptors (206 GB) already exceed what one GPU holds.
constexpr int64_t kMaxCount = int64_t(1) << 33;

size_t tc_copy_fragments_workspace(int64_t n) {
  if (n < 0 || n > kMaxCount) return 0;
  return tc::frag_workspace_bytes(n);
}

size_t tc_copy_fragments_workspace_min(int64_t n) {
  if (n < 0 || n > kMaxCount) return 0;
  return tc::frag_workspace_min_bytes(n);
}

// Debug checks of a descriptor list: no overflow, destination ranges pairwise
// disjoint and, when both bases are known, no destination range overlapping
// a source range.
static tc_status check_ranges(const void* src_base, const void* dst_base,
                              const std::vector<tc_fragment>& h) {
  std::vector<Range> d, sr;
  d.reserve(h.size());
  sr.reserve(h.size());
  const uint64_t sb = (uint64_t)(uintptr_t)src_base, db = (uint64_t)(uintptr_t)dst_base;
  for (const tc_fragment& f : h) {
    if (f.src_off + f.len < f.src_off || f.dst_off + f.len < f.dst_off) return TC_ERR_OUT_OF_RANGE;
    if (f.src_off + f.len > tc::kOffsetLimit || f.dst_off + f.len > tc::kOffsetLimit)
      return TC_ERR_OUT_OF_RANGE;
    if (sb + f.src_off + f.len < sb || db + f.dst_off + f.len < db) return TC_ERR_OUT_OF_RANGE;
    d.push_back({db + f.dst_off, db + f.dst_off + f.len});
    sr.push_back({sb + f.src_off, sb + f.src_off + f.len});
  }
  if (any_overlap(d)) return TC_ERR_ALIAS;
  if (src_base && dst_base && cross_overlap(d, sr)) return TC_ERR_ALIAS;
  return TC_OK;
}

// Checks shared by the planning entry points; *L receives the plan's layout.
static tc_status plan_args(const tc_fragment* frags, int64_t n, void* workspace,
                           size_t workspace_bytes, tc::PlanLayout* L, hipStream_t stream) {
  if (n < 0 || n > kMaxCount) return TC_ERR_INVALID_ARGUMENT;
  if (n == 0) return TC_OK;
  if (!frags || !workspace || (uintptr_t)workspace % 256) return TC_ERR_INVALID_ARGUMENT;
  *L = tc::plan_layout(n, workspace_bytes);
  if (L->capacity < uint64_t(n) + 1) return TC_ERR_WORKSPACE;
  if (validating()) {
    std::vector<tc_fragment> h;
    tc_status st = fetch(frags, n, &h, stream);
    if (st != TC_OK) return st;
    st = check_ranges(nullptr, nullptr, h);
    if (st != TC_OK) return st;
  }
  return TC_OK;
}

// The plan's header, read back after the stream has produced it.
static tc_status read_header(const void* workspace, tc::PlanHeader* hdr, hipStream_t stream) {
  hipError_t e = hipMemcpyAsync(hdr, workspace, sizeof(*hdr), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  return check(e);
}

tc_status tc_plan_fragments_async(const tc_fragment* frags, int64_t n, void* workspace,
                                  size_t workspace_bytes, hipStream_t stream) {
  try {
    tc::PlanLayout L;
    tc_status st = plan_args(frags, n, workspace, workspace_bytes, &L, stream);
    if (st != TC_OK || n == 0) return st;
    return check(tc::launch_plan(frags, n, workspace, L, stream));
  } catch (...) {
    return TC_ERR_HOST_RESOURCES;  // host memory or threads
  }
}

tc_status tc_plan_status(const void* workspace, size_t workspace_bytes, uint64_t* total_tasks,
                         hipStream_t stream) {
  try {
    if (total_tasks) *total_tasks = 0;
    if (!workspace || (uintptr_t)workspace % 256 || workspace_bytes < tc::kTasksOffset)
      return TC_ERR_INVALID_ARGUMENT;
    tc::PlanHeader hdr;
    tc_status st = read_header(workspace, &hdr, stream);
    if (st != TC_OK) return st;
    if (hdr.status != TC_OK) return (tc_status)hdr.status;
    if (total_tasks) *total_tasks = hdr.total_tasks;
    return TC_OK;
  } catch (...) {
    return TC_ERR_HOST_RESOURCES;  // host memory or threads
  }
}

tc_status tc_plan_fragments(const tc_fragment* frags, int64_t n, void* workspace,
                            size_t workspace_bytes, uint64_t* total_tasks, hipStream_t stream) {
  try {
    if (total_tasks) *total_tasks = 0;
    tc::PlanLayout L;
    tc_status st = plan_args(frags, n, workspace, workspace_bytes, &L, stream);
    if (st != TC_OK || n == 0) return st;
    st = check(tc::launch_plan(frags, n, workspace, L, stream));
    if (st != TC_OK) return st;
    // the caller asked for the task count: read it back
    return tc_plan_status(workspace, workspace_bytes, total_tasks, stream);
  } catch (...) {
    return TC_ERR_HOST_RESOURCES;  // host memory or threads
  }
}

tc_status tc_copy_planned(const void* src_base, void* dst_base, const void* workspace,
                          size_t workspace_bytes, uint64_t total_tasks, hipStream_t stream) {
  try {
    if (total_tasks == 0) return TC_OK;
    const bool from_plan = total_tasks == TC_TASKS_FROM_PLAN;
    if (!src_base || !dst_base || !workspace || (uintptr_t)workspace % 256 ||
        (!from_plan && total_tasks > uint64_t(kMaxCount)))
      return TC_ERR_INVALID_ARGUMENT;
    // Whatever the plan's fragment count, its task table lies inside the
    // workspace: a larger count cannot come from a plan made in it.
    if (workspace_bytes < tc::kTasksOffset) return TC_ERR_WORKSPACE;
    const uint64_t cap_tasks = (workspace_bytes - tc::kTasksOffset) / tc::kTaskBytes;
    if (!from_plan && total_tasks > cap_tasks) return TC_ERR_WORKSPACE;
    // The plan's own fragment count sizes its layout.
    tc::PlanHeader hdr;
    if (validating()) {
      tc_status hst = read_header(workspace, &hdr, stream);
      if (hst != TC_OK) return hst;
      if (from_plan) {
        if (hdr.status != TC_OK) return (tc_status)hdr.status;
        total_tasks = hdr.total_tasks;
        if (total_tasks == 0) return TC_OK;
      }
      if (hdr.total_tasks != total_tasks) return TC_ERR_INVALID_ARGUMENT;
      const tc::PlanLayout L = tc::plan_layout((int64_t)hdr.n, workspace_bytes);
      if (total_tasks > L.capacity) return TC_ERR_WORKSPACE;
      std::vector<tc::Task> packed;
      tc_status st = fetch(reinterpret_cast<const tc::Task*>(static_cast<const uint8_t*>(workspace) +
                                                             tc::kTasksOffset),
                           (int64_t)total_tasks, &packed, stream);
      if (st != TC_OK) return st;
      std::vector<tc_fragment> tasks(packed.size());
      for (size_t i = 0; i < packed.size(); ++i) {
        const tc::Task& t = packed[i];
        tasks[i] = tc_fragment{tc::task_src(t), tc::task_dst(t), tc::task_len(t)};
      }
      st = check_ranges(src_base, dst_base, tasks);
      if (st != TC_OK) return st;
    }
    return check(tc::launch_copy_tasks(static_cast<const uint8_t*>(src_base),
                                       static_cast<uint8_t*>(dst_base), workspace, total_tasks,
                                       cap_tasks, stream));
  } catch (...) {
    return TC_ERR_HOST_RESOURCES;  // host memory or threads
  }
}

// Shared by the digest entry points: argument checks, the plan's layout for
// n fragments, and (when validating) the header's agreement with n and the
// task count.
static tc_status digest_common(const void* read_base, void* workspace, size_t workspace_bytes,
                               uint64_t total_tasks, int64_t n, const uint64_t* digests,
                               hipStream_t stream, tc::PlanLayout* L) {
  if (n < 0 || n > kMaxCount) return TC_ERR_INVALID_ARGUMENT;
  if (n == 0) return total_tasks == 0 ? TC_OK : TC_ERR_INVALID_ARGUMENT;
  if (!digests || !workspace || (uintptr_t)workspace % 256 || (uintptr_t)digests % 8)
    return TC_ERR_INVALID_ARGUMENT;
  if ((total_tasks && !read_base) || total_tasks > uint64_t(kMaxCount)) return TC_ERR_INVALID_ARGUMENT;
  *L = tc::plan_layout(n, workspace_bytes);
  if (total_tasks > L->capacity) return TC_ERR_WORKSPACE;
  if (validating()) {
    tc::PlanHeader hdr;
    hipError_t e = hipMemcpyAsync(&hdr, workspace, sizeof(hdr), hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return hip_fail(e);
    if (hdr.total_tasks != total_tasks || hdr.n != uint64_t(n)) return TC_ERR_INVALID_ARGUMENT;
  }
  return TC_OK;
}

tc_status tc_copy_planned_digest(const void* src_base, void* dst_base, void* workspace,
                                 size_t workspace_bytes, uint64_t total_tasks, int64_t n,
                                 uint64_t* digests, hipStream_t stream) {
  try {
    if (total_tasks && !dst_base) return TC_ERR_INVALID_ARGUMENT;
    tc::PlanLayout L;
    tc_status st =
        digest_common(src_base, workspace, workspace_bytes, total_tasks, n, digests, stream, &L);
    if (st != TC_OK || n == 0) return st;
    if (validating() && total_tasks) {
      // the planned ranges must not alias, as for tc_copy_planned
      std::vector<tc::Task> packed;
      st = fetch(reinterpret_cast<const tc::Task*>(static_cast<const uint8_t*>(workspace) +
                                                   tc::kTasksOffset),
                 (int64_t)total_tasks, &packed, stream);
      if (st != TC_OK) return st;
      std::vector<tc_fragment> tasks(packed.size());
      for (size_t i = 0; i < packed.size(); ++i) {
        const tc::Task& t = packed[i];
        tasks[i] = tc_fragment{tc::task_src(t), tc::task_dst(t), tc::task_len(t)};
      }
      st = check_ranges(src_base, dst_base, tasks);
      if (st != TC_OK) return st;
    }
    return check(tc::launch_copy_digest(static_cast<const uint8_t*>(src_base),
                                        static_cast<uint8_t*>(dst_base), workspace, L, n,
                                        total_tasks, 0, digests, stream));
  } catch (...) {
    return TC_ERR_HOST_RESOURCES;  // host memory or threads
  }
}

tc_status tc_digest_planned(const void* base, int32_t side, void* workspace,
                            size_t workspace_bytes, uint64_t total_tasks, int64_t n,
                            uint64_t* digests, hipStream_t stream) {
  try {
    if (side != TC_DIGEST_SRC && side != TC_DIGEST_DST) return TC_ERR_INVALID_ARGUMENT;
    tc::PlanLayout L;
    tc_status st = digest_common(base, workspace, workspace_bytes, total_tasks, n, digests, stream, &L);
    if (st != TC_OK || n == 0) return st;
    return check(tc::launch_copy_digest(static_cast<const uint8_t*>(base), nullptr, workspace, L, n,
                                        total_tasks, side == TC_DIGEST_SRC ? 1 : 2, digests,
                                        stream));
  } catch (...) {
    return TC_ERR_HOST_RESOURCES;  // host memory or threads
  }
}

tc_status tc_copy_fragments(const void* src_base, void* dst_base, const tc_fragment* frags,
                            int64_t n, void* workspace, size_t workspace_bytes,
                            hipStream_t stream) {
  try {
    if (n < 0 || n > kMaxCount) return TC_ERR_INVALID_ARGUMENT;
    if (n == 0) return TC_OK;
    if (!src_base || !dst_base || !frags || !workspace) return TC_ERR_INVALID_ARGUMENT;
    if (validating()) {
      std::vector<tc_fragment> h;
      tc_status st = fetch(frags, n, &h, stream);
      if (st != TC_OK) return st;
      st = check_ranges(src_base, dst_base, h);
      if (st != TC_OK) return st;
    }
    tc::PlanLayout L;
    tc_status st = plan_args(frags, n, workspace, workspace_bytes, &L, stream);
    if (st != TC_OK) return st;
    st = check(tc::launch_plan(frags, n, workspace, L, stream));
    if (st != TC_OK) return st;
    // the copy takes its task count from the plan, on the device
    return check(tc::launch_copy_tasks(static_cast<const uint8_t*>(src_base),
                                       static_cast<uint8_t*>(dst_base), workspace,
                                       tc::kTasksFromPlan, L.capacity, stream));
  } catch (...) {
    return TC_ERR_HOST_RESOURCES;  // host memory or threads
  }
}

int64_t tc_tp_fragment_count(const tc_tp_view* views, int64_t n_views, int32_t tp, int32_t rank) {
  if (n_views < 0 || (n_views > 0 && !views)) return -1;
  int64_t count = 0;
  for (int64_t i = 0; i < n_views; ++i) {
    if (!view_ok(views[i], tp, rank)) return -1;
    view_fragments(views[i], tp, rank, [&](const tc_fragment&) { ++count; });
  }
  return count;
}

tc_status tc_tp_fragments(const tc_tp_view* views, int64_t n_views, int32_t tp, int32_t rank,
                          tc_fragment* out, int64_t capacity, int64_t* written) {
  try {
    if (!written || n_views < 0 || (n_views > 0 && !views) || capacity < 0) return TC_ERR_INVALID_ARGUMENT;
    const int64_t need = tc_tp_fragment_count(views, n_views, tp, rank);
    if (need < 0) return TC_ERR_INVALID_ARGUMENT;
    if (need > capacity || (need > 0 && !out)) return TC_ERR_WORKSPACE;
    int64_t k = 0;
    for (int64_t i = 0; i < n_views; ++i)
      view_fragments(views[i], tp, rank, [&](const tc_fragment& f) { out[k++] = f; });
    *written = k;
    return TC_OK;
  } catch (...) {
    return TC_ERR_HOST_RESOURCES;  // host memory or threads
  }
}

int64_t tc_reshard_fragment_count(const tc_reshard_view* views, int64_t n_views, int32_t dst_tp,
                                  int32_t dst_rank) {
  if (n_views < 0 || (n_views > 0 && !views)) return -1;
  int64_t count = 0;
  for (int64_t i = 0; i < n_views; ++i) {
    if (!reshard_ok(views[i], dst_tp, dst_rank)) return -1;
    reshard_fragments(views[i], dst_tp, dst_rank, [&](const tc_fragment&) { ++count; });
  }
  return count;
}

tc_status tc_reshard_fragments(const tc_reshard_view* views, int64_t n_views, int32_t dst_tp,
                               int32_t dst_rank, tc_fragment* out, int64_t capacity,
                               int64_t* written) {
  try {
    if (!written || n_views < 0 || (n_views > 0 && !views) || capacity < 0)
      return TC_ERR_INVALID_ARGUMENT;
    const int64_t need = tc_reshard_fragment_count(views, n_views, dst_tp, dst_rank);
    if (need < 0) return TC_ERR_INVALID_ARGUMENT;
    if (need > capacity || (need > 0 && !out)) return TC_ERR_WORKSPACE;
    int64_t k = 0;
    for (int64_t i = 0; i < n_views; ++i)
      reshard_fragments(views[i], dst_tp, dst_rank, [&](const tc_fragment& f) { out[k++] = f; });
    *written = k;
    return TC_OK;
  } catch (...) {
    return TC_ERR_HOST_RESOURCES;  // host memory or threads
  }
}

int64_t tc_reshard_cast_item_count(const tc_reshard_view* views, int64_t n_views, int32_t dst_tp,
                                   int32_t dst_rank) {
  if (n_views < 0 || (n_views > 0 && !views)) return -1;
  int64_t count = 0;
  for (int64_t i = 0; i < n_views; ++i) {
    if (!reshard_ok(views[i], dst_tp, dst_rank)) return -1;
    if (!reshard_cast_items(views[i], 0, dst_tp, dst_rank, [&](const tc_cast_item&) { ++count; }))
      return -1;
  }
  return count;
}

tc_status tc_reshard_cast_items(const tc_reshard_view* views, const uint64_t* scale_off,
                                int64_t n_views, int32_t dst_tp, int32_t dst_rank, tc_cast_item* out,
                                int64_t capacity, int64_t* written) {
  try {
    if (!written || n_views < 0 || (n_views > 0 && (!views || !scale_off)) || capacity < 0)
      return TC_ERR_INVALID_ARGUMENT;
    const int64_t need = tc_reshard_cast_item_count(views, n_views, dst_tp, dst_rank);
    if (need < 0) return TC_ERR_INVALID_ARGUMENT;
    if (need > capacity || (need > 0 && !out)) return TC_ERR_WORKSPACE;
    int64_t k = 0;
    for (int64_t i = 0; i < n_views; ++i)
      reshard_cast_items(views[i], scale_off[i], dst_tp, dst_rank,
                         [&](const tc_cast_item& it) { out[k++] = it; });
    *written = k;
    return TC_OK;
  } catch (...) {
    return TC_ERR_HOST_RESOURCES;  // host memory or threads
  }
}

tc_status tc_tp_cast_item(const tc_tp_view* view, int32_t tp, int32_t rank, uint64_t scale_off,
                          tc_cast_item* out) {
  if (!view || !out) return TC_ERR_INVALID_ARGUMENT;
  if (view->elem_bytes != 2 || !view_ok(*view, tp, rank)) return TC_ERR_INVALID_ARGUMENT;
  if (view->src_off % 2) return TC_ERR_INVALID_ARGUMENT;
  const Slice sl = slice_of(*view, tp, rank);
  tc_cast_item it;
  it.src_off = view->src_off / 2 + sl.src_elem;
  it.rows = sl.rows;
  it.cols = sl.cols;
  it.src_ld = view->src_ld;
  it.dst_off = view->dst_off;
  it.dst_ld = view->dst_ld;
  it.scale_off = scale_off;
  it.scale_ld = (sl.cols + 127) / 128;
  *out = it;
  return TC_OK;
}

size_t tc_cast_fp8_workspace(int64_t n_items) {
  if (n_items < 0 || n_items > kMaxCount) return 0;
  return tc::cast_workspace_bytes(n_items);
}

size_t tc_dequant_fp8_workspace(int64_t n_items) {
  if (n_items < 0 || n_items > kMaxCount) return 0;
  return tc::cast_workspace_bytes(n_items);
}

size_t tc_cast_fp8_workspace_tiles(const tc_cast_item* items, int64_t n_items) {
  return workspace_with_tiles(items, n_items);
}

size_t tc_dequant_fp8_workspace_tiles(const tc_dequant_item* items, int64_t n_items) {
  return workspace_with_tiles(items, n_items);
}

tc_status tc_cast_fp8_prepare(const void* src_base, const void* dst_base, const tc_cast_item* items,
                              int64_t n_items, int32_t tile, void* workspace, size_t workspace_bytes,
                              tc_tile_plan* plan, hipStream_t stream) {
  try {
    return prepare_tiles(src_base, dst_base, items, n_items, tile, workspace, workspace_bytes, true,
                         plan, stream);
  } catch (...) {
    return TC_ERR_HOST_RESOURCES;  // host memory or threads
  }
}

tc_status tc_cast_fp8_planned(const void* src_base, void* dst_base, float* scale_base,
                              const void* workspace, size_t workspace_bytes,
                              const tc_tile_plan* plan, hipStream_t stream) {
  tc_status st = planned_args(src_base, dst_base, scale_base, workspace, workspace_bytes, plan);
  if (st != TC_OK || plan->full_tiles + plan->edge_tiles == 0) return st;
  return check(tc::launch_cast_blockscaled(static_cast<const uint16_t*>(src_base),
                                           static_cast<uint8_t*>(dst_base), scale_base, workspace,
                                           plan->n_items, plan->full_tiles, plan->edge_tiles,
                                           plan->tiled != 0, stream));
}

tc_status tc_cast_fp8_blockscaled(const void* src_base, void* dst_base, float* scale_base,
                                  const tc_cast_item* items, int64_t n_items, int32_t tile,
                                  void* workspace, size_t workspace_bytes, hipStream_t stream) {
  try {
    if (n_items < 0 || n_items > kMaxCount || tile != 128) return TC_ERR_INVALID_ARGUMENT;
    if (n_items == 0) return TC_OK;
    if (!scale_base || (uintptr_t)scale_base % 4) return TC_ERR_INVALID_ARGUMENT;
    if (validating() && src_base && dst_base && items) {
      tc_status st = check_cast_ranges(src_base, dst_base, scale_base, items, n_items);
      if (st != TC_OK) return st;
    }
    tc_tile_plan plan;
    tc_status st = tc_cast_fp8_prepare(src_base, dst_base, items, n_items, tile, workspace,
                                       workspace_bytes, &plan, stream);
    if (st != TC_OK) return st;
    return tc_cast_fp8_planned(src_base, dst_base, scale_base, workspace, workspace_bytes, &plan,
                               stream);
  } catch (...) {
    return TC_ERR_HOST_RESOURCES;  // host memory or threads
  }
}

tc_status tc_dequant_fp8_prepare(const void* codes_base, const void* dst_base,
                                 const tc_dequant_item* items, int64_t n_items, int32_t tile,
                                 void* workspace, size_t workspace_bytes, tc_tile_plan* plan,
                                 hipStream_t stream) {
  try {
    return prepare_tiles(codes_base, dst_base, items, n_items, tile, workspace, workspace_bytes,
                         false, plan, stream);
  } catch (...) {
    return TC_ERR_HOST_RESOURCES;  // host memory or threads
  }
}

tc_status tc_dequant_fp8_planned(const void* codes_base, const float* scale_base, void* dst_base,
                                 const void* workspace, size_t workspace_bytes,
                                 const tc_tile_plan* plan, hipStream_t stream) {
  tc_status st = planned_args(codes_base, dst_base, scale_base, workspace, workspace_bytes, plan);
  if (st != TC_OK || plan->full_tiles + plan->edge_tiles == 0) return st;
  return check(tc::launch_dequant_blockscaled(static_cast<const uint8_t*>(codes_base), scale_base,
                                              static_cast<uint16_t*>(dst_base), workspace,
                                              plan->n_items, plan->full_tiles, plan->edge_tiles,
                                              plan->tiled != 0, stream));
}

tc_status tc_dequant_fp8_blockscaled(const void* codes_base, const float* scale_base,
                                     void* dst_base, const tc_dequant_item* items, int64_t n_items,
                                     int32_t tile, void* workspace, size_t workspace_bytes,
                                     hipStream_t stream) {
  try {
    if (n_items < 0 || n_items > kMaxCount || tile != 128) return TC_ERR_INVALID_ARGUMENT;
    if (n_items == 0) return TC_OK;
    if (!scale_base || (uintptr_t)scale_base % 4) return TC_ERR_INVALID_ARGUMENT;
    if (validating() && codes_base && dst_base && items) {
      tc_status st = check_dequant_ranges(codes_base, scale_base, dst_base, items, n_items);
      if (st != TC_OK) return st;
    }
    tc_tile_plan plan;
    tc_status st = tc_dequant_fp8_prepare(codes_base, dst_base, items, n_items, tile, workspace,
                                          workspace_bytes, &plan, stream);
    if (st != TC_OK) return st;
    return tc_dequant_fp8_planned(codes_base, scale_base, dst_base, workspace, workspace_bytes,
                                  &plan, stream);
  } catch (...) {
    return TC_ERR_HOST_RESOURCES;  // host memory or threads
  }
}

tc_status tc_cast_fp8_scaled(const void* src_bf16, int64_t n, float scale, void* dst_e4m3,
                             hipStream_t stream) {
  if (n < 0) return TC_ERR_INVALID_ARGUMENT;
  if (n == 0) return TC_OK;
  if (!src_bf16 || !dst_e4m3 || (uintptr_t)src_bf16 % 2) return TC_ERR_INVALID_ARGUMENT;
  return check(tc::launch_cast_scaled(static_cast<const uint16_t*>(src_bf16), n, scale,
                                      static_cast<uint8_t*>(dst_e4m3), stream));
}

const char* tc_status_string(tc_status s) {
  switch (s) {
    case TC_OK: return "ok";
    case TC_ERR_INVALID_ARGUMENT: return "invalid argument";
    case TC_ERR_OUT_OF_RANGE: return "descriptor out of range";
    case TC_ERR_ALIAS: return "aliasing writes";
    case TC_ERR_HIP: return "HIP runtime error";
    case TC_ERR_WORKSPACE: return "workspace too small";
    case TC_ERR_HOST_RESOURCES: return "host memory or threads unavailable";
  }
  return "unknown status";
}

int tc_last_hip_error(void) { return g_last_hip_error; }

void tc_set_validate(int on) { g_validate.store(on ? 1 : 0, std::memory_order_relaxed); }

int tc_get_validate(void) { return validating() ? 1 : 0; }

}  // extern "C"
