// Host <-> device staging: the pinned streaming buffers and asynchronous
// copy streams of the materialization pipeline (paper Sec. 5), for bytes that
// live in host memory (a host-resident transfer buffer, a host-memory tier
// of the Global Store).
//
// A stager owns a ring of pinned host slots, a copy stream and a few host
// threads.  Pageable host bytes pass through the ring: the host threads copy
// chunk k + 1 into a free slot while the DMA engine moves chunk k over PCIe
// and the device scatters chunk k - 1 into its block pool.  Pinned caller
// buffers skip the ring.  Measured on MI355X: one DMA reaches 57 GB/s each
// way over PCIe Gen5 x16, a host memcpy from pageable memory 27 GB/s per
// thread (90 GB/s with four), and hipMemcpy from pageable memory 27 GB/s
// host-to-device and 17 GB/s device-to-host.  The DMA engine, not a kernel,
// moves the bytes, so no compute unit is held while a transfer runs.
//
// Host-only code.  Every device copy is hipMemcpyAsync on the stager's copy
// stream; ordering against the caller's stream uses events only.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <condition_variable>
#include <cstring>
#include <functional>
#include <mutex>
#include <new>
#include <thread>
#include <vector>

#include "tc_internal.h"

namespace {

// Runs f(0 .. parts-1) on the worker threads and the calling thread.
class Workers {
 public:
  explicit Workers(int threads) {
    for (int i = 1; i < threads; ++i) th_.emplace_back([this] { loop(); });
  }
  ~Workers() {
    {
      std::lock_guard<std::mutex> l(m_);
      stop_ = true;
    }
    cv_.notify_all();
    for (std::thread& t : th_) t.join();
  }
  int size() const { return int(th_.size()) + 1; }
  void run(int parts, const std::function<void(int)>& f) {
    if (parts <= 0) return;
    if (th_.empty() || parts == 1) {
      for (int p = 0; p < parts; ++p) f(p);
      return;
    }
    {
      std::lock_guard<std::mutex> l(m_);
      job_ = &f;
      parts_ = parts;
      next_.store(0);
      busy_ = int(th_.size());
      ++gen_;
    }
    cv_.notify_all();
    work(f, parts);
    std::unique_lock<std::mutex> l(m_);
    done_.wait(l, [this] { return busy_ == 0; });
    job_ = nullptr;
  }

 private:
  void work(const std::function<void(int)>& f, int parts) {
    for (int p = next_.fetch_add(1); p < parts; p = next_.fetch_add(1)) f(p);
  }
  void loop() {
    uint64_t seen = 0;
    for (;;) {
      const std::function<void(int)>* job;
      int parts;
      {
        std::unique_lock<std::mutex> l(m_);
        cv_.wait(l, [&] { return stop_ || gen_ != seen; });
        if (stop_) return;
        seen = gen_;
        job = job_;
        parts = parts_;
      }
      work(*job, parts);
      {
        std::lock_guard<std::mutex> l(m_);
        if (--busy_ == 0) done_.notify_one();
      }
    }
  }
  std::vector<std::thread> th_;
  std::mutex m_;
  std::condition_variable cv_, done_;
  const std::function<void(int)>* job_ = nullptr;
  int parts_ = 0;
  std::atomic<int> next_{0};
  int busy_ = 0;
  uint64_t gen_ = 0;
  bool stop_ = false;
};

constexpr size_t kDefaultSlotBytes = size_t(32) << 20;
constexpr int kDefaultSlots = 4;
constexpr int kDefaultThreads = 4;
constexpr size_t kMinPart = size_t(1) << 20;  // smallest share of a host copy per thread
// Chunks in flight on the copy stream at most.  The host waits for chunk
// k - kDepth before it enqueues chunk k, in every path.  With the host far
// ahead (pinned buffers, rings of six slots) the same copies measured 15-30
// GB/s instead of 54 on MI355X.  Two stagers moving opposite directions at
// once reach 94-96 GB/s together at depths 2 and 3 but 63-71 at depth 4; at
// depth 1 a lone hydrate from pageable memory falls from 54 to 34 GB/s.
constexpr size_t kDepth = 2;

}  // namespace

struct tc_stager {
  int device = -1;
  size_t slot_bytes = 0;
  std::vector<void*> pinned;
  std::vector<hipEvent_t> pinned_free;  // the last DMA on the slot has finished
  std::vector<bool> pinned_used;
  std::vector<hipEvent_t> dev_free;     // the last reader/writer of a device slot has finished
  std::vector<hipEvent_t> dev_ready;    // a device slot's bytes are in place
  std::vector<bool> dev_used;
  hipEvent_t start = nullptr, end = nullptr;
  hipStream_t copy = nullptr;
  Workers* workers = nullptr;
  std::mutex mu;
};

namespace {

tc_status fail(hipError_t e) { return tc::hip_status(e); }

void release(tc_stager* st) {
  if (!st) return;
  if (st->copy) (void)hipStreamSynchronize(st->copy);
  for (void* p : st->pinned)
    if (p) (void)hipHostFree(p);
  for (hipEvent_t e : st->pinned_free)
    if (e) (void)hipEventDestroy(e);
  for (hipEvent_t e : st->dev_free)
    if (e) (void)hipEventDestroy(e);
  for (hipEvent_t e : st->dev_ready)
    if (e) (void)hipEventDestroy(e);
  if (st->start) (void)hipEventDestroy(st->start);
  if (st->end) (void)hipEventDestroy(st->end);
  if (st->copy) (void)hipStreamDestroy(st->copy);
  delete st->workers;
  delete st;
}

hipError_t new_event(hipEvent_t* e) { return hipEventCreateWithFlags(e, hipEventDisableTiming); }

// The calling thread must be on the stager's device.
tc_status same_device(const tc_stager* st) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(e);
  return dev == st->device ? TC_OK : TC_ERR_INVALID_ARGUMENT;
}

// At least `count` device-slot events.
tc_status ensure_dev_slots(tc_stager* st, size_t count) {
  while (st->dev_free.size() < count) {
    hipEvent_t a = nullptr, b = nullptr;
    hipError_t e = new_event(&a);
    if (e == hipSuccess) e = new_event(&b);
    if (e != hipSuccess) {
      if (a) (void)hipEventDestroy(a);
      return fail(e);
    }
    st->dev_free.push_back(a);
    st->dev_ready.push_back(b);
    st->dev_used.push_back(false);
  }
  return TC_OK;
}

// Host copy split over the workers in shares of at least 1 MiB.
void par_copy(tc_stager* st, void* dst, const void* src, size_t bytes) {
  const int parts = (int)std::max<size_t>(1, std::min<size_t>(st->workers->size(), bytes / kMinPart));
  const size_t share = (bytes + parts - 1) / parts;
  st->workers->run(parts, [&](int p) {
    const size_t a = size_t(p) * share;
    if (a >= bytes) return;
    std::memcpy(static_cast<uint8_t*>(dst) + a, static_cast<const uint8_t*>(src) + a,
                std::min(share, bytes - a));
  });
}

// Wait until pinned slot j is no longer read or written by a DMA.
tc_status wait_pinned(tc_stager* st, size_t j) {
  if (!st->pinned_used[j]) return TC_OK;
  return fail(hipEventSynchronize(st->pinned_free[j]));
}

// Before chunk k is enqueued: chunk k - min(S, kDepth) has left the copy
// stream (DMAs complete in order), which also frees pinned slot k % S.
tc_status pace(tc_stager* st, size_t k) {
  const size_t S = st->pinned.size(), W = std::min(S, kDepth);
  if (k < W) return wait_pinned(st, k % S);  // a previous call's DMA on this slot
  return fail(hipEventSynchronize(st->pinned_free[(k - W) % S]));
}

// The copy stream starts after everything already enqueued on `stream`.
tc_status copy_after(tc_stager* st, hipStream_t stream) {
  hipError_t e = hipEventRecord(st->start, stream);
  if (e == hipSuccess) e = hipStreamWaitEvent(st->copy, st->start, 0);
  return fail(e);
}

// `stream` continues after everything enqueued on the copy stream.
tc_status stream_after_copy(tc_stager* st, hipStream_t stream) {
  hipError_t e = hipEventRecord(st->end, st->copy);
  if (e == hipSuccess) e = hipStreamWaitEvent(stream, st->end, 0);
  return fail(e);
}

// Validation mode: every id in range and, for a scatter, no id twice (the
// per-chunk calls cannot see repeats across chunks).
tc_status check_ids(const tc_block_pool* pool, const int32_t* ids, int64_t n, bool scatter,
                    hipStream_t stream) {
  std::vector<int32_t> h((size_t)n);
  hipError_t e = hipStreamSynchronize(stream);
  if (e == hipSuccess) e = hipMemcpy(h.data(), ids, sizeof(int32_t) * (size_t)n, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return fail(e);
  std::vector<uint8_t> seen((size_t)std::max<int64_t>(pool->num_blocks, 0), 0);
  for (int32_t id : h) {
    if (id < 0 || id >= pool->num_blocks) return TC_ERR_OUT_OF_RANGE;
    if (scatter && seen[(size_t)id]) return TC_ERR_ALIAS;
    seen[(size_t)id] = 1;
  }
  return TC_OK;
}

}  // namespace

extern "C" {

tc_status tc_stager_create(size_t slot_bytes, int32_t slots, int32_t host_threads,
                           tc_stager** out) {
  if (!out) return TC_ERR_INVALID_ARGUMENT;
  *out = nullptr;
  if (slots < 0 || host_threads < 0 || slots > 64 || host_threads > 64)
    return TC_ERR_INVALID_ARGUMENT;
  if (slot_bytes == 0) slot_bytes = kDefaultSlotBytes;
  if (slots == 0) slots = kDefaultSlots;
  if (host_threads == 0) host_threads = kDefaultThreads;
  if (slots < 2 || slot_bytes < 4096) return TC_ERR_INVALID_ARGUMENT;
  tc_stager* st = new (std::nothrow) tc_stager;
  if (!st) return TC_ERR_HOST_RESOURCES;
  st->slot_bytes = slot_bytes;
  hipError_t e = hipGetDevice(&st->device);
  if (e == hipSuccess) e = hipStreamCreateWithFlags(&st->copy, hipStreamNonBlocking);
  if (e == hipSuccess) e = new_event(&st->start);
  if (e == hipSuccess) e = new_event(&st->end);
  st->pinned.reserve(size_t(slots));
  st->pinned_free.reserve(size_t(slots));
  st->pinned_used.reserve(size_t(slots));
  for (int32_t j = 0; e == hipSuccess && j < slots; ++j) {
    void* p = nullptr;
    hipEvent_t ev = nullptr;
    e = hipHostMalloc(&p, slot_bytes, hipHostMallocDefault);
    if (e == hipSuccess) st->pinned.push_back(p);
    if (e == hipSuccess) e = new_event(&ev);
    if (e == hipSuccess) {
      st->pinned_free.push_back(ev);
      st->pinned_used.push_back(false);
    }
  }
  if (e != hipSuccess) {
    release(st);
    return fail(e);
  }
  try {
    st->workers = new Workers(host_threads);
  } catch (...) {  // threads or memory unavailable
    release(st);
    return TC_ERR_HOST_RESOURCES;
  }
  *out = st;
  return TC_OK;
}

tc_status tc_stager_destroy(tc_stager* st) {
  if (!st) return TC_OK;
  release(st);
  return TC_OK;
}

tc_status tc_stage_h2d(tc_stager* st, const void* host_src, void* dev_dst, size_t bytes,
                       int32_t flags, hipStream_t stream) {
  try {
    if (!st || (flags & ~TC_HOST_PINNED)) return TC_ERR_INVALID_ARGUMENT;
    if (bytes == 0) return TC_OK;
    if (!host_src || !dev_dst) return TC_ERR_INVALID_ARGUMENT;
    std::lock_guard<std::mutex> lock(st->mu);
    tc_status s = same_device(st);
    if (s == TC_OK) s = copy_after(st, stream);
    if (s != TC_OK) return s;
    const uint8_t* src = static_cast<const uint8_t*>(host_src);
    uint8_t* dst = static_cast<uint8_t*>(dev_dst);
    const bool pinned = flags & TC_HOST_PINNED;
    const size_t C = st->slot_bytes, S = st->pinned.size();
    for (size_t k = 0, off = 0; off < bytes; ++k, off += C) {
      const size_t j = k % S, len = std::min(C, bytes - off);
      if ((s = pace(st, k)) != TC_OK) return s;
      const void* from = src + off;
      if (!pinned) {
        par_copy(st, st->pinned[j], from, len);
        from = st->pinned[j];
      }
      hipError_t e = hipMemcpyAsync(dst + off, from, len, hipMemcpyHostToDevice, st->copy);
      if (e == hipSuccess) e = hipEventRecord(st->pinned_free[j], st->copy);
      if (e != hipSuccess) return fail(e);
      st->pinned_used[j] = true;
    }
    return stream_after_copy(st, stream);
  } catch (...) {
    return TC_ERR_HOST_RESOURCES;  // host memory or threads
  }
}

tc_status tc_stage_d2h(tc_stager* st, const void* dev_src, void* host_dst, size_t bytes,
                       int32_t flags, hipStream_t stream) {
  try {
    if (!st || (flags & ~TC_HOST_PINNED)) return TC_ERR_INVALID_ARGUMENT;
    if (bytes == 0) return TC_OK;
    if (!host_dst || !dev_src) return TC_ERR_INVALID_ARGUMENT;
    std::lock_guard<std::mutex> lock(st->mu);
    tc_status s = same_device(st);
    if (s == TC_OK) s = copy_after(st, stream);
    if (s != TC_OK) return s;
    const uint8_t* src = static_cast<const uint8_t*>(dev_src);
    uint8_t* dst = static_cast<uint8_t*>(host_dst);
    const bool pinned = flags & TC_HOST_PINNED;
    const size_t C = st->slot_bytes, S = st->pinned.size();
    const size_t chunks = (bytes + C - 1) / C;
    // Pageable: chunk k lands in slot k % S and is copied out by the host once
    // its DMA is done; the host drains chunk k - S before chunk k reuses the
    // slot, so later DMAs stay queued while the host copies.
    auto drain = [&](size_t k) -> tc_status {
      const size_t j = k % S, off = k * C, len = std::min(C, bytes - off);
      tc_status r = fail(hipEventSynchronize(st->pinned_free[j]));
      if (r != TC_OK) return r;
      par_copy(st, dst + off, st->pinned[j], len);
      return TC_OK;
    };
    for (size_t k = 0; k < chunks; ++k) {
      const size_t j = k % S, off = k * C, len = std::min(C, bytes - off);
      if (!pinned && k >= S && (s = drain(k - S)) != TC_OK) return s;
      if ((s = pace(st, k)) != TC_OK) return s;
      void* to = pinned ? static_cast<void*>(dst + off) : st->pinned[j];
      hipError_t e = hipMemcpyAsync(to, src + off, len, hipMemcpyDeviceToHost, st->copy);
      if (e == hipSuccess) e = hipEventRecord(st->pinned_free[j], st->copy);
      if (e != hipSuccess) return fail(e);
      st->pinned_used[j] = true;
    }
    if (pinned) return fail(hipStreamSynchronize(st->copy));
    for (size_t k = chunks > S ? chunks - S : 0; k < chunks; ++k)
      if ((s = drain(k)) != TC_OK) return s;
    return TC_OK;
  } catch (...) {
    return TC_ERR_HOST_RESOURCES;  // host memory or threads
  }
}

tc_status tc_hydrate_from_host(tc_stager* st, const tc_block_pool* pool, const int32_t* ids,
                               int64_t n, const void* host_src, int32_t flags, void* dev_stage,
                               size_t dev_stage_bytes, hipStream_t stream) {
  try {
    if (!st || n < 0 || !tc::pool_valid(pool) || (flags & ~TC_HOST_PINNED))
      return TC_ERR_INVALID_ARGUMENT;
    if (n == 0) return TC_OK;
    if (!ids || !host_src || !dev_stage) return TC_ERR_INVALID_ARGUMENT;
    const uint64_t per_id = uint64_t(pool->num_regions) * uint64_t(pool->block_bytes);
    const uint64_t m = std::min<uint64_t>(st->slot_bytes / per_id, uint64_t(n));  // ids per chunk
    if (m == 0) return TC_ERR_WORKSPACE;
    const uint64_t chunk = m * per_id;
    const uint64_t D = std::min<uint64_t>(dev_stage_bytes / chunk, 8);  // device slots
    if (D == 0) return TC_ERR_WORKSPACE;
    std::lock_guard<std::mutex> lock(st->mu);
    tc_status s = same_device(st);
    if (s == TC_OK && tc_get_validate()) s = check_ids(pool, ids, n, true, stream);
    if (s == TC_OK) s = ensure_dev_slots(st, D);
    if (s == TC_OK) s = copy_after(st, stream);
    if (s != TC_OK) return s;
    const bool pinned = flags & TC_HOST_PINNED;
    const size_t S = st->pinned.size();
    const uint8_t* src = static_cast<const uint8_t*>(host_src);
    uint8_t* stage = static_cast<uint8_t*>(dev_stage);
    for (uint64_t k = 0, i0 = 0; i0 < uint64_t(n); ++k, i0 += m) {
      const uint64_t cnt = std::min<uint64_t>(m, uint64_t(n) - i0), bytes = cnt * per_id;
      const size_t j = k % S, dj = k % D;
      const uint8_t* from = src + i0 * per_id;
      if ((s = pace(st, k)) != TC_OK) return s;
      if (!pinned) {
        par_copy(st, st->pinned[j], from, bytes);
        from = static_cast<const uint8_t*>(st->pinned[j]);
      }
      hipError_t e = hipSuccess;
      if (st->dev_used[dj]) e = hipStreamWaitEvent(st->copy, st->dev_free[dj], 0);
      if (e == hipSuccess)
        e = hipMemcpyAsync(stage + dj * chunk, from, bytes, hipMemcpyHostToDevice, st->copy);
      if (e == hipSuccess) e = hipEventRecord(st->pinned_free[j], st->copy);
      if (e == hipSuccess) e = hipEventRecord(st->dev_ready[dj], st->copy);
      if (e == hipSuccess) e = hipStreamWaitEvent(stream, st->dev_ready[dj], 0);
      if (e != hipSuccess) return fail(e);
      st->pinned_used[j] = true;
      s = tc_scatter_blocks(pool, ids + i0, int64_t(cnt), stage + dj * chunk, stream);
      if (s != TC_OK) return s;
      if ((e = hipEventRecord(st->dev_free[dj], stream)) != hipSuccess) return fail(e);
      st->dev_used[dj] = true;
    }
    return TC_OK;
  } catch (...) {
    return TC_ERR_HOST_RESOURCES;  // host memory or threads
  }
}

tc_status tc_publish_to_host(tc_stager* st, const tc_block_pool* pool, const int32_t* ids,
                             int64_t n, void* host_dst, int32_t flags, void* dev_stage,
                             size_t dev_stage_bytes, hipStream_t stream) {
  try {
    if (!st || n < 0 || !tc::pool_valid(pool) || (flags & ~TC_HOST_PINNED))
      return TC_ERR_INVALID_ARGUMENT;
    if (n == 0) return TC_OK;
    if (!ids || !host_dst || !dev_stage) return TC_ERR_INVALID_ARGUMENT;
    const uint64_t per_id = uint64_t(pool->num_regions) * uint64_t(pool->block_bytes);
    const uint64_t m = std::min<uint64_t>(st->slot_bytes / per_id, uint64_t(n));
    if (m == 0) return TC_ERR_WORKSPACE;
    const uint64_t chunk = m * per_id;
    const uint64_t D = std::min<uint64_t>(dev_stage_bytes / chunk, 8);
    if (D == 0) return TC_ERR_WORKSPACE;
    std::lock_guard<std::mutex> lock(st->mu);
    tc_status s = same_device(st);
    if (s == TC_OK && tc_get_validate()) s = check_ids(pool, ids, n, false, stream);
    if (s == TC_OK) s = ensure_dev_slots(st, D);
    if (s != TC_OK) return s;
    const bool pinned = flags & TC_HOST_PINNED;
    const size_t S = st->pinned.size();
    uint8_t* dst = static_cast<uint8_t*>(host_dst);
    uint8_t* stage = static_cast<uint8_t*>(dev_stage);
    const uint64_t chunks = (uint64_t(n) + m - 1) / m;
    auto chunk_of = [&](uint64_t k, uint64_t* off, uint64_t* bytes) {
      const uint64_t i0 = k * m, cnt = std::min<uint64_t>(m, uint64_t(n) - i0);
      *off = i0 * per_id;
      *bytes = cnt * per_id;
    };
    auto drain = [&](uint64_t k) -> tc_status {
      uint64_t off, bytes;
      chunk_of(k, &off, &bytes);
      const size_t j = k % S;
      tc_status r = fail(hipEventSynchronize(st->pinned_free[j]));
      if (r != TC_OK) return r;
      par_copy(st, dst + off, st->pinned[j], bytes);
      return TC_OK;
    };
    for (uint64_t k = 0; k < chunks; ++k) {
      uint64_t off, bytes;
      chunk_of(k, &off, &bytes);
      const size_t j = k % S, dj = k % D;
      hipError_t e = hipSuccess;
      if (st->dev_used[dj]) e = hipStreamWaitEvent(stream, st->dev_free[dj], 0);
      if (e != hipSuccess) return fail(e);
      s = tc_gather_blocks(pool, ids + k * m, int64_t(bytes / per_id), stage + dj * chunk, stream);
      if (s != TC_OK) return s;
      e = hipEventRecord(st->dev_ready[dj], stream);
      if (e == hipSuccess) e = hipStreamWaitEvent(st->copy, st->dev_ready[dj], 0);
      if (e != hipSuccess) return fail(e);
      if (!pinned && k >= S && (s = drain(k - S)) != TC_OK) return s;
      if ((s = pace(st, k)) != TC_OK) return s;
      void* to = pinned ? static_cast<void*>(dst + off) : st->pinned[j];
      e = hipMemcpyAsync(to, stage + dj * chunk, bytes, hipMemcpyDeviceToHost, st->copy);
      if (e == hipSuccess) e = hipEventRecord(st->pinned_free[j], st->copy);
      if (e == hipSuccess) e = hipEventRecord(st->dev_free[dj], st->copy);
      if (e != hipSuccess) return fail(e);
      st->pinned_used[j] = true;
      st->dev_used[dj] = true;
    }
    if (pinned) return fail(hipStreamSynchronize(st->copy));
    for (uint64_t k = chunks > S ? chunks - S : 0; k < chunks; ++k)
      if ((s = drain(k)) != TC_OK) return s;
    return TC_OK;
  } catch (...) {
    return TC_ERR_HOST_RESOURCES;  // host memory or threads
  }
}

}  // extern "C"
