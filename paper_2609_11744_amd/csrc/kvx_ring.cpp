// Bounded pinned staging ring and the staged restore (Sec. 6.4: one
// contiguous, aligned, pinned host allocation cut into fixed slots; a
// transfer larger than the pool moves piece by piece; a slot is reused only
// after the device event of the copy that read it has completed).
//
// Pipeline for piece i on slot s = i mod n_slots:
//   fill   host threads copy image bytes into host slot s, after the H2D copy
//          of piece i - n_slots (which read host slot s) has completed;
//   H2D    the side stream waits until the scatter of piece i - n_slots has
//          read device slot s, copies host slot s to device slot s, records
//          h2d_done[s];
//   scatter the caller's stream waits on h2d_done[s], runs the scatter kernel
//          from device slot s, records scatter_done[s].
// So the fill of piece i + 2, the H2D of piece i + 1 and the scatter of piece
// i overlap. The enqueuing thread never waits for the device; fill threads
// wait on h2d_done events (blocking-sync events, so they sleep).
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <new>
#include <thread>
#include <vector>

#include "kvx.h"
#include "kvx_internal.h"

struct kvx_ring {
  int device = 0;
  int32_t n_slots = 0;
  int64_t slot_bytes = 0;
  uint8_t* host = nullptr;     // n_slots * slot_bytes pinned bytes
  uint8_t* landing = nullptr;  // n_slots * slot_bytes device bytes
  bool owns_landing = false;
  hipStream_t side = nullptr;
  std::vector<hipEvent_t> h2d_done;
  std::vector<hipEvent_t> scatter_done;

  // binding
  bool bound = false;
  std::vector<void*> kptr, vptr;
  kvx_cache cache{};
  int32_t l0 = 0, l1 = 0, n_blocks = 0, chunk_tokens = 0;
  const uint8_t* source = nullptr;
  int32_t fill_threads = 0;
  std::vector<kvx_piece> pieces;

  // restore state: `closed` is set by kvx_ring_abort and stays set; `stop`
  // ends the current restore (closed, or an internal failure).
  std::atomic<bool> closed{false};
  std::atomic<bool> stop{false};
  std::atomic<int> worker_error{0};
  std::mutex mu;
  std::condition_variable cv_filled, cv_enqueued;
  int64_t enqueued = 0;
  std::vector<int32_t> parts_done;
  std::atomic<int64_t> fill_ns{0};
  kvx_ring_stats stats{};
};

namespace {

using clk = std::chrono::steady_clock;

double ms_since(clk::time_point t0) {
  return std::chrono::duration<double, std::milli>(clk::now() - t0).count();
}

// Restores the calling thread's current device on scope exit.
struct DeviceGuard {
  int prev = -1;
  bool ok = false;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) == hipSuccess) ok = hipSetDevice(dev) == hipSuccess;
  }
  ~DeviceGuard() {
    if (prev >= 0) (void)hipSetDevice(prev);
  }
};

void destroy_resources(kvx_ring* r) {
  if (r->side) (void)hipStreamSynchronize(r->side);
  for (hipEvent_t e : r->scatter_done)
    if (e) { (void)hipEventSynchronize(e); (void)hipEventDestroy(e); }
  for (hipEvent_t e : r->h2d_done)
    if (e) { (void)hipEventSynchronize(e); (void)hipEventDestroy(e); }
  r->scatter_done.clear();
  r->h2d_done.clear();
  if (r->side) (void)hipStreamDestroy(r->side);
  r->side = nullptr;
  if (r->host) (void)hipHostFree(r->host);
  r->host = nullptr;
  if (r->owns_landing && r->landing) (void)hipFree(r->landing);
  r->landing = nullptr;
}

// Fill thread w of t: copies its share of every piece into the piece's slot.
void fill_worker(kvx_ring* r, int w) {
  const int32_t S = r->n_slots;
  const int32_t T = r->fill_threads;
  const int64_t P = (int64_t)r->pieces.size();
  int64_t busy_ns = 0;
  for (int64_t i = 0; i < P; ++i) {
    const int32_t s = (int32_t)(i % S);
    if (i >= S) {
      // h2d_done[s] must hold the record of piece i - S before we wait on it.
      std::unique_lock<std::mutex> lock(r->mu);
      r->cv_enqueued.wait(lock, [&] { return r->enqueued > i - S || r->stop.load(); });
    }
    if (r->stop.load()) break;
    if (hipEventSynchronize(r->h2d_done[s]) != hipSuccess) {
      r->worker_error.store(1);
      r->stop.store(true);
      std::lock_guard<std::mutex> lock(r->mu);
      r->cv_filled.notify_all();
      r->cv_enqueued.notify_all();
      break;
    }
    const kvx_piece& p = r->pieces[(size_t)i];
    int64_t per = (p.bytes + T - 1) / T;
    per = (per + 4095) & ~(int64_t)4095;
    const int64_t a = std::min<int64_t>(p.bytes, per * w);
    const int64_t b = std::min<int64_t>(p.bytes, a + per);
    if (b > a) {
      auto t0 = clk::now();
      std::memcpy(r->host + (int64_t)s * r->slot_bytes + a, r->source + p.src_offset + a,
                  (size_t)(b - a));
      busy_ns += std::chrono::duration_cast<std::chrono::nanoseconds>(clk::now() - t0).count();
    }
    std::lock_guard<std::mutex> lock(r->mu);
    if (++r->parts_done[(size_t)i] == T) r->cv_filled.notify_all();
  }
  r->fill_ns.fetch_add(busy_ns);
}

kvx_status restore(kvx_ring* r, const int32_t* bt, hipStream_t stream) {
  if (!r->bound) return KVX_EINVAL;
  if (r->closed.load()) return KVX_ECLOSED;
  if (r->pieces.empty()) return KVX_OK;
  if (!bt) return KVX_EINVAL;
  DeviceGuard dg(r->device);
  if (!dg.ok) return KVX_EHIP;
  const auto t_start = clk::now();
  const int32_t S = r->n_slots;
  const int32_t T = r->fill_threads;
  const int64_t P = (int64_t)r->pieces.size();
  {
    std::lock_guard<std::mutex> lock(r->mu);
    r->enqueued = 0;
    r->parts_done.assign((size_t)P, 0);
  }
  r->worker_error.store(0);
  r->stop.store(false);
  r->fill_ns.store(0);
  std::vector<std::thread> workers;
  kvx_status st = KVX_OK;
  double wait_ms = 0;
  try {
    for (int w = 0; w < T; ++w) workers.emplace_back(fill_worker, r, w);
  } catch (...) {
    st = KVX_ENOMEM;
  }
  for (int64_t i = 0; st == KVX_OK && i < P; ++i) {
    const int32_t s = (int32_t)(i % S);
    const kvx_piece& p = r->pieces[(size_t)i];
    if (T > 0) {
      auto t0 = clk::now();
      std::unique_lock<std::mutex> lock(r->mu);
      r->cv_filled.wait(lock, [&] { return r->parts_done[(size_t)i] == T || r->stop.load(); });
      wait_ms += ms_since(t0);
    }
    if (r->stop.load() || r->closed.load()) {
      st = r->worker_error.load() ? KVX_EHIP : KVX_ECLOSED;
      break;
    }
    uint8_t* dslot = r->landing + (int64_t)s * r->slot_bytes;
    const uint8_t* hsrc = T > 0 ? r->host + (int64_t)s * r->slot_bytes : r->source + p.src_offset;
    if (hipStreamWaitEvent(r->side, r->scatter_done[s], 0) != hipSuccess ||
        hipMemcpyAsync(dslot, hsrc, (size_t)p.bytes, hipMemcpyHostToDevice, r->side) !=
            hipSuccess ||
        hipEventRecord(r->h2d_done[s], r->side) != hipSuccess) {
      st = KVX_EHIP;
      break;
    }
    {
      std::lock_guard<std::mutex> lock(r->mu);
      r->enqueued = i + 1;
    }
    r->cv_enqueued.notify_all();
    if (hipStreamWaitEvent(stream, r->h2d_done[s], 0) != hipSuccess) {
      st = KVX_EHIP;
      break;
    }
    kvx::Geometry g;
    st = kvx::validate(&r->cache, p.l_begin, p.l_end, p.n_blocks, p.chunk_tokens, true, &g);
    if (st != KVX_OK) break;
    st = kvx::launch_copy(false, &r->cache, p.l_begin, p.l_end, bt + p.bt_first, g, dslot, stream);
    if (st != KVX_OK) break;
    if (hipEventRecord(r->scatter_done[s], stream) != hipSuccess) {
      st = KVX_EHIP;
      break;
    }
  }
  if (st != KVX_OK) {
    r->stop.store(true);
    std::lock_guard<std::mutex> lock(r->mu);
    r->cv_filled.notify_all();
    r->cv_enqueued.notify_all();
  }
  for (auto& th : workers) th.join();
  r->stop.store(false);
  r->stats.pieces = st == KVX_OK ? P : 0;
  r->stats.bytes = 0;
  if (st == KVX_OK)
    for (const auto& p : r->pieces) r->stats.bytes += p.bytes;
  r->stats.fill_ms = (double)r->fill_ns.load() / 1e6;
  r->stats.wait_fill_ms = wait_ms;
  r->stats.enqueue_ms = ms_since(t_start);
  return st;
}

}  // namespace

extern "C" {

kvx_status kvx_ring_create(int device, int32_t n_slots, int64_t slot_bytes, void* device_landing,
                           kvx_ring** out) {
  if (!out) return KVX_EINVAL;
  *out = nullptr;
  if (n_slots < 1 || n_slots > 1024 || slot_bytes <= 0 || slot_bytes % 4096 != 0)
    return KVX_EINVAL;
  int64_t total = 0;
  if (__builtin_mul_overflow((int64_t)n_slots, slot_bytes, &total)) return KVX_EINVAL;
  if (device_landing && ((uintptr_t)device_landing & 15)) return KVX_EINVAL;
  kvx_ring* r = new (std::nothrow) kvx_ring();
  if (!r) return KVX_ENOMEM;
  try {
    DeviceGuard dg(device);
    if (!dg.ok) {
      delete r;
      return KVX_EINVAL;
    }
    r->device = device;
    r->n_slots = n_slots;
    r->slot_bytes = slot_bytes;
    kvx_status st = KVX_OK;
    void* h = nullptr;
    if (hipHostMalloc(&h, (size_t)total, hipHostMallocDefault) != hipSuccess) st = KVX_ENOMEM;
    r->host = (uint8_t*)h;
    if (st == KVX_OK) {
      if (device_landing) {
        r->landing = (uint8_t*)device_landing;
      } else {
        void* d = nullptr;
        if (hipMalloc(&d, (size_t)total) != hipSuccess) st = KVX_ENOMEM;
        r->landing = (uint8_t*)d;
        r->owns_landing = true;
      }
    }
    if (st == KVX_OK && hipStreamCreateWithFlags(&r->side, hipStreamNonBlocking) != hipSuccess)
      st = KVX_EHIP;
    r->h2d_done.assign((size_t)n_slots, nullptr);
    r->scatter_done.assign((size_t)n_slots, nullptr);
    for (int32_t s = 0; st == KVX_OK && s < n_slots; ++s) {
      if (hipEventCreateWithFlags(&r->h2d_done[s], hipEventDisableTiming | hipEventBlockingSync) !=
              hipSuccess ||
          hipEventCreateWithFlags(&r->scatter_done[s], hipEventDisableTiming) != hipSuccess)
        st = KVX_EHIP;
    }
    if (st != KVX_OK) {
      destroy_resources(r);
      delete r;
      return st;
    }
    *out = r;
    return KVX_OK;
  } catch (...) {
    destroy_resources(r);
    delete r;
    return KVX_EINTERNAL;
  }
}

kvx_status kvx_ring_bind(kvx_ring* r, const kvx_cache* cache, int32_t l0, int32_t l1,
                         int32_t n_blocks, int32_t chunk_tokens, const void* host_source,
                         int32_t fill_threads) {
  if (!r || !cache) return KVX_EINVAL;
  if (fill_threads < 0 || fill_threads > 64) return KVX_EINVAL;
  try {
    kvx::Geometry g;
    kvx_status st = kvx::validate(cache, l0, l1, n_blocks, chunk_tokens, true, &g);
    if (st != KVX_OK) return st;
    if (g.n_units > 0 && !host_source) return KVX_EINVAL;
    if (g.n_units > 0 && kvx::overlaps_cache(cache, l0, l1, r->landing,
                                             (int64_t)r->n_slots * r->slot_bytes))
      return KVX_EINVAL;
    if (g.n_units > 0 && fill_threads == 0) {
      hipPointerAttribute_t attr{};
      if (hipPointerGetAttributes(&attr, host_source) != hipSuccess ||
          attr.type != hipMemoryTypeHost)
        return KVX_EINVAL;  // direct H2D needs pinned memory
    }
    std::vector<kvx_piece> pieces;
    st = kvx::plan_pieces(g, l0, l1, cache->block_size, r->slot_bytes, &pieces);
    if (st != KVX_OK) return st;
    r->kptr.assign(cache->k, cache->k + cache->num_layers);
    r->vptr.assign(cache->v, cache->v + cache->num_layers);
    r->cache = *cache;
    r->cache.k = r->kptr.data();
    r->cache.v = r->vptr.data();
    r->l0 = l0;
    r->l1 = l1;
    r->n_blocks = n_blocks;
    r->chunk_tokens = chunk_tokens;
    r->source = (const uint8_t*)host_source;
    r->fill_threads = fill_threads;
    r->pieces.swap(pieces);
    r->bound = true;
    return KVX_OK;
  } catch (...) {
    return KVX_EINTERNAL;
  }
}

kvx_status kvx_restore_from_staging(kvx_ring* ring, const int32_t* block_table,
                                    hipStream_t stream) {
  if (!ring) return KVX_EINVAL;
  try {
    return restore(ring, block_table, stream);
  } catch (...) {
    return KVX_EINTERNAL;
  }
}

kvx_status kvx_ring_stats_get(const kvx_ring* ring, kvx_ring_stats* out) {
  if (!ring || !out) return KVX_EINVAL;
  *out = ring->stats;
  return KVX_OK;
}

kvx_status kvx_ring_abort(kvx_ring* ring) {
  if (!ring) return KVX_EINVAL;
  ring->closed.store(true);
  ring->stop.store(true);
  std::lock_guard<std::mutex> lock(ring->mu);
  ring->cv_filled.notify_all();
  ring->cv_enqueued.notify_all();
  return KVX_OK;
}

kvx_status kvx_ring_destroy(kvx_ring* ring) {
  if (!ring) return KVX_OK;
  try {
    DeviceGuard dg(ring->device);
    destroy_resources(ring);
  } catch (...) {
  }
  delete ring;
  return KVX_OK;
}

}  // extern "C"
