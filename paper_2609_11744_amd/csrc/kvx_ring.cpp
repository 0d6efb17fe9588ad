// Bounded pinned staging ring: the staged restore (load) and the staged
// offload (store) of Sec. 6.4. The pool is one contiguous, aligned, pinned
// host allocation cut into fixed slots; a transfer larger than the pool moves
// piece by piece; a slot is reused only after the copy that last used it has
// completed. Stores use the reverse pipeline.
//
// Restore, piece i on slot s = i mod n_slots:
//   fill    host threads copy the piece's chunk images into host slot s, after
//           the H2D copy of piece i - n_slots (which read host slot s) is done;
//   H2D     once the scatter of piece i - n_slots has finished reading device
//           slot s (the host waits on dev_done[s]), host slot s is copied to
//           device slot s by a DMA engine, completion on dma_done[s];
//   scatter once the host has seen that copy complete, the caller's stream
//           runs one fused chunk-list scatter from device slot s and records
//           dev_done[s]. The copy of piece i + 1 is issued before the host
//           waits for the copy of piece i, so the engine always holds the
//           next copy and the link does not idle while a scatter is launched.
// Offload, piece i on slot s:
//   gather  once the D2H copy of piece i - n_slots has left device slot s,
//           the caller's stream runs one fused chunk-list gather into it and
//           records dev_done[s] (a system-scope release);
//   D2H     when dev_done[s] has completed and the drain threads have emptied
//           host slot s, device slot s is copied to host slot s by a DMA
//           engine, completion on dma_done[s];
//   drain   host threads wait on dma_done[s] and copy host slot s to the
//           chunks' destinations.
// The copies are issued to the GPU's DMA engines directly (HSA async copy).
// Enqueued through the HIP runtime, a device-to-host copy may run as a copy
// kernel instead, which occupies compute units for the whole link-bound
// transfer and starves the kernels it was meant to overlap (Sec. 5.1 contrasts
// DMA copies with a copy kernel that consumes GPU compute); and choosing the
// engines makes a restore and an offload running at once use the link in
// both directions (an H2D and a D2H engine that share a link path split it
// instead). The engines are chosen once per device by timing (pick_engines).
// A kernel launched after the host has observed a DMA completion reads the
// copied bytes: the launch acquires device memory at system scope. If the DMA
// engines cannot be set up, both directions fall back to HIP copies on a side
// stream ordered by copy_done / dev_done events (the restore's enqueuing
// thread then never waits for the device), and the ring's stats say so.
// Fill and drain threads wait on copy_done events or DMA signals (they sleep).
#include <hip/hip_runtime_api.h>
#include <hsa/hsa.h>
#include <hsa/hsa_ext_amd.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <thread>
#include <unordered_map>
#include <utility>
#include <vector>

#include "kvx.h"
#include "kvx_internal.h"
#include "kvx_io.h"
#include "kvx_preload.h"

namespace {
enum class Dir { kNone, kRestore, kOffload };
}

struct kvx_ring {
  int device = 0;
  int32_t n_slots = 0;
  int64_t slot_bytes = 0;
  uint8_t* host = nullptr;     // n_slots * slot_bytes pinned bytes
  uint8_t* landing = nullptr;  // n_slots * slot_bytes device bytes
  bool owns_landing = false;
  hipStream_t side = nullptr;
  std::vector<hipEvent_t> copy_done;  // H2D / D2H of the slot's last piece (host waits)
  std::vector<hipEvent_t> dev_done;   // scatter / gather of the slot's last piece

  // host-link copies on the DMA engines
  bool dma = false;
  bool hsa_up = false;
  hsa_agent_t gpu_agent{}, cpu_agent{};
  uint32_t d2h_engine = 0, h2d_engine = 0;  // SDMA engine id bits; 0: the runtime's choice
  std::vector<hsa_signal_t> dma_done;       // per slot: copies of its last piece still running

  // binding
  Dir dir = Dir::kNone;
  std::vector<void*> kptr, vptr;
  kvx_cache cache{};
  int32_t chunk_tokens = 0;
  int32_t threads = 0;  // fill (restore) or drain (offload) threads
  kvx::Plan plan;
  kvx_chunk_ref* d_refs = nullptr;  // device copy of plan.refs
  size_t d_refs_cap = 0;

  // transfer state: `closed` is set by kvx_ring_abort and stays set; `stop`
  // ends the current transfer (closed, or an internal failure).
  std::atomic<bool> closed{false};
  std::atomic<bool> stop{false};
  std::atomic<int> worker_error{0};  // a fill / drain failure's kvx_status (0: none)
  std::mutex mu;
  std::condition_variable cv_host, cv_enqueued;
  int64_t enqueued = 0;               // pieces whose slot copy is enqueued
  std::vector<int32_t> parts_done;    // per piece: fill / drain parts finished
  std::atomic<int64_t> busy_ns{0};
  kvx_ring_stats stats{};

  // fill (restore) or drain (offload) threads, kept from one transfer to the
  // next: started by the first transfer that needs them (or again when a
  // bind changes their direction or count), parked on cv_pool in between,
  // joined by kvx_ring_destroy. Creating them per transfer put their start-up
  // on every transfer's path: the first piece's fill shares began 0-130 us
  // apart, one thread created at a time.
  std::vector<std::thread> pool;
  Dir pool_dir = Dir::kNone;
  uint64_t pool_gen = 0;   // transfers handed to the pool (guarded by mu)
  int32_t pool_done = 0;   // workers done with the current one (guarded by mu)
  bool pool_quit = false;  // guarded by mu
  std::condition_variable cv_pool, cv_pool_done;

  // test hooks (kvx_ring_set_test_hooks)
  int32_t hook_max_delay_us = 0;
  bool hook_poison = false;
  bool hook_hip_copies = false;  // copies through the HIP runtime even with the DMA engines set up

  // the running transfer's kernels report bad block ids here: the error word
  // of the stream the caller passed
  int* err_word = nullptr;

  // deferred store (kvx_offload_begin / kvx_offload_wait) and asynchronous
  // restore (kvx_restore_begin / kvx_restore_wait): the gathers or scatters
  // run on store_stream after store_begin (recorded on the caller's stream);
  // an asynchronous restore records restore_end on it after its last scatter
  hipStream_t store_stream = nullptr;
  hipEvent_t store_begin = nullptr;
  hipEvent_t restore_end = nullptr;
  std::atomic<bool> async_busy{false};
  Dir async_dir = Dir::kNone;
  kvx_status async_status = KVX_OK;
  // The thread that runs them, kept from one call to the next: started by
  // the first begin, parked on cv_async in between, joined by
  // kvx_ring_destroy once a posted transfer has run. A begin posts the
  // transfer (async_posted) and its wait waits for async_done.
  std::thread async_th;
  std::mutex async_mu;
  std::condition_variable cv_async;
  bool async_posted = false, async_done = false, async_quit = false;  // guarded by async_mu
  const int32_t* async_bt = nullptr;
  hipStream_t async_own = nullptr;
  int* async_err = nullptr;

  // storage tier: the bound chunks live in files (kvx_ring_bind_files /
  // kvx_ring_bind_offload_files); a reactor thread replaces the fill / drain
  // threads
  bool files_mode = false;
  int32_t io_depth = 0;
  std::vector<kvx::TierFile> files;

  // restore out of a preloader's pool (kvx_ring_bind_preloaded): bound chunk c
  // is the image of file pre_paths[pre_file[c]], held for each restore and
  // copied to the device as soon as it is staged
  kvx_preloader* pre = nullptr;
  std::vector<std::string> pre_paths;  // distinct files, in chunk order
  std::vector<int32_t> pre_file;       // per bound chunk
  std::vector<int64_t> pre_bytes;      // per distinct file: its image bytes

  // timeline (kvx_ring_set_trace): the last traced transfer's intervals.
  // trace is the switch; trace_run its value for the running transfer, read
  // by its threads (set before they start).
  bool trace = false;
  bool trace_run = false;
  bool traced = false;                    // the last transfer was traced and succeeded
  bool trace_resolved = false;            // its device intervals are in trace_ev
  bool trace_to_packed = false;
  int64_t trace_pieces = 0;
  std::vector<kvx_trace_event> trace_ev;  // host-clock intervals (guarded by mu)
  std::vector<hipEvent_t> trace_k;        // per piece: timing events around its launch
  std::vector<hipEvent_t> trace_c;        // per piece: around its runtime host-link copy
  std::vector<uint8_t> trace_k_used, trace_c_used;
  std::vector<int64_t> trace_k_bytes, trace_c_bytes;
  std::vector<int64_t> trace_dma_piece;   // per slot: piece whose copy time is unread, or -1
  std::vector<int64_t> trace_dma_bytes;
  hipEvent_t trace_ref = nullptr;         // recorded and waited for at the transfer's start
  int64_t trace_ref_ns = 0;               // host clock when it was seen complete
  uint64_t trace_hsa0 = 0, trace_hsa_hz = 0;
  int64_t trace_host0 = 0;                // host clock at HSA system time trace_hsa0
};

namespace {

using clk = std::chrono::steady_clock;

int64_t now_ns() {
  return std::chrono::duration_cast<std::chrono::nanoseconds>(clk::now().time_since_epoch())
      .count();
}

// HSA async-copy profiling is process-wide: on while any ring traces.
void copy_profiling(bool on) {
  static std::mutex mu;
  static int users = 0;
  std::lock_guard<std::mutex> lock(mu);
  if (on) {
    if (users++ == 0) (void)hsa_amd_profiling_async_copy_enable(true);
  } else if (users > 0 && --users == 0) {
    (void)hsa_amd_profiling_async_copy_enable(false);
  }
}

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

// Whether this ring's copies go to the DMA engines.
bool use_dma(const kvx_ring* r) { return r->dma && !r->hook_hip_copies; }

// Block until the slot's DMA copies have finished; false if one failed.
bool wait_dma(kvx_ring* r, int32_t s) {
  return hsa_signal_wait_scacquire(r->dma_done[(size_t)s], HSA_SIGNAL_CONDITION_LT, 1, UINT64_MAX,
                                   HSA_WAIT_STATE_BLOCKED) == 0;
}

// Block until the host-link copy of the slot's last piece has finished.
bool wait_copy(kvx_ring* r, int32_t s) {
  return use_dma(r) ? wait_dma(r, s) : hipEventSynchronize(r->copy_done[(size_t)s]) == hipSuccess;
}

// Whether that copy has finished successfully (a failed one never counts as
// finished: wait_copy reports it).
bool copy_finished(kvx_ring* r, int32_t s) {
  if (use_dma(r)) return hsa_signal_load_scacquire(r->dma_done[(size_t)s]) == 0;
  return hipEventQuery(r->copy_done[(size_t)s]) == hipSuccess;
}

// Wait until nothing the ring enqueued can still touch its slots or tables.
void drain_device(kvx_ring* r) {
  for (size_t s = 0; s < r->dma_done.size(); ++s) (void)wait_dma(r, (int32_t)s);
  if (r->side) (void)hipStreamSynchronize(r->side);
  if (r->store_stream) (void)hipStreamSynchronize(r->store_stream);
  for (hipEvent_t e : r->dev_done)
    if (e) (void)hipEventSynchronize(e);
  for (hipEvent_t e : r->copy_done)
    if (e) (void)hipEventSynchronize(e);
}

void signal_stop(kvx_ring* r);
void stop_pool(kvx_ring* r);

void destroy_resources(kvx_ring* r) {
  signal_stop(r);  // pool threads blocked inside a transfer return to the pool
  stop_pool(r);
  drain_device(r);
  for (hipEvent_t e : r->dev_done)
    if (e) (void)hipEventDestroy(e);
  for (hipEvent_t e : r->copy_done)
    if (e) (void)hipEventDestroy(e);
  r->dev_done.clear();
  r->copy_done.clear();
  for (hsa_signal_t sig : r->dma_done) (void)hsa_signal_destroy(sig);
  r->dma_done.clear();
  for (hipEvent_t e : r->trace_k) (void)hipEventDestroy(e);
  for (hipEvent_t e : r->trace_c) (void)hipEventDestroy(e);
  r->trace_k.clear();
  r->trace_c.clear();
  if (r->trace_ref) (void)hipEventDestroy(r->trace_ref);
  r->trace_ref = nullptr;
  if (r->trace && r->hsa_up) copy_profiling(false);
  r->trace = false;
  r->traced = false;
  if (r->hsa_up) (void)hsa_shut_down();
  r->hsa_up = false;
  r->dma = false;
  if (r->side) (void)hipStreamDestroy(r->side);
  r->side = nullptr;
  if (r->store_stream) {
    (void)hipStreamSynchronize(r->store_stream);
    (void)hipStreamDestroy(r->store_stream);
  }
  r->store_stream = nullptr;
  if (r->store_begin) (void)hipEventDestroy(r->store_begin);
  r->store_begin = nullptr;
  if (r->restore_end) (void)hipEventDestroy(r->restore_end);
  r->restore_end = nullptr;
  if (r->host) (void)hipHostFree(r->host);
  r->host = nullptr;
  if (r->owns_landing && r->landing) (void)hipFree(r->landing);
  r->landing = nullptr;
  if (r->d_refs) (void)hipFree(r->d_refs);
  r->d_refs = nullptr;
  r->d_refs_cap = 0;
  for (auto& f : r->files) kvx::close_tier_file(&f);
  r->files.clear();
}

// Copy share w of T of a piece between host slot s and its spans.
int64_t copy_share(kvx_ring* r, const kvx::Piece& p, int32_t s, int w, int T, bool to_slot) {
  int64_t per = (p.bytes + T - 1) / T;
  per = (per + 4095) & ~(int64_t)4095;
  const int64_t a = std::min<int64_t>(p.bytes, per * w);
  const int64_t b = std::min<int64_t>(p.bytes, a + per);
  uint8_t* slot = r->host + (int64_t)s * r->slot_bytes;
  for (const kvx::Span& sp : p.spans) {
    const int64_t lo = std::max<int64_t>(a, sp.slot_off);
    const int64_t hi = std::min<int64_t>(b, sp.slot_off + sp.bytes);
    if (hi <= lo) continue;
    uint8_t* h = sp.host + (lo - sp.slot_off);
    if (to_slot)
      std::memcpy(slot + lo, h, (size_t)(hi - lo));
    else
      std::memcpy(h, slot + lo, (size_t)(hi - lo));
  }
  return b - a;
}

void signal_stop(kvx_ring* r) {
  r->stop.store(true);
  std::lock_guard<std::mutex> lock(r->mu);
  r->cv_host.notify_all();
  r->cv_enqueued.notify_all();
}

// Test hook: a deterministic pseudo-random pause of 0..max microseconds.
void hook_pause(kvx_ring* r, uint64_t* state) {
  if (r->hook_max_delay_us <= 0) return;
  *state = *state * 6364136223846793005ULL + 1442695040888963407ULL;
  const int64_t us = (int64_t)((*state >> 33) % (uint64_t)(r->hook_max_delay_us + 1));
  std::this_thread::sleep_for(std::chrono::microseconds(us));
}

// Restore fill thread w: copies its share of every piece into the piece's slot.
void fill_worker(kvx_ring* r, int w) {
  const int32_t S = r->n_slots, T = r->threads;
  const int64_t P = (int64_t)r->plan.pieces.size();
  int64_t busy = 0;
  uint64_t rng = 0x9E3779B97F4A7C15ULL * (uint64_t)(w + 1);
  for (int64_t i = 0; i < P; ++i) {
    hook_pause(r, &rng);
    const int32_t s = (int32_t)(i % S);
    if (i >= S) {
      // The copy of piece i - S must have been issued before we wait for it.
      std::unique_lock<std::mutex> lock(r->mu);
      r->cv_enqueued.wait(lock, [&] { return r->enqueued > i - S || r->stop.load(); });
    }
    if (r->stop.load()) break;
    if (!wait_copy(r, s)) {
      r->worker_error.store(KVX_EHIP);
      signal_stop(r);
      break;
    }
    if (r->hook_poison) {
      // The slot is released: overwrite this thread's share before refilling
      // it, so a copy that still read it would carry the poison.
      const kvx::Piece& p = r->plan.pieces[(size_t)i];
      int64_t per = (p.bytes + T - 1) / T;
      per = (per + 4095) & ~(int64_t)4095;
      const int64_t a = std::min<int64_t>(p.bytes, per * w);
      const int64_t b = std::min<int64_t>(p.bytes, a + per);
      if (b > a) std::memset(r->host + (int64_t)s * r->slot_bytes + a, 0xA5, (size_t)(b - a));
      hook_pause(r, &rng);
    }
    const int64_t t0 = now_ns();
    const int64_t bytes = copy_share(r, r->plan.pieces[(size_t)i], s, w, T, true);
    const int64_t t1 = now_ns();
    busy += t1 - t0;
    std::lock_guard<std::mutex> lock(r->mu);
    if (r->trace_run) r->trace_ev.push_back(kvx_trace_event{KVX_TRACE_FILL, (int32_t)i, w, s, bytes, t0, t1});
    if (++r->parts_done[(size_t)i] == T) r->cv_host.notify_all();
  }
  r->busy_ns.fetch_add(busy);
}

// Offload drain thread w: copies its share of every piece out of its slot.
void drain_worker(kvx_ring* r, int w) {
  const int32_t S = r->n_slots, T = r->threads;
  const int64_t P = (int64_t)r->plan.pieces.size();
  int64_t busy = 0;
  uint64_t rng = 0xD1B54A32D192ED03ULL * (uint64_t)(w + 1);
  for (int64_t i = 0; i < P; ++i) {
    const int32_t s = (int32_t)(i % S);
    hook_pause(r, &rng);
    {
      std::unique_lock<std::mutex> lock(r->mu);
      r->cv_enqueued.wait(lock, [&] { return r->enqueued > i || r->stop.load(); });
    }
    if (r->stop.load()) break;
    if (!wait_copy(r, s)) {
      r->worker_error.store(KVX_EHIP);
      signal_stop(r);
      break;
    }
    const int64_t t0 = now_ns();
    const int64_t bytes = copy_share(r, r->plan.pieces[(size_t)i], s, w, T, false);
    const int64_t t1 = now_ns();
    busy += t1 - t0;
    std::lock_guard<std::mutex> lock(r->mu);
    if (r->trace_run) r->trace_ev.push_back(kvx_trace_event{KVX_TRACE_DRAIN, (int32_t)i, w, s, bytes, t0, t1});
    if (++r->parts_done[(size_t)i] == T) r->cv_host.notify_all();
  }
  r->busy_ns.fetch_add(busy);
}

// A pool thread: runs worker w of every transfer handed to the pool (a new
// pool_gen) until told to quit. `seen` starts at the generation current when
// the thread is created, before the transfer it is created for is handed
// over, so that it cannot miss that transfer.
void pool_worker(kvx_ring* r, Dir dir, int w, uint64_t seen) {
  for (;;) {
    {
      std::unique_lock<std::mutex> lock(r->mu);
      r->cv_pool.wait(lock, [&] { return r->pool_quit || r->pool_gen != seen; });
      if (r->pool_quit) return;
      seen = r->pool_gen;
    }
    if (dir == Dir::kRestore)
      fill_worker(r, w);
    else
      drain_worker(r, w);
    std::lock_guard<std::mutex> lock(r->mu);
    if (++r->pool_done == (int32_t)r->pool.size()) r->cv_pool_done.notify_all();
  }
}

// Join the pool's threads (none may be running a transfer).
void stop_pool(kvx_ring* r) {
  {
    std::lock_guard<std::mutex> lock(r->mu);
    r->pool_quit = true;
  }
  r->cv_pool.notify_all();
  for (auto& th : r->pool) th.join();
  r->pool.clear();
  r->pool_dir = Dir::kNone;
  std::lock_guard<std::mutex> lock(r->mu);
  r->pool_quit = false;
}

// Hand the transfer about to run to T pool threads of direction dir, starting
// them first where the pool has another direction or count. Called by the
// transfer's own thread, the only one that changes pool_gen. Throws if a
// thread cannot be created (the pool is then empty).
void start_pool(kvx_ring* r, Dir dir, int32_t T) {
  if (r->pool_dir != dir || (int32_t)r->pool.size() != T) {
    stop_pool(r);
    r->pool_dir = dir;
    try {
      for (int w = 0; w < T; ++w) r->pool.emplace_back(pool_worker, r, dir, w, r->pool_gen);
    } catch (...) {
      stop_pool(r);
      throw;
    }
  }
  {
    std::lock_guard<std::mutex> lock(r->mu);
    r->pool_done = 0;
    ++r->pool_gen;
  }
  r->cv_pool.notify_all();
}

// Wait until every pool thread is done with the current transfer.
void wait_pool(kvx_ring* r) {
  std::unique_lock<std::mutex> lock(r->mu);
  r->cv_pool_done.wait(lock, [&] { return r->pool_done == (int32_t)r->pool.size(); });
}

// ---- storage tier -----------------------------------------------------------
//
// A bound chunk file f is planned as if its image sat at the notional host
// address (f + 1) << kFileShift (never dereferenced), so the planner's spans
// name (file, byte offset in the file) directly.
constexpr int kFileShift = 40;

int32_t span_file(const kvx::Span& sp) {
  return (int32_t)(((uintptr_t)sp.host >> kFileShift) - 1);
}

int64_t span_offset(const kvx::Span& sp) {
  return (int64_t)((uintptr_t)sp.host & (((uintptr_t)1 << kFileShift) - 1));
}

// Status of a transfer stopped early: the worker's failure, else an abort.
kvx_status worker_status(const kvx_ring* r) {
  const int e = r->worker_error.load();
  return e ? (kvx_status)e : KVX_ECLOSED;
}

void mark_piece_done(kvx_ring* r, int64_t i) {
  std::lock_guard<std::mutex> lock(r->mu);
  r->parts_done[(size_t)i] = r->threads;
  r->cv_host.notify_all();
}

void fail_worker(kvx_ring* r, kvx_status st) {
  r->worker_error.store(st);
  signal_stop(r);
}

// Restore reactor: read each piece's spans from the chunk files into its host
// slot, up to io_depth reads in flight, starting a piece only once its slot's
// previous H2D copy has completed; a piece is handed to the enqueuing thread
// when all of its reads have landed.
void file_fill_worker(kvx_ring* r) {
  const int32_t S = r->n_slots;
  const int64_t P = (int64_t)r->plan.pieces.size();
  const auto t0 = clk::now();
  kvx::IoEngine io;
  if (io.init(r->io_depth, false) != KVX_OK) {
    fail_worker(r, KVX_EINTERNAL);
    return;
  }
  std::vector<int32_t> left((size_t)P, 0);
  std::vector<uint64_t> done;
  int64_t next = 0;  // next piece to start
  size_t span = 0;   // next span of that piece
  int64_t complete = 0;
  kvx_status st = KVX_OK;
  while (st == KVX_OK && complete < P && !r->stop.load()) {
    // Start reads while the depth allows and the next piece's slot is free.
    bool blocked = false;
    while (st == KVX_OK && next < P && io.inflight() < io.depth()) {
      const int32_t s = (int32_t)(next % S);
      const kvx::Piece& p = r->plan.pieces[(size_t)next];
      if (span == 0) {
        if (next >= S) {
          bool enq;
          {
            std::lock_guard<std::mutex> lock(r->mu);
            enq = r->enqueued > next - S;
          }
          if (!enq || !copy_finished(r, s)) {
            blocked = true;
            break;
          }
        }
        left[(size_t)next] = (int32_t)p.spans.size();
      }
      const kvx::Span& sp = p.spans[span];
      kvx::TierFile& f = r->files[(size_t)span_file(sp)];
      st = kvx::open_tier_file(&f, false);
      if (st == KVX_OK)
        st = io.start(&f, r->host + (int64_t)s * r->slot_bytes + sp.slot_off, span_offset(sp),
                      sp.bytes, (uint64_t)next);
      if (++span == p.spans.size()) {
        span = 0;
        ++next;
      }
      if (!io.uring()) break;  // synchronous: report each read as it finishes
    }
    if (st != KVX_OK) break;
    if (io.pending() == 0 && blocked) {
      // Nothing in flight: wait for the slot of piece `next` to be released.
      const int32_t s = (int32_t)(next % S);
      {
        std::unique_lock<std::mutex> lock(r->mu);
        r->cv_enqueued.wait(lock, [&] { return r->enqueued > next - S || r->stop.load(); });
      }
      if (r->stop.load()) break;
      if (!wait_copy(r, s)) st = KVX_EHIP;
      continue;
    }
    done.clear();
    st = io.wait(&done);
    for (uint64_t t : done)
      if (--left[(size_t)t] == 0) {
        mark_piece_done(r, (int64_t)t);
        ++complete;
      }
  }
  while (io.inflight() > 0) {  // reads still landing in the slots
    const int32_t before = io.inflight();
    done.clear();
    if (io.wait(&done) != KVX_OK && io.inflight() == before) break;
  }
  for (auto& f : r->files) kvx::close_tier_file(&f);
  r->busy_ns.fetch_add(std::chrono::duration_cast<std::chrono::nanoseconds>(clk::now() - t0).count());
  if (st != KVX_OK) fail_worker(r, st);
}

// Offload reactor: as each piece's D2H copy completes, write its spans from
// the host slot into the chunk files (up to io_depth writes in flight),
// publishing each file once all of its bytes landed; a piece's slot is
// released when all of its writes have landed.
void file_drain_worker(kvx_ring* r) {
  const int32_t S = r->n_slots;
  const int64_t P = (int64_t)r->plan.pieces.size();
  const auto t0 = clk::now();
  kvx::IoEngine io;
  if (io.init(r->io_depth, true) != KVX_OK) {
    fail_worker(r, KVX_EINTERNAL);
    return;
  }
  std::vector<int32_t> left((size_t)P, 0);
  std::vector<uint64_t> done;
  std::vector<int32_t> to_sync;  // buffered files fully written, to flush before publishing
  kvx_status st = KVX_OK;
  // Finish what has landed: release pieces whose writes are all done, publish
  // direct files at once and queue buffered ones for their flush; then start
  // queued flushes while the depth allows.
  auto reap = [&]() {
    done.clear();
    kvx_status w = io.wait(&done);
    for (uint64_t t : done) {
      if (t & kvx::kSyncTag) {
        if (w == KVX_OK) w = kvx::publish_tier_file(&r->files[(size_t)(t & ~kvx::kSyncTag)]);
        continue;
      }
      const kvx::Piece& p = r->plan.pieces[(size_t)(t >> 20)];
      const kvx::Span& sp = p.spans[(size_t)(t & 0xFFFFF)];
      kvx::TierFile& f = r->files[(size_t)span_file(sp)];
      // (several of a file's transfers can finish in one wait: act once)
      if (w == KVX_OK && f.written == f.size && !f.published && !f.flushing) {
        if (f.direct) {
          w = kvx::publish_tier_file(&f);
        } else {
          f.flushing = true;
          to_sync.push_back(span_file(sp));
        }
      }
      if (--left[(size_t)(t >> 20)] == 0) mark_piece_done(r, (int64_t)(t >> 20));
    }
    while (w == KVX_OK && !to_sync.empty() && io.inflight() < io.depth()) {
      const int32_t fi = to_sync.back();
      to_sync.pop_back();
      w = io.start_datasync(&r->files[(size_t)fi], kvx::kSyncTag | (uint64_t)fi);
    }
    return w;
  };
  for (int64_t i = 0; st == KVX_OK && i < P && !r->stop.load(); ++i) {
    const int32_t s = (int32_t)(i % S);
    const kvx::Piece& p = r->plan.pieces[(size_t)i];
    // Wait for piece i's D2H copy to be enqueued. The enqueuing thread may be
    // waiting for an earlier piece's slot, which only reaping its writes
    // releases: sleep only with nothing in flight, else reap meanwhile.
    for (;;) {
      {
        std::lock_guard<std::mutex> lock(r->mu);
        if (r->enqueued > i || r->stop.load()) break;
      }
      if (io.pending() > 0) {
        st = reap();
        if (st != KVX_OK) break;
        continue;
      }
      std::unique_lock<std::mutex> lock(r->mu);
      r->cv_enqueued.wait(lock, [&] { return r->enqueued > i || r->stop.load(); });
      break;
    }
    if (st != KVX_OK || r->stop.load()) break;
    if (!wait_copy(r, s)) {
      st = KVX_EHIP;
      break;
    }
    left[(size_t)i] = (int32_t)p.spans.size();
    for (size_t k = 0; st == KVX_OK && k < p.spans.size(); ++k) {
      while (st == KVX_OK && io.inflight() >= io.depth()) st = reap();
      if (st != KVX_OK) break;
      const kvx::Span& sp = p.spans[k];
      kvx::TierFile& f = r->files[(size_t)span_file(sp)];
      st = kvx::open_tier_file(&f, true);
      if (st == KVX_OK)
        st = io.start(&f, r->host + (int64_t)s * r->slot_bytes + sp.slot_off, span_offset(sp),
                      sp.bytes, ((uint64_t)i << 20) | (uint64_t)k);
    }
  }
  while (st == KVX_OK && (io.pending() > 0 || !to_sync.empty())) st = reap();
  while (io.inflight() > 0) {  // after an error: let what is in flight land
    const int32_t before = io.inflight();
    done.clear();
    if (io.wait(&done) != KVX_OK && io.inflight() == before) break;
  }
  for (auto& f : r->files) kvx::close_tier_file(&f);  // unpublished temporaries are removed
  r->busy_ns.fetch_add(std::chrono::duration_cast<std::chrono::nanoseconds>(clk::now() - t0).count());
  if (st != KVX_OK) fail_worker(r, st);
}

kvx_status launch_piece(kvx_ring* r, bool to_packed, const kvx::Piece& p, const int32_t* bt,
                        uint8_t* dslot, hipStream_t stream) {
  return kvx::launch_copy_chunks(to_packed, &r->cache, p.l_begin, p.l_end, bt, r->plan.table_len,
                                 r->d_refs + p.ref_first, p.ref_count, r->chunk_tokens, dslot,
                                 r->slot_bytes, stream, r->err_word);
}

// ---- timeline (kvx_ring_set_trace) ----------------------------------------------

bool grow_events(std::vector<hipEvent_t>* v, size_t n) {
  while (v->size() < n) {
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return false;  // timing events
    v->push_back(e);
  }
  return true;
}

// Start the record of a traced transfer of P pieces whose launches go to
// `stream`: a reference event on it (waited for, so its time on the host
// clock is known) and the HSA system clock against the host clock.
kvx_status trace_begin(kvx_ring* r, hipStream_t stream, int64_t P, bool to_packed) {
  {
    std::lock_guard<std::mutex> lock(r->mu);
    r->trace_ev.clear();
  }
  r->traced = false;
  r->trace_resolved = false;
  r->trace_pieces = P;
  r->trace_to_packed = to_packed;
  if (!grow_events(&r->trace_k, 2 * (size_t)P) || !grow_events(&r->trace_c, 2 * (size_t)P))
    return KVX_EHIP;
  if (!r->trace_ref && hipEventCreate(&r->trace_ref) != hipSuccess) return KVX_EHIP;
  r->trace_k_used.assign((size_t)P, 0);
  r->trace_c_used.assign((size_t)P, 0);
  r->trace_k_bytes.assign((size_t)P, 0);
  r->trace_c_bytes.assign((size_t)P, 0);
  r->trace_dma_piece.assign((size_t)r->n_slots, -1);
  r->trace_dma_bytes.assign((size_t)r->n_slots, 0);
  if (hipEventRecord(r->trace_ref, stream) != hipSuccess ||
      hipEventSynchronize(r->trace_ref) != hipSuccess)
    return KVX_EHIP;
  r->trace_ref_ns = now_ns();
  r->trace_hsa_hz = 0;
  uint64_t hz = 0, t = 0;
  if (r->hsa_up &&
      hsa_system_get_info(HSA_SYSTEM_INFO_TIMESTAMP_FREQUENCY, &hz) == HSA_STATUS_SUCCESS && hz) {
    const int64_t a = now_ns();
    if (hsa_system_get_info(HSA_SYSTEM_INFO_TIMESTAMP, &t) == HSA_STATUS_SUCCESS) {
      const int64_t b = now_ns();
      r->trace_host0 = a + (b - a) / 2;
      r->trace_hsa0 = t;
      r->trace_hsa_hz = hz;
    }
  }
  return KVX_OK;
}

void trace_push(kvx_ring* r, const kvx_trace_event& e) {
  std::lock_guard<std::mutex> lock(r->mu);
  r->trace_ev.push_back(e);
}

// Record the DMA copy interval of the piece last copied through slot s (its
// copies have finished); nothing if it had several copies or no timestamps.
void trace_dma_read(kvx_ring* r, int32_t s, bool h2d) {
  const int64_t i = r->trace_dma_piece[(size_t)s];
  if (i < 0) return;
  r->trace_dma_piece[(size_t)s] = -1;
  hsa_amd_profiling_async_copy_time_t t{};
  if (!r->trace_hsa_hz ||
      hsa_amd_profiling_get_async_copy_time(r->dma_done[(size_t)s], &t) != HSA_STATUS_SUCCESS ||
      t.end < t.start)
    return;
  auto host = [&](uint64_t v) {
    const long double d = ((long double)v - (long double)r->trace_hsa0) * 1e9L /
                          (long double)r->trace_hsa_hz;
    return r->trace_host0 + (int64_t)d;
  };
  trace_push(r, kvx_trace_event{h2d ? KVX_TRACE_H2D : KVX_TRACE_D2H, (int32_t)i, 0, s,
                                r->trace_dma_bytes[(size_t)s], host(t.start), host(t.end)});
}

// launch_piece for piece i, between two timing events when tracing.
kvx_status launch_piece_traced(kvx_ring* r, bool to_packed, int64_t i, const kvx::Piece& p,
                               const int32_t* bt, uint8_t* dslot, hipStream_t stream) {
  const bool t = r->trace_run;
  if (t && hipEventRecord(r->trace_k[2 * (size_t)i], stream) != hipSuccess) return KVX_EHIP;
  const kvx_status st = launch_piece(r, to_packed, p, bt, dslot, stream);
  if (st != KVX_OK) return st;
  if (t) {
    if (hipEventRecord(r->trace_k[2 * (size_t)i + 1], stream) != hipSuccess) return KVX_EHIP;
    r->trace_k_used[(size_t)i] = 1;
    r->trace_k_bytes[(size_t)i] = p.bytes;
  }
  return KVX_OK;
}

// The device intervals of the last traced transfer (launches, runtime copies)
// onto the host clock, once; then every interval ordered by start.
kvx_status trace_resolve(kvx_ring* r) {
  if (r->trace_resolved) return KVX_OK;
  std::vector<kvx_trace_event> dev;
  const int32_t S = r->n_slots;
  auto at = [&](hipEvent_t e, int64_t* ns) {
    float ms = 0;
    if (hipEventSynchronize(e) != hipSuccess ||
        hipEventElapsedTime(&ms, r->trace_ref, e) != hipSuccess)
      return false;
    *ns = r->trace_ref_ns + (int64_t)((double)ms * 1e6);
    return true;
  };
  for (int64_t i = 0; i < r->trace_pieces; ++i) {
    int64_t a = 0, b = 0;
    if (r->trace_k_used[(size_t)i]) {
      if (!at(r->trace_k[2 * (size_t)i], &a) || !at(r->trace_k[2 * (size_t)i + 1], &b))
        return KVX_EHIP;
      dev.push_back(kvx_trace_event{r->trace_to_packed ? KVX_TRACE_GATHER : KVX_TRACE_SCATTER,
                                    (int32_t)i, 0, (int32_t)(i % S), r->trace_k_bytes[(size_t)i], a,
                                    b});
    }
    if (r->trace_c_used[(size_t)i]) {
      if (!at(r->trace_c[2 * (size_t)i], &a) || !at(r->trace_c[2 * (size_t)i + 1], &b))
        return KVX_EHIP;
      dev.push_back(kvx_trace_event{r->trace_to_packed ? KVX_TRACE_D2H : KVX_TRACE_H2D,
                                    (int32_t)i, 0, (int32_t)(i % S), r->trace_c_bytes[(size_t)i],
                                    a, b});
    }
  }
  std::lock_guard<std::mutex> lock(r->mu);
  r->trace_ev.insert(r->trace_ev.end(), dev.begin(), dev.end());
  std::stable_sort(r->trace_ev.begin(), r->trace_ev.end(),
                   [](const kvx_trace_event& x, const kvx_trace_event& y) { return x.t0_ns < y.t0_ns; });
  r->trace_resolved = true;
  return KVX_OK;
}

// One async copy on a DMA engine (engine 0: the runtime's choice); the copy
// decrements sig when it has finished.
hsa_status_t engine_copy(void* dst, hsa_agent_t dst_agent, const void* src, hsa_agent_t src_agent,
                         size_t bytes, uint32_t engine, hsa_signal_t sig) {
  if (engine)
    return hsa_amd_memory_async_copy_on_engine(dst, dst_agent, src, src_agent, bytes, 0, nullptr,
                                               sig, (hsa_amd_sdma_engine_id_t)engine, true);
  return hsa_amd_memory_async_copy(dst, dst_agent, src, src_agent, bytes, 0, nullptr, sig);
}

// The host-link copies of piece p on slot s: H2D (restore) host slot s to
// device slot s, or D2H (offload) device slot s to host slot s; without fill
// or drain threads, one copy per span between its host address and its place
// in the device slot. dma_done[s] counts the piece's copies down to 0.
kvx_status issue_dma(kvx_ring* r, int64_t piece, const kvx::Piece& p, int32_t s, uint8_t* dslot,
                     uint8_t* hslot, bool h2d) {
  hsa_signal_t sig = r->dma_done[(size_t)s];
  const bool whole = r->threads > 0;
  const int64_t n = whole ? 1 : (int64_t)p.spans.size();
  if (n == 0) return KVX_OK;
  // the slot's previous copies have finished (every caller waited for them):
  // read their interval before the signal is reused
  if (r->trace_run) trace_dma_read(r, s, h2d);
  hsa_signal_store_screlease(sig, n);
  int64_t issued = 0;
  for (int64_t k = 0; k < n; ++k) {
    uint8_t* host = whole ? hslot : p.spans[(size_t)k].host;
    uint8_t* dev = whole ? dslot : dslot + p.spans[(size_t)k].slot_off;
    const size_t bytes = (size_t)(whole ? p.bytes : p.spans[(size_t)k].bytes);
    const hsa_status_t hs =
        h2d ? engine_copy(dev, r->gpu_agent, host, r->cpu_agent, bytes, r->h2d_engine, sig)
            : engine_copy(host, r->cpu_agent, dev, r->gpu_agent, bytes, r->d2h_engine, sig);
    if (hs != HSA_STATUS_SUCCESS) break;
    ++issued;
  }
  if (issued < n) {  // the copies never issued will never count down: do it here
    hsa_signal_subtract_screlease(sig, n - issued);
    return KVX_EHIP;
  }
  if (r->trace_run) {
    r->trace_dma_piece[(size_t)s] = n == 1 ? piece : -1;
    r->trace_dma_bytes[(size_t)s] = p.bytes;
  }
  return KVX_OK;
}

// Restore on the DMA engines: scatter piece j once the host has seen its copy
// complete (the launch then reads the copied bytes of device slot j mod S).
kvx_status scatter_copied(kvx_ring* r, int64_t j, const int32_t* bt, hipStream_t stream) {
  const int32_t s = (int32_t)(j % r->n_slots);
  if (!wait_dma(r, s)) return KVX_EHIP;
  kvx_status st = launch_piece_traced(r, false, j, r->plan.pieces[(size_t)j], bt,
                                      r->landing + (int64_t)s * r->slot_bytes, stream);
  if (st != KVX_OK) return st;
  return hipEventRecord(r->dev_done[(size_t)s], stream) == hipSuccess ? KVX_OK : KVX_EHIP;
}

// Restore out of a preloader's pool: piece p with the notional addresses of
// its spans replaced by the images of the held files (imgs caches those already
// staged). Without `wait`, *ready is false if a file is not staged yet;
// with it, blocks until every file is (KVX_ECLOSED on an abort meanwhile).
kvx_status resolve_piece(kvx_ring* r, const kvx::Piece& p, const std::vector<void*>& holds,
                         std::vector<uint8_t*>* imgs, bool wait, kvx::Piece* out, bool* ready) {
  *ready = false;
  *out = p;
  for (kvx::Span& sp : out->spans) {
    const int32_t u = r->pre_file[(size_t)span_file(sp)];
    uint8_t*& img = (*imgs)[(size_t)u];
    if (!img) {
      int64_t size = 0;
      const kvx_status st = kvx::preload_image(r->pre, holds[(size_t)u], wait, &r->closed, &img, &size);
      if (st != KVX_OK) return st;
      if (!img) return KVX_OK;
      if (size != r->pre_bytes[(size_t)u]) {  // not this chunk's image: never use it again
        kvx::preload_discard(r->pre, holds[(size_t)u]);
        img = nullptr;
        return KVX_EIO;
      }
    }
    sp.host = img + span_offset(sp);
  }
  *ready = true;
  return KVX_OK;
}

// Run the bound transfer, its kernels on `stream` reporting bad ids to err.
kvx_status run(kvx_ring* r, Dir dir, const int32_t* bt, hipStream_t stream, int* err) {
  r->traced = false;
  if (r->dir != dir) return KVX_EINVAL;
  if (r->closed.load()) return KVX_ECLOSED;
  if (r->plan.pieces.empty()) return KVX_OK;
  if (!bt) return KVX_EINVAL;
  DeviceGuard dg(r->device);
  if (!dg.ok) return KVX_EHIP;
  if (!err) return KVX_EHIP;
  r->err_word = err;
  const auto t_start = clk::now();
  const int32_t S = r->n_slots, T = r->threads;
  const int64_t P = (int64_t)r->plan.pieces.size();
  {
    std::lock_guard<std::mutex> lock(r->mu);
    r->enqueued = 0;
    r->parts_done.assign((size_t)P, 0);
  }
  r->worker_error.store(0);
  r->stop.store(false);
  r->busy_ns.store(0);
  r->trace_run = r->trace;
  if (r->trace_run) {
    const kvx_status ts = trace_begin(r, stream, P, dir == Dir::kOffload);
    if (ts != KVX_OK) return ts;
  }
  std::vector<std::thread> workers;
  kvx_status st = KVX_OK;
  double wait_ms = 0;
  // restore out of a preloader's pool: hold every file now (those not staged
  // are read as demand work, in chunk order) and copy each piece once its
  // files are staged
  std::vector<void*> holds;
  std::vector<uint8_t*> imgs;
  kvx::Piece resolved;
  if (r->pre) {
    st = kvx::preload_hold(r->pre, r->pre_paths, &holds);
    if (st != KVX_OK) return st;
    imgs.assign(r->pre_paths.size(), nullptr);
  }
  bool pooled = false;  // the pool's threads run this transfer
  // Whatever way this function is left, the pool is done with the transfer
  // first (on an exception: told to stop, then waited for).
  struct PoolGuard {
    kvx_ring* r;
    bool* pooled;
    ~PoolGuard() {
      if (*pooled) {
        signal_stop(r);
        wait_pool(r);
      }
    }
  } pool_guard{r, &pooled};
  try {
    if (r->files_mode) {
      workers.emplace_back(dir == Dir::kRestore ? file_fill_worker : file_drain_worker, r);
    } else if (T > 0) {
      start_pool(r, dir, T);
      pooled = true;
    }
  } catch (...) {
    st = KVX_ENOMEM;
  }
  auto wait_parts = [&](int64_t i) {
    const int64_t t0 = now_ns();
    std::unique_lock<std::mutex> lock(r->mu);
    r->cv_host.wait(lock, [&] { return r->parts_done[(size_t)i] == T || r->stop.load(); });
    const int64_t t1 = now_ns();
    wait_ms += (double)(t1 - t0) / 1e6;
    if (r->trace_run)
      r->trace_ev.push_back(kvx_trace_event{KVX_TRACE_WAIT, (int32_t)i, 0, (int32_t)(i % S), 0, t0, t1});
  };
  int64_t copied = -1;  // restore on the DMA engines: the piece copied but not yet scattered
  for (int64_t i = 0; st == KVX_OK && i < P; ++i) {
    const int32_t s = (int32_t)(i % S);
    const kvx::Piece& p = r->plan.pieces[(size_t)i];
    uint8_t* dslot = r->landing + (int64_t)s * r->slot_bytes;
    uint8_t* hslot = r->host + (int64_t)s * r->slot_bytes;
    const kvx::Piece* pp = &p;  // p, or p resolved to the held images
    if (dir == Dir::kRestore && r->pre) {
      bool ready = false;
      st = resolve_piece(r, p, holds, &imgs, false, &resolved, &ready);
      if (st == KVX_OK && !ready) {
        // a file of this piece is still being read: scatter the copied piece
        // meanwhile, then wait
        if (copied >= 0) {
          st = scatter_copied(r, copied, bt, stream);
          copied = -1;
        }
        const auto t0 = clk::now();
        if (st == KVX_OK) st = resolve_piece(r, p, holds, &imgs, true, &resolved, &ready);
        wait_ms += ms_since(t0);
      }
      if (st != KVX_OK) break;
      pp = &resolved;
    }
    if (dir == Dir::kRestore && use_dma(r)) {
      if (T > 0) wait_parts(i);
      if (r->stop.load() || r->closed.load()) {
        st = worker_status(r);
        break;
      }
      // With one slot, the pending piece must be scattered out of it first.
      if (copied >= 0 && copied % S == s) {
        st = scatter_copied(r, copied, bt, stream);
        copied = -1;
        if (st != KVX_OK) break;
      }
      // Device slot s is free once the scatter that last read it (piece
      // i - S, or the previous transfer's) has finished.
      if (hipEventSynchronize(r->dev_done[s]) != hipSuccess) {
        st = KVX_EHIP;
        break;
      }
      st = issue_dma(r, i, *pp, s, dslot, hslot, true);
      if (st != KVX_OK) break;
      {
        std::lock_guard<std::mutex> lock(r->mu);
        r->enqueued = i + 1;
      }
      r->cv_enqueued.notify_all();
      // The copy of piece i is queued behind that of the pending piece: wait
      // for the pending one and scatter it meanwhile.
      if (copied >= 0) st = scatter_copied(r, copied, bt, stream);
      copied = i;
    } else if (dir == Dir::kRestore) {
      if (T > 0) wait_parts(i);
      if (r->stop.load() || r->closed.load()) {
        st = worker_status(r);
        break;
      }
      bool ok = hipStreamWaitEvent(r->side, r->dev_done[s], 0) == hipSuccess;
      if (r->trace_run) ok = ok && hipEventRecord(r->trace_c[2 * (size_t)i], r->side) == hipSuccess;
      if (T > 0) {
        ok = ok && hipMemcpyAsync(dslot, hslot, (size_t)p.bytes, hipMemcpyHostToDevice, r->side) ==
                       hipSuccess;
      } else {
        for (const kvx::Span& sp : pp->spans)
          ok = ok && hipMemcpyAsync(dslot + sp.slot_off, sp.host, (size_t)sp.bytes,
                                    hipMemcpyHostToDevice, r->side) == hipSuccess;
      }
      if (r->trace_run && ok) {
        ok = hipEventRecord(r->trace_c[2 * (size_t)i + 1], r->side) == hipSuccess;
        r->trace_c_used[(size_t)i] = ok ? 1 : 0;
        r->trace_c_bytes[(size_t)i] = p.bytes;
      }
      ok = ok && hipEventRecord(r->copy_done[s], r->side) == hipSuccess;
      if (!ok) {
        st = KVX_EHIP;
        break;
      }
      {
        std::lock_guard<std::mutex> lock(r->mu);
        r->enqueued = i + 1;
      }
      r->cv_enqueued.notify_all();
      if (hipStreamWaitEvent(stream, r->copy_done[s], 0) != hipSuccess) {
        st = KVX_EHIP;
        break;
      }
      st = launch_piece_traced(r, false, i, p, bt, dslot, stream);
      if (st != KVX_OK) break;
      if (hipEventRecord(r->dev_done[s], stream) != hipSuccess) st = KVX_EHIP;
    } else if (use_dma(r)) {
      if (r->closed.load()) {
        st = KVX_ECLOSED;
        break;
      }
      // Device slot s is free once the copy of piece i - S has finished.
      if (i >= S && !wait_dma(r, s)) {
        st = KVX_EHIP;
        break;
      }
      st = launch_piece_traced(r, true, i, p, bt, dslot, stream);
      if (st != KVX_OK) break;
      if (hipEventRecord(r->dev_done[s], stream) != hipSuccess) {
        st = KVX_EHIP;
        break;
      }
      // Host slot s is free once the drains of piece i - S are done; the
      // gather runs meanwhile.
      if (T > 0 && i >= S) wait_parts(i - S);
      if (r->stop.load()) {
        st = worker_status(r);
        break;
      }
      if (hipEventSynchronize(r->dev_done[s]) != hipSuccess) {
        st = KVX_EHIP;
        break;
      }
      st = issue_dma(r, i, p, s, dslot, hslot, false);
      if (st != KVX_OK) break;
      {
        std::lock_guard<std::mutex> lock(r->mu);
        r->enqueued = i + 1;
      }
      r->cv_enqueued.notify_all();
    } else {  // offload through the HIP runtime
      if (r->closed.load()) {
        st = KVX_ECLOSED;
        break;
      }
      if (hipStreamWaitEvent(stream, r->copy_done[s], 0) != hipSuccess) {
        st = KVX_EHIP;
        break;
      }
      st = launch_piece_traced(r, true, i, p, bt, dslot, stream);
      if (st != KVX_OK) break;
      if (hipEventRecord(r->dev_done[s], stream) != hipSuccess) {
        st = KVX_EHIP;
        break;
      }
      if (T > 0 && i >= S) wait_parts(i - S);  // host slot s emptied by the drains
      if (r->stop.load()) {
        st = worker_status(r);
        break;
      }
      bool ok = hipStreamWaitEvent(r->side, r->dev_done[s], 0) == hipSuccess;
      if (r->trace_run) ok = ok && hipEventRecord(r->trace_c[2 * (size_t)i], r->side) == hipSuccess;
      if (T > 0) {
        ok = ok && hipMemcpyAsync(hslot, dslot, (size_t)p.bytes, hipMemcpyDeviceToHost, r->side) ==
                       hipSuccess;
      } else {
        for (const kvx::Span& sp : p.spans)
          ok = ok && hipMemcpyAsync(sp.host, dslot + sp.slot_off, (size_t)sp.bytes,
                                    hipMemcpyDeviceToHost, r->side) == hipSuccess;
      }
      if (r->trace_run && ok) {
        ok = hipEventRecord(r->trace_c[2 * (size_t)i + 1], r->side) == hipSuccess;
        r->trace_c_used[(size_t)i] = ok ? 1 : 0;
        r->trace_c_bytes[(size_t)i] = p.bytes;
      }
      ok = ok && hipEventRecord(r->copy_done[s], r->side) == hipSuccess;
      if (!ok) {
        st = KVX_EHIP;
        break;
      }
      {
        std::lock_guard<std::mutex> lock(r->mu);
        r->enqueued = i + 1;
      }
      r->cv_enqueued.notify_all();
    }
  }
  if (st == KVX_OK && copied >= 0) st = scatter_copied(r, copied, bt, stream);
  if (st == KVX_OK && dir == Dir::kOffload) {
    // The destinations are complete once the last drains (or, without drain
    // threads, the last device-to-host copies) have finished.
    if (T > 0) {
      for (int64_t i = std::max<int64_t>(0, P - S); i < P && !r->stop.load(); ++i) wait_parts(i);
      if (r->stop.load()) st = worker_status(r);
    } else if (use_dma(r)) {
      for (int32_t s = 0; s < S; ++s)
        if (!wait_dma(r, s)) st = KVX_EHIP;
    } else if (hipStreamSynchronize(r->side) != hipSuccess) {
      st = KVX_EHIP;
    }
  }
  if (st == KVX_OK && r->trace_run && use_dma(r)) {
    // the last pieces' copies (finished: waited for above)
    for (int32_t s = 0; s < S; ++s)
      if (r->trace_dma_piece[(size_t)s] >= 0) {
        if (!wait_dma(r, s)) {
          st = KVX_EHIP;
          break;
        }
        trace_dma_read(r, s, dir == Dir::kRestore);
      }
  }
  if (st != KVX_OK) {
    signal_stop(r);
    if (dir == Dir::kOffload || use_dma(r)) {
      // Nothing may still write a destination or a device slot once the call
      // has returned (a restore's HIP copies are ordered by events instead).
      if (use_dma(r)) {
        for (int32_t s = 0; s < S; ++s) (void)wait_dma(r, s);
      } else {
        (void)hipStreamSynchronize(r->side);
      }
    }
  }
  for (auto& th : workers) th.join();
  if (pooled) {
    wait_pool(r);
    pooled = false;
  }
  if (!holds.empty()) {
    // the images may be evicted once released: the copies out of them first
    if (!use_dma(r) && hipStreamSynchronize(r->side) != hipSuccess && st == KVX_OK) st = KVX_EHIP;
    kvx::preload_unhold(r->pre, holds);
  }
  r->stop.store(false);
  r->stats.pieces = st == KVX_OK ? P : 0;
  r->stats.bytes = 0;
  if (st == KVX_OK)
    for (const auto& p : r->plan.pieces) r->stats.bytes += p.bytes;
  r->stats.fill_ms = (double)r->busy_ns.load() / 1e6;
  r->stats.wait_fill_ms = wait_ms;
  r->stats.enqueue_ms = ms_since(t_start);
  r->stats.dma = use_dma(r) ? 1 : 0;
  r->stats.dma_engine =
      use_dma(r) ? (int32_t)(dir == Dir::kRestore ? r->h2d_engine : r->d2h_engine) : 0;
  r->traced = r->trace_run && st == KVX_OK;
  return st;
}

struct AgentSearch {
  uint32_t domain = 0, bus = 0, dev = 0;
  hsa_agent_t gpu{}, cpu{};
  bool gpu_found = false, cpu_found = false;
};

hsa_status_t find_agent(hsa_agent_t a, void* data) {
  AgentSearch* q = static_cast<AgentSearch*>(data);
  hsa_device_type_t type;
  if (hsa_agent_get_info(a, HSA_AGENT_INFO_DEVICE, &type) != HSA_STATUS_SUCCESS)
    return HSA_STATUS_SUCCESS;
  if (type == HSA_DEVICE_TYPE_CPU && !q->cpu_found) {
    q->cpu = a;
    q->cpu_found = true;
  } else if (type == HSA_DEVICE_TYPE_GPU && !q->gpu_found) {
    uint32_t bdf = 0, domain = 0;  // bdf = bus << 8 | device << 3 | function
    if (hsa_agent_get_info(a, (hsa_agent_info_t)HSA_AMD_AGENT_INFO_BDFID, &bdf) ==
            HSA_STATUS_SUCCESS &&
        hsa_agent_get_info(a, (hsa_agent_info_t)HSA_AMD_AGENT_INFO_DOMAIN, &domain) ==
            HSA_STATUS_SUCCESS &&
        domain == q->domain && (bdf >> 8) == q->bus && ((bdf >> 3) & 31) == q->dev) {
      q->gpu = a;
      q->gpu_found = true;
    }
  }
  return HSA_STATUS_SUCCESS;
}

// Copies between the device and pinned host memory on chosen engines, timed
// from the host. Each direction has its own half of both buffers, so the two
// directions can run at once.
struct EngineProbe {
  static constexpr size_t kHalf = 16 << 20;
  hsa_agent_t gpu{}, cpu{};
  uint8_t* dev = nullptr;   // 2 * kHalf device bytes
  uint8_t* host = nullptr;  // 2 * kHalf pinned bytes
  hsa_signal_t sig[2]{};    // D2H, H2D
  bool ready = false;

  bool init(const kvx_ring* r) {
    gpu = r->gpu_agent;
    cpu = r->cpu_agent;
    void* d = nullptr;
    void* h = nullptr;
    if (hipMalloc(&d, 2 * kHalf) != hipSuccess) return false;
    dev = (uint8_t*)d;
    if (hipHostMalloc(&h, 2 * kHalf, hipHostMallocDefault) != hipSuccess) return false;
    host = (uint8_t*)h;
    if (hsa_signal_create(0, 0, nullptr, &sig[0]) != HSA_STATUS_SUCCESS) return false;
    if (hsa_signal_create(0, 0, nullptr, &sig[1]) != HSA_STATUS_SUCCESS) {
      (void)hsa_signal_destroy(sig[0]);
      sig[0].handle = 0;
      return false;
    }
    ready = true;
    return true;
  }

  ~EngineProbe() {
    for (hsa_signal_t s : sig)
      if (s.handle) (void)hsa_signal_destroy(s);
    if (host) (void)hipHostFree(host);
    if (dev) (void)hipFree(dev);
  }

  // Issue `reps` copies of `bytes` in each direction (engine id bits, 0: the
  // runtime's choice), both directions interleaved so they start together;
  // wait for all and return the combined rate in bytes per second, 0 if a
  // copy failed.
  double run(uint32_t d2h, int d2h_reps, uint32_t h2d, int h2d_reps, size_t bytes) {
    const int reps[2] = {d2h_reps, h2d_reps};
    int issued[2] = {0, 0};
    hsa_signal_store_screlease(sig[0], reps[0]);
    hsa_signal_store_screlease(sig[1], reps[1]);
    const auto t0 = clk::now();
    for (int k = 0; k < std::max(reps[0], reps[1]); ++k) {
      if (k < reps[0] && issued[0] == k &&
          engine_copy(host, cpu, dev, gpu, bytes, d2h, sig[0]) == HSA_STATUS_SUCCESS)
        ++issued[0];
      if (k < reps[1] && issued[1] == k &&
          engine_copy(dev + kHalf, gpu, host + kHalf, cpu, bytes, h2d, sig[1]) ==
              HSA_STATUS_SUCCESS)
        ++issued[1];
    }
    bool ok = true;
    for (int d = 0; d < 2; ++d) {
      if (issued[d] < reps[d]) {
        hsa_signal_subtract_screlease(sig[d], reps[d] - issued[d]);
        ok = false;
      }
      ok = hsa_signal_wait_scacquire(sig[d], HSA_SIGNAL_CONDITION_LT, 1, UINT64_MAX,
                                     HSA_WAIT_STATE_ACTIVE) == 0 &&
           ok;
    }
    const double sec = std::chrono::duration<double>(clk::now() - t0).count();
    return ok ? (double)bytes * (reps[0] + reps[1]) / std::max(1e-9, sec) : 0;
  }
};

// The runtime's preferred engines for copies from src to dst, else every
// available one (id bits; 0: none named).
uint32_t engine_candidates(hsa_agent_t dst, hsa_agent_t src) {
  uint32_t c = 0;
  if (hsa_amd_memory_get_preferred_copy_engine(dst, src, &c) != HSA_STATUS_SUCCESS) c = 0;
  if (c == 0 && hsa_amd_memory_copy_engine_status(dst, src, &c) != HSA_STATUS_SUCCESS) c = 0;
  return c;
}

// The candidates whose rate alone, in one direction, is within 15 % of the
// best candidate's.
uint32_t fast_engines(EngineProbe* pr, uint32_t cand, bool h2d) {
  if ((cand & (cand - 1)) == 0) return cand;  // none or one
  double rate[32] = {};
  double best = 0;
  for (int b = 0; b < 32; ++b)
    if (cand >> b & 1) {
      const uint32_t e = 1u << b;
      rate[b] = h2d ? pr->run(0, 0, e, 2, EngineProbe::kHalf) : pr->run(e, 2, 0, 0, EngineProbe::kHalf);
      best = std::max(best, rate[b]);
    }
  uint32_t fast = 0;
  for (int b = 0; b < 32; ++b)
    if ((cand >> b & 1) && rate[b] > 0 && rate[b] >= 0.85 * best) fast |= 1u << b;
  return fast;
}

struct Engines {
  uint32_t d2h = 0, h2d = 0;
};

// Choose the D2H and H2D engines of a device. Engines differ several-fold in
// host-link bandwidth (only some sit close to the link), an engine left to
// the runtime may be any of them, and one of the fast ids can be slow in a
// given process; an H2D and a D2H engine running at once reach the link's
// full duplex rate only on some pairs (others share a path and split it).
// So: every candidate gets an untimed small copy first (an engine's first
// copy in a process pays a one-time setup many times a large copy), then each
// direction keeps the candidates that are fast alone (2 x 16 MiB each), and of
// those the (D2H, H2D) pair with the highest combined rate running at once
// (4 x 16 MiB each way) is chosen. Copies of 16 MiB separate the pairs by ~5 %
// with a spread under 0.5 % between repeats; at 4 MiB the margin shrinks to
// ~2 % against a ~1 % spread. A direction with no candidate stays with the
// runtime's choice.
Engines pick_engines(const kvx_ring* r) {
  Engines e;
  const uint32_t cd = engine_candidates(r->cpu_agent, r->gpu_agent);
  const uint32_t ch = engine_candidates(r->gpu_agent, r->cpu_agent);
  EngineProbe pr;
  if (!pr.init(r)) {  // untimed: a lone candidate, else the runtime's choice
    e.d2h = (cd & (cd - 1)) == 0 ? cd : 0;
    e.h2d = (ch & (ch - 1)) == 0 ? ch : 0;
    return e;
  }
  for (int b = 0; b < 32; ++b) {
    if (cd >> b & 1) (void)pr.run(1u << b, 1, 0, 0, 64 << 10);
    if (ch >> b & 1) (void)pr.run(0, 0, 1u << b, 1, 64 << 10);
  }
  const uint32_t fd = fast_engines(&pr, cd, false);
  const uint32_t fh = fast_engines(&pr, ch, true);
  e.d2h = fd & (~fd + 1);  // lowest fast id until a pair is timed
  e.h2d = fh & (~fh + 1);
  if ((fd & (fd - 1)) == 0 && (fh & (fh - 1)) == 0) return e;
  double best = 0;
  for (int bd = 0; bd < 32; ++bd) {
    const uint32_t d = 1u << bd;
    if (fd ? !(fd & d) : bd > 0) continue;  // no fast D2H engine: the runtime's (0) only
    for (int bh = 0; bh < 32; ++bh) {
      const uint32_t h = 1u << bh;
      if (fh ? !(fh & h) : bh > 0) continue;
      const double rate =
          pr.run(fd ? d : 0, 4, fh ? h : 0, 4, EngineProbe::kHalf);
      if (rate > best) {
        best = rate;
        e.d2h = fd ? d : 0;
        e.h2d = fh ? h : 0;
      }
    }
  }
  return e;
}

// Find the HSA agents of the ring's GPU (by PCI location) and of the host,
// and make one completion signal per slot. On any failure the ring keeps the
// HIP copy path.
void setup_dma(kvx_ring* r) {
  int bus = -1, dev = -1, domain = -1;
  if (hipDeviceGetAttribute(&bus, hipDeviceAttributePciBusId, r->device) != hipSuccess ||
      hipDeviceGetAttribute(&dev, hipDeviceAttributePciDeviceId, r->device) != hipSuccess ||
      hipDeviceGetAttribute(&domain, hipDeviceAttributePciDomainId, r->device) != hipSuccess)
    return;
  if (hsa_init() != HSA_STATUS_SUCCESS) return;
  r->hsa_up = true;
  AgentSearch q;
  q.domain = (uint32_t)domain;
  q.bus = (uint32_t)bus;
  q.dev = (uint32_t)dev;
  if (hsa_iterate_agents(find_agent, &q) != HSA_STATUS_SUCCESS || !q.gpu_found || !q.cpu_found)
    return;
  r->gpu_agent = q.gpu;
  r->cpu_agent = q.cpu;
  for (int32_t s = 0; s < r->n_slots; ++s) {
    hsa_signal_t sig{};
    if (hsa_signal_create(0, 0, nullptr, &sig) != HSA_STATUS_SUCCESS) return;
    r->dma_done.push_back(sig);
  }
  r->dma = true;
  // The choice is a property of the device: timed by the first ring created on
  // it in this process, reused by the others.
  static std::mutex mu;
  static std::vector<std::pair<int, Engines>> picked;
  std::lock_guard<std::mutex> lock(mu);
  Engines e;
  bool found = false;
  for (const auto& d : picked)
    if (d.first == r->device) {
      e = d.second;
      found = true;
    }
  if (!found) {
    e = pick_engines(r);
    picked.emplace_back(r->device, e);
  }
  r->d2h_engine = e.d2h;
  r->h2d_engine = e.h2d;
}

bool is_pinned(const void* p) {
  hipPointerAttribute_t attr{};
  return hipPointerGetAttributes(&attr, p) == hipSuccess && attr.type == hipMemoryTypeHost;
}

// Common part of every bind: validate, plan, upload the chunk table.
kvx_status bind(kvx_ring* r, Dir dir, const kvx_cache* cache, int32_t l0, int32_t l1,
                int32_t chunk_tokens, std::vector<kvx::HostChunk> chunks, int32_t threads,
                bool notional = false) {
  if (threads < 0 || threads > 64) return KVX_EINVAL;
  kvx::Geometry g;
  kvx_status st = kvx::validate(cache, l0, l1, 0, chunk_tokens, false, &g);
  if (st != KVX_OK) return st;
  if (!cache->k || !cache->v) return KVX_EINVAL;
  for (int32_t l = l0; l < l1; ++l) {
    if (!cache->k[l] || !cache->v[l]) return KVX_EINVAL;
    if (((uintptr_t)cache->k[l] | (uintptr_t)cache->v[l]) & 15) return KVX_EINVAL;
  }
  if (kvx::overlaps_cache(cache, l0, l1, r->landing, (int64_t)r->n_slots * r->slot_bytes))
    return KVX_EINVAL;
  int32_t bpc = chunk_tokens / cache->block_size;
  // A chunk's layout depends only on its own block count, so the launches only
  // need blocks-per-chunk up to the largest chunk (keeps padded unit counts small).
  int32_t most = 1;
  for (const auto& c : chunks) most = std::max(most, c.n_blocks);
  for (const auto& c : chunks)
    if (c.n_blocks > bpc) return KVX_EINVAL;
  bpc = std::min(bpc, most);
  kvx::Plan plan;
  st = kvx::plan_chunks(chunks, l0, l1, g.slab, bpc, r->slot_bytes, &plan,
                        dir == Dir::kRestore ? kvx::Ramp::kFirst : kvx::Ramp::kLast);
  if (st != KVX_OK) return st;
  if (threads == 0 && !notional)
    for (const auto& p : plan.pieces)
      for (const auto& sp : p.spans)
        if (!is_pinned(sp.host)) return KVX_EINVAL;  // direct copies need pinned memory
  DeviceGuard dg(r->device);
  if (!dg.ok) return KVX_EHIP;
  drain_device(r);  // the previous transfer may still read d_refs
  const size_t need = std::max<size_t>(plan.refs.size(), 1);
  if (need > r->d_refs_cap) {
    if (r->d_refs) (void)hipFree(r->d_refs);
    r->d_refs = nullptr;
    r->d_refs_cap = 0;
    if (hipMalloc((void**)&r->d_refs, need * sizeof(kvx_chunk_ref)) != hipSuccess) {
      r->d_refs = nullptr;
      r->dir = Dir::kNone;
      return KVX_ENOMEM;
    }
    r->d_refs_cap = need;
  }
  if (!plan.refs.empty() &&
      hipMemcpy(r->d_refs, plan.refs.data(), plan.refs.size() * sizeof(kvx_chunk_ref),
                hipMemcpyHostToDevice) != hipSuccess) {
    r->dir = Dir::kNone;
    return KVX_EHIP;
  }
  r->kptr.assign(cache->k, cache->k + cache->num_layers);
  r->vptr.assign(cache->v, cache->v + cache->num_layers);
  r->cache = *cache;
  r->cache.k = r->kptr.data();
  r->cache.v = r->vptr.data();
  r->chunk_tokens = bpc * cache->block_size;
  r->threads = threads;
  r->plan.pieces.swap(plan.pieces);
  r->plan.refs.swap(plan.refs);
  r->plan.table_len = plan.table_len;
  r->dir = dir;
  for (auto& f : r->files) kvx::close_tier_file(&f);
  r->files.clear();
  r->files_mode = false;
  r->io_depth = 0;
  r->pre = nullptr;
  r->pre_paths.clear();
  r->pre_file.clear();
  r->pre_bytes.clear();
  return KVX_OK;
}

// Bind to chunk files: plan the chunks at their notional addresses.
kvx_status bind_files(kvx_ring* r, Dir dir, const kvx_cache* cache, int32_t l0, int32_t l1,
                      int32_t chunk_tokens, const kvx_file_chunk* chunks, int32_t n_chunks,
                      int32_t io_depth) {
  if (n_chunks < 0 || (n_chunks > 0 && !chunks) || n_chunks >= (1 << 22) || io_depth < 1 ||
      io_depth > 256)
    return KVX_EINVAL;
  kvx::Geometry g;
  kvx_status st = kvx::validate(cache, l0, l1, 0, chunk_tokens, false, &g);
  if (st != KVX_OK) return st;
  std::vector<kvx::TierFile> files((size_t)n_chunks);
  std::vector<kvx::HostChunk> hc((size_t)n_chunks);
  for (int32_t f = 0; f < n_chunks; ++f) {
    const kvx_file_chunk& c = chunks[f];
    if (!c.path || !c.path[0] || c.n_blocks < 1) return KVX_EINVAL;
    files[(size_t)f].path = c.path;
    files[(size_t)f].size = (int64_t)(l1 - l0) * 2 * c.n_blocks * g.slab;
    if (files[(size_t)f].size >= ((int64_t)1 << kFileShift)) return KVX_EINVAL;
    hc[(size_t)f] = kvx::HostChunk{reinterpret_cast<uint8_t*>((uintptr_t)(f + 1) << kFileShift),
                                   c.bt_offset, c.n_blocks};
  }
  st = bind(r, dir, cache, l0, l1, chunk_tokens, std::move(hc), 1, true);
  if (st != KVX_OK) return st;
  // The staging slots are pinned host memory, which cannot be the target of a
  // direct transfer here (EFAULT): the ring's files use buffered I/O, flushed
  // before publication and dropped from the page cache after use.
  for (auto& f : files) f.direct = false;
  r->files = std::move(files);
  r->files_mode = true;
  r->io_depth = io_depth;
  return KVX_OK;
}

// Bind a restore to chunk files held in a preloader's pool: chunks planned at
// notional addresses like files, no fill threads (the DMA engine copies out of
// the pool).
kvx_status bind_preloaded(kvx_ring* r, const kvx_cache* cache, int32_t l0, int32_t l1,
                          int32_t chunk_tokens, kvx_preloader* pre, const kvx_file_chunk* chunks,
                          int32_t n_chunks) {
  if (!pre || !kvx::preload_pinned(pre) || n_chunks < 0 || (n_chunks > 0 && !chunks) ||
      n_chunks >= (1 << 22))
    return KVX_EINVAL;
  kvx::Geometry g;
  kvx_status st = kvx::validate(cache, l0, l1, 0, chunk_tokens, false, &g);
  if (st != KVX_OK) return st;
  std::vector<kvx::HostChunk> hc((size_t)n_chunks);
  std::vector<std::string> paths;
  std::unordered_map<std::string, int32_t> index;
  std::vector<int32_t> file_of((size_t)n_chunks);
  std::vector<int64_t> bytes;
  for (int32_t f = 0; f < n_chunks; ++f) {
    const kvx_file_chunk& c = chunks[f];
    if (!c.path || !c.path[0] || c.n_blocks < 1) return KVX_EINVAL;
    const int64_t size = (int64_t)(l1 - l0) * 2 * c.n_blocks * g.slab;
    if (size >= ((int64_t)1 << kFileShift)) return KVX_EINVAL;
    const auto ins = index.emplace(c.path, (int32_t)paths.size());
    file_of[(size_t)f] = ins.first->second;
    if (ins.second) {
      paths.emplace_back(c.path);
      bytes.push_back(size);
    } else if (bytes[(size_t)ins.first->second] != size) {
      return KVX_EINVAL;  // one file named for chunks of two sizes
    }
    hc[(size_t)f] = kvx::HostChunk{reinterpret_cast<uint8_t*>((uintptr_t)(f + 1) << kFileShift),
                                   c.bt_offset, c.n_blocks};
  }
  st = bind(r, Dir::kRestore, cache, l0, l1, chunk_tokens, std::move(hc), 0, true);
  if (st != KVX_OK) return st;
  r->pre = pre;
  r->pre_paths = std::move(paths);
  r->pre_file = std::move(file_of);
  r->pre_bytes = std::move(bytes);
  return KVX_OK;
}

kvx_status host_chunks(const kvx_host_chunk* chunks, int32_t n,
                       std::vector<kvx::HostChunk>* out) {
  if (n < 0 || (n > 0 && !chunks)) return KVX_EINVAL;
  out->clear();
  for (int32_t i = 0; i < n; ++i)
    out->push_back(kvx::HostChunk{(uint8_t*)chunks[i].host, chunks[i].bt_offset,
                                  chunks[i].n_blocks});
  return KVX_OK;
}

// The deferred store's own stream. The runtime shares a few hardware queues
// round-robin among a process's streams, and a store whose stream shared the
// forward pass's queue waited behind all of it; a stream created with a
// compute-unit mask gets a queue of its own, and a mask of every compute unit
// restricts nothing. Without CU masking, a non-blocking stream.
bool make_store_stream(kvx_ring* r) {
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, r->device) != hipSuccess ||
      cus <= 0)
    return false;
  std::vector<uint32_t> mask((size_t)(cus + 31) / 32, 0u);
  for (int c = 0; c < cus; ++c) mask[(size_t)c / 32] |= 1u << (c % 32);
  if (hipExtStreamCreateWithCUMask(&r->store_stream, (uint32_t)mask.size(), mask.data()) !=
      hipSuccess) {
    (void)hipGetLastError();
    r->store_stream = nullptr;
    if (hipStreamCreateWithFlags(&r->store_stream, hipStreamNonBlocking) != hipSuccess) {
      r->store_stream = nullptr;
      return false;
    }
  }
  if (hipEventCreateWithFlags(&r->store_begin, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&r->restore_end, hipEventDisableTiming) != hipSuccess) {
    if (r->store_begin) (void)hipEventDestroy(r->store_begin);
    (void)hipStreamDestroy(r->store_stream);
    r->store_stream = nullptr;
    r->store_begin = nullptr;
    r->restore_end = nullptr;
    return false;
  }
  return true;
}

// The ring's asynchronous thread: runs each posted transfer, then reports
// its status (an asynchronous restore also records restore_end on the
// ring's stream, after a failure too, so that the caller's stream never
// waits on an event that was not recorded). Returns once told to quit with
// nothing posted.
void async_worker(kvx_ring* r) {
  std::unique_lock<std::mutex> lock(r->async_mu);
  for (;;) {
    r->cv_async.wait(lock, [&] { return r->async_posted || r->async_quit; });
    if (!r->async_posted) return;
    r->async_posted = false;
    const Dir dir = r->async_dir;
    const int32_t* bt = r->async_bt;
    hipStream_t own = r->async_own;
    int* err = r->async_err;
    lock.unlock();
    kvx_status st;
    try {
      st = run(r, dir, bt, own, err);
    } catch (...) {
      st = KVX_EINTERNAL;
    }
    if (dir == Dir::kRestore) {
      DeviceGuard g(r->device);
      if ((!g.ok || hipEventRecord(r->restore_end, own) != hipSuccess) && st == KVX_OK)
        st = KVX_EHIP;
    }
    lock.lock();
    r->async_status = st;
    r->async_done = true;
    r->cv_async.notify_all();
  }
}

// Wait for the posted transfer and return its status.
kvx_status wait_async(kvx_ring* r) {
  std::unique_lock<std::mutex> lock(r->async_mu);
  r->cv_async.wait(lock, [&] { return r->async_done; });
  return r->async_status;
}

// Stop the asynchronous thread (after a posted transfer has run).
void stop_async(kvx_ring* r) {
  {
    std::lock_guard<std::mutex> lock(r->async_mu);
    r->async_quit = true;
  }
  r->cv_async.notify_all();
  if (r->async_th.joinable()) r->async_th.join();
}

// kvx_offload_begin / kvx_restore_begin: the bound transfer on the ring's
// asynchronous thread, its kernels on the ring's stream after the work
// already enqueued on the caller's stream, reporting bad ids to the caller's
// stream.
kvx_status start_async(kvx_ring* ring, Dir dir, const int32_t* block_table, hipStream_t stream) {
  if (!ring) return KVX_EINVAL;
  if (ring->dir != dir) return KVX_EINVAL;
  if (ring->closed.load()) return KVX_ECLOSED;
  if (!block_table && !ring->plan.pieces.empty()) return KVX_EINVAL;
  // claim the ring: of two begins racing on it, one gets KVX_EBUSY
  bool idle = false;
  if (!ring->async_busy.compare_exchange_strong(idle, true)) return KVX_EBUSY;
  auto release = [ring](kvx_status st) {
    ring->async_busy.store(false);
    return st;
  };
  try {
    DeviceGuard dg(ring->device);
    if (!dg.ok) return release(KVX_EHIP);
    if (!ring->store_stream && !make_store_stream(ring)) return release(KVX_EHIP);
    int* err = kvx::stream_error_word(stream);
    if (!err) return release(KVX_EHIP);
    if (hipEventRecord(ring->store_begin, stream) != hipSuccess ||
        hipStreamWaitEvent(ring->store_stream, ring->store_begin, 0) != hipSuccess)
      return release(KVX_EHIP);
    if (!ring->async_th.joinable()) ring->async_th = std::thread(async_worker, ring);
    {
      std::lock_guard<std::mutex> lock(ring->async_mu);
      ring->async_status = KVX_OK;
      ring->async_dir = dir;
      ring->async_bt = block_table;
      ring->async_own = ring->store_stream;
      ring->async_err = err;
      ring->async_done = false;
      ring->async_posted = true;
    }
    ring->cv_async.notify_all();
    return KVX_OK;
  } catch (...) {
    return release(KVX_EINTERNAL);
  }
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
    r->copy_done.assign((size_t)n_slots, nullptr);
    r->dev_done.assign((size_t)n_slots, nullptr);
    for (int32_t s = 0; st == KVX_OK && s < n_slots; ++s) {
      if (hipEventCreateWithFlags(&r->copy_done[s], hipEventDisableTiming | hipEventBlockingSync) !=
              hipSuccess ||
          hipEventCreateWithFlags(&r->dev_done[s], hipEventDisableTiming | hipEventBlockingSync |
                                                       hipEventReleaseToSystem) != hipSuccess)
        st = KVX_EHIP;
    }
    if (st == KVX_OK) setup_dma(r);
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
  if (r->async_busy.load()) return KVX_EBUSY;
  try {
    kvx::Geometry g;
    kvx_status st = kvx::validate(cache, l0, l1, n_blocks, chunk_tokens, false, &g);
    if (st != KVX_OK) return st;
    if (g.n_units > 0 && !host_source) return KVX_EINVAL;
    std::vector<kvx::HostChunk> chunks;
    if (g.n_units > 0) chunks = kvx::image_chunks((uint8_t*)host_source, g);
    return bind(r, Dir::kRestore, cache, l0, l1, g.bpc * cache->block_size, std::move(chunks),
                fill_threads);
  } catch (...) {
    return KVX_EINTERNAL;
  }
}

kvx_status kvx_ring_bind_chunks(kvx_ring* r, const kvx_cache* cache, int32_t l0, int32_t l1,
                                int32_t chunk_tokens, const kvx_host_chunk* chunks,
                                int32_t n_chunks, int32_t fill_threads) {
  if (!r || !cache) return KVX_EINVAL;
  if (r->async_busy.load()) return KVX_EBUSY;
  try {
    std::vector<kvx::HostChunk> v;
    kvx_status st = host_chunks(chunks, n_chunks, &v);
    if (st != KVX_OK) return st;
    return bind(r, Dir::kRestore, cache, l0, l1, chunk_tokens, std::move(v), fill_threads);
  } catch (...) {
    return KVX_EINTERNAL;
  }
}

kvx_status kvx_ring_bind_offload(kvx_ring* r, const kvx_cache* cache, int32_t l0, int32_t l1,
                                 int32_t chunk_tokens, const kvx_host_chunk* chunks,
                                 int32_t n_chunks, int32_t drain_threads) {
  if (!r || !cache) return KVX_EINVAL;
  if (r->async_busy.load()) return KVX_EBUSY;
  try {
    std::vector<kvx::HostChunk> v;
    kvx_status st = host_chunks(chunks, n_chunks, &v);
    if (st != KVX_OK) return st;
    return bind(r, Dir::kOffload, cache, l0, l1, chunk_tokens, std::move(v), drain_threads);
  } catch (...) {
    return KVX_EINTERNAL;
  }
}

kvx_status kvx_ring_bind_files(kvx_ring* r, const kvx_cache* cache, int32_t l0, int32_t l1,
                               int32_t chunk_tokens, const kvx_file_chunk* chunks,
                               int32_t n_chunks, int32_t io_depth) {
  if (!r || !cache) return KVX_EINVAL;
  if (r->async_busy.load()) return KVX_EBUSY;
  try {
    return bind_files(r, Dir::kRestore, cache, l0, l1, chunk_tokens, chunks, n_chunks, io_depth);
  } catch (...) {
    return KVX_EINTERNAL;
  }
}

kvx_status kvx_ring_bind_offload_files(kvx_ring* r, const kvx_cache* cache, int32_t l0,
                                       int32_t l1, int32_t chunk_tokens,
                                       const kvx_file_chunk* chunks, int32_t n_chunks,
                                       int32_t io_depth) {
  if (!r || !cache) return KVX_EINVAL;
  if (r->async_busy.load()) return KVX_EBUSY;
  try {
    return bind_files(r, Dir::kOffload, cache, l0, l1, chunk_tokens, chunks, n_chunks, io_depth);
  } catch (...) {
    return KVX_EINTERNAL;
  }
}

kvx_status kvx_ring_bind_preloaded(kvx_ring* r, const kvx_cache* cache, int32_t l0, int32_t l1,
                                   int32_t chunk_tokens, kvx_preloader* preloader,
                                   const kvx_file_chunk* chunks, int32_t n_chunks) {
  if (!r || !cache) return KVX_EINVAL;
  if (r->async_busy.load()) return KVX_EBUSY;
  try {
    return bind_preloaded(r, cache, l0, l1, chunk_tokens, preloader, chunks, n_chunks);
  } catch (...) {
    return KVX_EINTERNAL;
  }
}

kvx_status kvx_restore_from_staging(kvx_ring* ring, const int32_t* block_table,
                                    hipStream_t stream) {
  if (!ring) return KVX_EINVAL;
  if (ring->async_busy.load()) return KVX_EBUSY;
  try {
    return run(ring, Dir::kRestore, block_table, stream, kvx::stream_error_word(stream));
  } catch (...) {
    return KVX_EINTERNAL;
  }
}

kvx_status kvx_offload_to_staging(kvx_ring* ring, const int32_t* block_table, hipStream_t stream) {
  if (!ring) return KVX_EINVAL;
  if (ring->async_busy.load()) return KVX_EBUSY;
  try {
    return run(ring, Dir::kOffload, block_table, stream, kvx::stream_error_word(stream));
  } catch (...) {
    return KVX_EINTERNAL;
  }
}

kvx_status kvx_offload_begin(kvx_ring* ring, const int32_t* block_table, hipStream_t stream) {
  return start_async(ring, Dir::kOffload, block_table, stream);
}

kvx_status kvx_offload_wait(kvx_ring* ring) {
  if (!ring) return KVX_EINVAL;
  if (!ring->async_busy.load()) return KVX_OK;
  if (ring->async_dir != Dir::kOffload) return KVX_EINVAL;
  const kvx_status st = wait_async(ring);
  ring->async_busy.store(false);
  return st;
}

kvx_status kvx_restore_begin(kvx_ring* ring, const int32_t* block_table, hipStream_t stream) {
  return start_async(ring, Dir::kRestore, block_table, stream);
}

kvx_status kvx_restore_wait(kvx_ring* ring, hipStream_t stream) {
  if (!ring) return KVX_EINVAL;
  if (!ring->async_busy.load()) return KVX_OK;
  if (ring->async_dir != Dir::kRestore) return KVX_EINVAL;
  kvx_status st = wait_async(ring);
  try {
    // the caller's stream continues after the last scatter (restore_end was
    // recorded on the ring's stream after it, also after a failure, so that
    // the stream never waits on an event that was not recorded)
    DeviceGuard dg(ring->device);
    if (!dg.ok || hipStreamWaitEvent(stream, ring->restore_end, 0) != hipSuccess) {
      if (st == KVX_OK) st = KVX_EHIP;
    }
  } catch (...) {
    if (st == KVX_OK) st = KVX_EINTERNAL;
  }
  ring->async_busy.store(false);
  return st;
}

kvx_status kvx_ring_set_test_hooks(kvx_ring* ring, int32_t max_delay_us, int32_t flags) {
  if (!ring || max_delay_us < 0 || max_delay_us > 1000000 || (flags & ~3)) return KVX_EINVAL;
  if (ring->async_busy.load()) return KVX_EBUSY;
  const bool hip_copies = (flags & 2) != 0;
  if (hip_copies != ring->hook_hip_copies) {
    // A restore through the HIP runtime returns with copies still in flight;
    // the other path's waits do not see them: let them finish first.
    try {
      DeviceGuard dg(ring->device);
      if (!dg.ok) return KVX_EHIP;
      drain_device(ring);
    } catch (...) {
      return KVX_EINTERNAL;
    }
  }
  ring->hook_max_delay_us = max_delay_us;
  ring->hook_poison = (flags & 1) != 0;
  ring->hook_hip_copies = hip_copies;
  return KVX_OK;
}

kvx_status kvx_ring_stats_get(const kvx_ring* ring, kvx_ring_stats* out) {
  if (!ring || !out) return KVX_EINVAL;
  if (ring->async_busy.load()) return KVX_EBUSY;
  *out = ring->stats;
  return KVX_OK;
}

kvx_status kvx_ring_set_trace(kvx_ring* ring, int32_t enable) {
  if (!ring || (enable != 0 && enable != 1)) return KVX_EINVAL;
  if (ring->async_busy.load()) return KVX_EBUSY;
  const bool on = enable == 1;
  if (on == ring->trace) return KVX_OK;
  if (ring->hsa_up) copy_profiling(on);
  ring->trace = on;
  return KVX_OK;
}

kvx_status kvx_ring_trace_get(kvx_ring* ring, kvx_trace_event* out, int32_t cap, int32_t* n) {
  if (!ring || !n || cap < 0 || (cap > 0 && !out)) return KVX_EINVAL;
  *n = 0;
  if (ring->async_busy.load()) return KVX_EBUSY;
  if (!ring->traced) return KVX_OK;
  try {
    DeviceGuard dg(ring->device);
    if (!dg.ok) return KVX_EHIP;
    const kvx_status st = trace_resolve(ring);
    if (st != KVX_OK) return st;
    std::lock_guard<std::mutex> lock(ring->mu);
    if (ring->trace_ev.size() > (size_t)INT32_MAX) return KVX_EINTERNAL;
    *n = (int32_t)ring->trace_ev.size();
    for (int32_t i = 0; i < cap && i < *n; ++i) out[i] = ring->trace_ev[(size_t)i];
    return KVX_OK;
  } catch (...) {
    return KVX_EINTERNAL;
  }
}

kvx_status kvx_ring_abort(kvx_ring* ring) {
  if (!ring) return KVX_EINVAL;
  ring->closed.store(true);
  signal_stop(ring);
  return KVX_OK;
}

kvx_status kvx_ring_destroy(kvx_ring* ring) {
  if (!ring) return KVX_OK;
  stop_async(ring);  // after a deferred store or restore still running
  try {
    DeviceGuard dg(ring->device);
    destroy_resources(ring);
  } catch (...) {
  }
  delete ring;
  return KVX_OK;
}

}  // extern "C"
