// Preloading from the storage tier (Sec. 6.5): chunk files of requests that
// are still waiting are read ahead of time into a bounded pool of host slots,
// so that when such a request runs only the host-to-device copy is left on its
// path. One reactor thread owns the pool and an io_uring engine and decides
// what to read next:
//   * demand reads (kvx_preload_fetch) before speculative ones
//     (kvx_preload_hint); speculative pieces are issued only while no demand
//     file has pieces left to issue, so a demand arriving in the middle of a
//     speculative read takes the engine from it at the next piece (the
//     speculative file keeps what it has read and resumes later);
//   * a demand file that finds no slot (none free, no staged image nobody
//     holds) takes one from speculation: if no speculative file has all its
//     pieces issued (which soon frees a slot by staging), the speculative
//     file with the least read stops, hands its slot over once its pieces in
//     flight have landed and is queued to be read again later;
//   * one speculative preload at a time: the files of one hint call (one
//     waiting request) are read concurrently, and the next hint call's files
//     start only when none of them is left; speculative reads take only
//     slots beyond the `reserve`;
//   * a file already staged, being read or queued is never read twice: hints
//     for it are dropped, and a demand fetch claims the staged image or joins
//     the read in progress;
//   * released images stay staged, so the pool is also a cache of chunk
//     images: a speculative read may take the slot of a cached image nobody
//     holds (least recently used first), but never that of a preloaded image
//     not yet fetched; a demand fetch may take either (cached images first).
// A file is read in pieces of kPiece bytes into its slot, with at most
// io_depth pieces in flight (without io_uring, where each piece is read inside
// the issuing call, at most io_depth pieces per hold of the lock). Slots are host memory (pinned for the staged
// restore; plain for host-only use).
#include <hip/hip_runtime_api.h>
#include <sys/stat.h>
#include <unistd.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstdlib>
#include <deque>
#include <memory>
#include <mutex>
#include <new>
#include <string>
#include <thread>
#include <unordered_map>
#include <unordered_set>
#include <vector>

#include "kvx.h"
#include "kvx_io.h"
#include "kvx_preload.h"

namespace {

// 32 MiB: one transfer per 256-token chunk file of an 8B-shaped cache; with
// eight in flight, reads into the pool ran 13 % faster than in 16 MiB pieces.
constexpr int64_t kPiece = 32 << 20;

enum class St { kQueued, kReading, kReady, kFailed };

struct Entry {
  std::string path;
  St st = St::kQueued;
  bool demand = false;   // a fetch waits for it (read before speculative work)
  int32_t slot = -1;
  int64_t size = 0;      // file bytes (known once opened)
  int32_t claims = 0;    // fetches holding its image
  uint64_t group = 0;    // the hint call that queued it
  bool used = false;     // fetched at least once (released, it is a cached image)
  uint64_t last_use = 0;
  kvx::TierFile file;
  int64_t pieces = 0, issued = 0, completed = 0, inflight = 0;
  bool io_error = false;
  bool preempted = false;  // gives its slot to demand once its pieces in flight land
};

}  // namespace

struct kvx_preloader {
  int32_t n_slots = 0;
  int64_t slot_bytes = 0;
  int32_t io_depth = 0;
  int32_t reserve = 0;
  bool pinned = false;
  uint8_t* pool = nullptr;

  std::mutex mu;
  std::condition_variable cv_work;  // the reactor: new work or stop
  std::condition_variable cv_done;  // fetches: an entry became ready or failed
  bool stop = false;
  bool engine_failed = false;
  std::unordered_map<std::string, std::unique_ptr<Entry>> entries;
  std::deque<Entry*> demand_q;  // demand entries with pieces left to issue
  std::deque<Entry*> spec_q;    // speculative entries not yet started
  std::vector<Entry*> spec_reading;  // speculative entries of the active preload being read
  uint64_t groups = 0;          // hint calls so far
  std::vector<int32_t> free_slots;
  uint64_t clock = 0;
  int32_t test_delay_us = 0;  // kvx_preload_set_test_hooks
  kvx_preload_stats stats{};
  std::thread reactor;
};

namespace {

// Remove e from every queue and forget it (the map owns it). The queues hold
// raw pointers, so nothing may erase an entry any other way.
void forget(kvx_preloader* p, Entry* e) {
  auto drop = [e](std::deque<Entry*>& q) {
    for (auto it = q.begin(); it != q.end();) it = *it == e ? q.erase(it) : it + 1;
  };
  drop(p->spec_q);
  drop(p->demand_q);
  p->spec_reading.erase(std::remove(p->spec_reading.begin(), p->spec_reading.end(), e),
                        p->spec_reading.end());
  kvx::close_tier_file(&e->file);
  const std::string path = e->path;
  p->entries.erase(path);
}

// Forget a failed entry nobody holds, freeing the slot it may still have (an
// image discarded as not matching what its holder expected).
void drop_failed(kvx_preloader* p, Entry* e) {
  if (e->slot >= 0) p->free_slots.push_back(e->slot);
  e->slot = -1;
  forget(p, e);
}

// The least recently used staged entry nobody holds: a cached one (fetched
// before), else, if `preloads`, one never fetched. Null if none.
Entry* victim_of(kvx_preloader* p, bool preloads) {
  Entry* best[2] = {nullptr, nullptr};  // cached, preloaded
  for (auto& kv : p->entries) {
    Entry* e = kv.second.get();
    if (e->st != St::kReady || e->claims != 0) continue;
    Entry*& b = best[e->used ? 0 : 1];
    if (!b || e->last_use < b->last_use) b = e;
  }
  return best[0] ? best[0] : (preloads ? best[1] : nullptr);
}

// A slot: a free one (speculation only above the reserve), else that of the
// entry victim_of gives up (demand: any unheld image; speculation: cached
// images only). -1 if none.
int32_t take_slot(kvx_preloader* p, bool demand) {
  if (!p->free_slots.empty() && (demand || (int32_t)p->free_slots.size() > p->reserve)) {
    const int32_t s = p->free_slots.back();
    p->free_slots.pop_back();
    return s;
  }
  Entry* victim = victim_of(p, demand);
  if (!victim) return -1;
  const int32_t s = victim->slot;
  ++p->stats.evictions;
  forget(p, victim);
  return s;
}

// Open e's file and size its read; false (e failed) if it cannot be read
// into one slot.
bool open_entry(kvx_preloader* p, Entry* e) {
  e->file.path = e->path;
  e->file.direct = !p->pinned;  // pinned memory cannot take direct transfers here
  if (kvx::open_tier_file(&e->file, false) != KVX_OK) return false;
  struct stat sb;
  if (fstat(e->file.fd, &sb) != 0 || sb.st_size <= 0 || sb.st_size > p->slot_bytes) return false;
  e->size = sb.st_size;
  e->pieces = (e->size + kPiece - 1) / kPiece;
  // direct transfers need 4 KiB-aligned lengths: a file of another size is
  // read buffered
  if (e->file.direct && (e->size & 4095)) {
    kvx::close_tier_file(&e->file);
    e->file.direct = false;
    if (kvx::open_tier_file(&e->file, false) != KVX_OK) return false;
  }
  return true;
}

void finish_entry(kvx_preloader* p, Entry* e, bool ok) {
  kvx::close_tier_file(&e->file);
  if (ok) {
    e->st = St::kReady;
    e->last_use = ++p->clock;
    p->stats.bytes_read += e->size;
    if (e->demand) ++p->stats.demand_reads;
    else ++p->stats.spec_reads;
  } else {
    e->st = St::kFailed;
    if (e->slot >= 0) p->free_slots.push_back(e->slot);
    e->slot = -1;
    for (auto q = p->demand_q.begin(); q != p->demand_q.end();)
      q = *q == e ? p->demand_q.erase(q) : q + 1;
  }
  p->spec_reading.erase(std::remove(p->spec_reading.begin(), p->spec_reading.end(), e),
                        p->spec_reading.end());
  p->cv_done.notify_all();
}

// A preempted speculative entry whose pieces have all landed: its slot is
// freed and it is queued to be read again from the start, ahead of the
// speculative files not yet started.
void requeue_preempted(kvx_preloader* p, Entry* e) {
  kvx::close_tier_file(&e->file);
  p->free_slots.push_back(e->slot);
  e->slot = -1;
  e->st = St::kQueued;
  e->preempted = false;
  e->io_error = false;
  e->size = e->pieces = e->issued = e->completed = 0;
  p->spec_q.push_front(e);
}

// A demand file found no slot. If a speculative file has all its pieces
// issued, it is staged soon and then gives up its slot: wait for that.
// Otherwise stop the speculative file with the least read. True if that
// freed a slot at once (nothing of it was in flight).
bool preempt_for_demand(kvx_preloader* p) {
  Entry* pick = nullptr;
  for (Entry* e : p->spec_reading) {
    if (e->issued == e->pieces) return false;
    if (!pick || e->completed < pick->completed) pick = e;
  }
  if (!pick) return false;
  ++p->stats.spec_preempted;
  p->spec_reading.erase(std::remove(p->spec_reading.begin(), p->spec_reading.end(), pick),
                        p->spec_reading.end());
  if (pick->inflight > 0) {
    pick->preempted = true;
    return false;
  }
  requeue_preempted(p, pick);
  return true;
}

// Issue pieces (under the lock) while the engine has room: demand entries
// first, then the active speculative entry, then a new speculative entry.
void schedule(kvx_preloader* p, kvx::IoEngine* io) {
  auto issue = [&](Entry* e) {
    while (io->pending() < io->depth() && e->issued < e->pieces && e->st == St::kReading) {
      const int64_t off = e->issued * kPiece;
      const int64_t len = std::min(kPiece, e->size - off);
      if (io->start(&e->file, p->pool + (int64_t)e->slot * p->slot_bytes + off, off, len,
                    (uint64_t)(uintptr_t)e) != KVX_OK) {
        e->io_error = true;
        e->issued = e->pieces;  // issue nothing more; in-flight pieces drain
        break;
      }
      ++e->issued;
      ++e->inflight;  // reported by io->wait (at once without io_uring)
    }
    if (e->issued == e->pieces && e->inflight == 0 && e->st == St::kReading)
      finish_entry(p, e, !e->io_error && e->completed == e->pieces);
  };
  // demand, slots in arrival order; the demand files already being read go
  // on while an earlier one waits for a slot
  bool waiting = false;
  for (size_t i = 0; i < p->demand_q.size() && io->pending() < io->depth();) {
    Entry* e = p->demand_q[i];
    if (e->st == St::kQueued) {
      if (waiting) {
        ++i;
        continue;
      }
      int32_t s = take_slot(p, true);
      if (s < 0 && preempt_for_demand(p)) s = take_slot(p, true);
      if (s < 0) {  // wait for a completion or a release
        waiting = true;
        ++i;
        continue;
      }
      e->slot = s;
      if (!open_entry(p, e)) {
        finish_entry(p, e, false);  // leaves the demand queue
        continue;
      }
      e->st = St::kReading;
    }
    issue(e);  // (a failure inside removes e from the queue itself)
    if (i < p->demand_q.size() && p->demand_q[i] == e) {
      if (e->st != St::kReading || e->issued == e->pieces) p->demand_q.erase(p->demand_q.begin() + (long)i);
      else ++i;
    }
  }
  if (!p->demand_q.empty()) return;  // demand first
  // speculative: the active preload's files being read, then more of its files
  for (size_t i = 0; i < p->spec_reading.size() && io->pending() < io->depth();) {
    Entry* e = p->spec_reading[i];
    issue(e);  // (finishing removes e from spec_reading)
    if (i < p->spec_reading.size() && p->spec_reading[i] == e) ++i;
  }
  while (!p->spec_q.empty() && io->pending() < io->depth()) {
    Entry* e = p->spec_q.front();
    if (e->st != St::kQueued || e->demand) {  // claimed by a demand in the meantime
      p->spec_q.pop_front();
      continue;
    }
    if (!p->spec_reading.empty() && p->spec_reading.front()->group != e->group) return;
    const int32_t s = take_slot(p, false);
    if (s < 0) return;  // keep the reserve for demand
    p->spec_q.pop_front();
    e->slot = s;
    if (!open_entry(p, e)) {
      finish_entry(p, e, false);
      continue;
    }
    e->st = St::kReading;
    p->spec_reading.push_back(e);
    issue(e);
  }
}

// Whether a speculative read could get a slot now.
bool spec_slot_available(kvx_preloader* p) {
  return (int32_t)p->free_slots.size() > p->reserve || victim_of(p, false) != nullptr;
}

// Whether schedule() can make progress now (called with nothing in flight).
bool has_work(kvx_preloader* p) {
  if (!p->demand_q.empty()) {
    for (Entry* e : p->demand_q)
      if (e->st != St::kQueued) return true;  // pieces to issue, or an entry to drop
    // a demand file waits for a slot: a free one, a staged image to evict or
    // a speculative read to stop (with nothing in flight, every speculative
    // file being read has pieces left)
    return !p->free_slots.empty() || victim_of(p, true) != nullptr || !p->spec_reading.empty();
  }
  for (Entry* e : p->spec_reading)
    if (e->issued < e->pieces) return true;
  if (p->spec_q.empty()) return false;
  const Entry* f = p->spec_q.front();
  if (f->st != St::kQueued || f->demand) return true;  // a stale entry to drop
  if (!p->spec_reading.empty() && p->spec_reading.front()->group != f->group) return false;
  return spec_slot_available(p);
}

void reactor_main(kvx_preloader* p) {
  kvx::IoEngine io;
  const bool ok = io.init(p->io_depth, false) == KVX_OK;
  std::vector<uint64_t> done, failed;
  std::unique_lock<std::mutex> lock(p->mu);
  if (!ok) {
    p->engine_failed = true;
    p->cv_done.notify_all();
    return;
  }
  for (;;) {
    if (!p->stop) schedule(p, &io);
    if (io.pending() == 0) {
      if (p->stop) break;
      p->cv_done.notify_all();  // idle: kvx_preload_wait_idle may return
      p->cv_work.wait(lock, [&] { return p->stop || has_work(p); });
      continue;
    }
    const int32_t delay_us = p->test_delay_us;
    lock.unlock();
    done.clear();
    failed.clear();
    const kvx_status st = io.wait(&done, &failed);
    if (delay_us > 0) std::this_thread::sleep_for(std::chrono::microseconds(delay_us));
    lock.lock();
    for (uint64_t t : failed) {
      Entry* e = reinterpret_cast<Entry*>((uintptr_t)t);
      e->io_error = true;
      --e->inflight;
      e->issued = e->pieces;
    }
    for (uint64_t t : done) {
      Entry* e = reinterpret_cast<Entry*>((uintptr_t)t);
      --e->inflight;
      ++e->completed;
    }
    for (std::vector<uint64_t>* tags : {&failed, &done})
      for (uint64_t t : *tags) {
        Entry* e = reinterpret_cast<Entry*>((uintptr_t)t);
        if (e->inflight != 0 || e->st != St::kReading) continue;
        if (e->preempted) requeue_preempted(p, e);
        else if (e->issued == e->pieces) finish_entry(p, e, !e->io_error && e->completed == e->pieces);
      }
    if (st != KVX_OK) {
      // the engine itself failed (not a transfer): fail everything being read
      // and stop; the engine's destructor waits for what is still in flight
      p->engine_failed = true;
      for (auto& kv : p->entries)
        if (kv.second->st == St::kReading) {
          kv.second->inflight = 0;
          finish_entry(p, kv.second.get(), false);
        }
      p->cv_done.notify_all();
      break;
    }
  }
}

bool valid_paths(const char* const* paths, int32_t n) {
  if (n < 0 || (n > 0 && !paths)) return false;
  for (int32_t i = 0; i < n; ++i)
    if (!paths[i] || !paths[i][0]) return false;
  return true;
}

// The distinct paths, in the order of their first occurrence.
std::vector<std::string> distinct(const char* const* paths, int32_t n) {
  std::vector<std::string> out;
  std::unordered_set<std::string> seen;
  for (int32_t i = 0; i < n; ++i)
    if (seen.insert(paths[i]).second) out.emplace_back(paths[i]);
  return out;
}

// Hold each of the distinct files (all or none), in order: staged images are
// claimed, speculative reads in progress joined (their remaining pieces become
// demand), queued hints promoted, other files queued as demand reads. Called
// with the lock held; KVX_ENOMEM if the files held afterwards would exceed the
// pool, KVX_EIO if a file failed and is still held or draining elsewhere.
kvx_status hold_locked(kvx_preloader* p, const std::vector<std::string>& uniq,
                       std::vector<Entry*>* out) {
  if (p->engine_failed) return KVX_EIO;
  int32_t held = 0, held_here = 0;
  for (auto& kv : p->entries)
    if (kv.second->claims > 0) ++held;
  for (const auto& path : uniq) {
    auto it = p->entries.find(path);
    if (it != p->entries.end() && it->second->claims > 0) ++held_here;
  }
  if (held + (int32_t)uniq.size() - held_here > p->n_slots) return KVX_ENOMEM;
  std::vector<Entry*> es;
  for (const auto& path : uniq) {
    auto it = p->entries.find(path);
    Entry* e;
    if (it == p->entries.end() || it->second->st == St::kFailed) {
      // a failed entry another holder still holds, or whose reads still
      // drain, is left alone: that holder reports the failure
      if (it != p->entries.end() && (it->second->inflight > 0 || it->second->claims > 0)) {
        for (Entry* h : es) --h->claims;
        return KVX_EIO;
      }
      if (it != p->entries.end()) drop_failed(p, it->second.get());  // a failed entry nobody holds
      auto ne = std::make_unique<Entry>();
      ne->path = path;
      e = ne.get();
      p->entries[path] = std::move(ne);
      e->demand = true;
      p->demand_q.push_back(e);
    } else {
      e = it->second.get();
      if (e->st == St::kReady) {
        ++p->stats.hits_ready;
      } else if (e->st == St::kReading && !e->demand) {
        ++p->stats.hits_inflight;
        if (e->issued < e->pieces) p->demand_q.push_back(e);  // its remaining pieces now have priority
        e->demand = true;
        e->preempted = false;  // stopped for another demand file: it keeps its slot after all
        p->spec_reading.erase(std::remove(p->spec_reading.begin(), p->spec_reading.end(), e),
                              p->spec_reading.end());
      } else if (e->st == St::kQueued && !e->demand) {
        e->demand = true;  // a hinted file not yet started: read it now
        for (auto q = p->spec_q.begin(); q != p->spec_q.end();)
          q = *q == e ? p->spec_q.erase(q) : q + 1;
        p->demand_q.push_back(e);
      }
    }
    ++e->claims;
    e->used = true;
    es.push_back(e);
  }
  p->stats.demand_fetches += (int64_t)uniq.size();
  p->cv_work.notify_one();
  *out = std::move(es);
  return KVX_OK;
}

// Drop one hold of each entry (distinct, each held). Failed entries nobody
// holds any more are forgotten, so that a later fetch reads them again.
void unhold_locked(kvx_preloader* p, const std::vector<Entry*>& es) {
  for (Entry* e : es) {
    --e->claims;
    e->last_use = ++p->clock;
  }
  for (Entry* e : es)
    if (e->st == St::kFailed && e->claims == 0 && e->inflight == 0) drop_failed(p, e);
  p->cv_work.notify_one();
}

}  // namespace

extern "C" {

kvx_status kvx_preloader_create(int32_t n_slots, int64_t slot_bytes, int32_t io_depth,
                                int32_t reserve, int32_t pinned, kvx_preloader** out) {
  if (!out) return KVX_EINVAL;
  *out = nullptr;
  if (n_slots < 1 || n_slots > 65536 || slot_bytes <= 0 || slot_bytes % 4096 != 0 ||
      io_depth < 1 || io_depth > 256 || reserve < 0 || reserve >= n_slots ||
      (pinned != 0 && pinned != 1))
    return KVX_EINVAL;
  int64_t total = 0;
  if (__builtin_mul_overflow((int64_t)n_slots, slot_bytes, &total)) return KVX_EINVAL;
  kvx_preloader* p = new (std::nothrow) kvx_preloader();
  if (!p) return KVX_ENOMEM;
  p->n_slots = n_slots;
  p->slot_bytes = slot_bytes;
  p->io_depth = io_depth;
  p->reserve = reserve;
  p->pinned = pinned == 1;
  void* mem = nullptr;
  if (p->pinned) {
    if (hipHostMalloc(&mem, (size_t)total, hipHostMallocDefault) != hipSuccess) mem = nullptr;
  } else {
    mem = std::aligned_alloc(4096, (size_t)total);
  }
  if (!mem) {
    delete p;
    return KVX_ENOMEM;
  }
  p->pool = static_cast<uint8_t*>(mem);
  // The pool's pages are mapped on first touch: reads into a freshly
  // allocated pinned pool ran at less than half the rate of reads into a
  // touched one. Touch every page now, off the request path.
  for (int64_t off = 0; off < total; off += 4096) p->pool[off] = 0;
  try {
    for (int32_t s = n_slots - 1; s >= 0; --s) p->free_slots.push_back(s);
    p->reactor = std::thread(reactor_main, p);
  } catch (...) {
    if (p->pinned) (void)hipHostFree(p->pool);
    else std::free(p->pool);
    delete p;
    return KVX_EINTERNAL;
  }
  *out = p;
  return KVX_OK;
}

kvx_status kvx_preload_hint(kvx_preloader* p, const char* const* paths, int32_t n) {
  if (!p || !valid_paths(paths, n)) return KVX_EINVAL;
  try {
    std::lock_guard<std::mutex> lock(p->mu);
    const uint64_t group = ++p->groups;
    for (int32_t i = 0; i < n; ++i) {
      const std::string path(paths[i]);
      auto it = p->entries.find(path);
      if (it != p->entries.end() && (it->second->st != St::kFailed || it->second->claims > 0 ||
                                     it->second->inflight > 0)) {
        ++p->stats.spec_deduped;
        continue;
      }
      if ((int32_t)p->spec_q.size() >= p->n_slots) {  // bounded lookahead
        ++p->stats.spec_dropped;
        continue;
      }
      if (it != p->entries.end()) drop_failed(p, it->second.get());  // a failed entry nobody holds
      auto e = std::make_unique<Entry>();
      e->path = path;
      e->group = group;
      p->spec_q.push_back(e.get());
      p->entries[path] = std::move(e);
      ++p->stats.hints;
    }
    p->cv_work.notify_one();
    return KVX_OK;
  } catch (...) {
    return KVX_EINTERNAL;
  }
}

kvx_status kvx_preload_fetch(kvx_preloader* p, const char* const* paths, int32_t n, void** images,
                             int64_t* sizes) {
  if (!p || !valid_paths(paths, n) || (n > 0 && (!images || !sizes))) return KVX_EINVAL;
  try {
    std::unique_lock<std::mutex> lock(p->mu);
    std::vector<Entry*> es;
    kvx_status st = hold_locked(p, distinct(paths, n), &es);
    if (st != KVX_OK) return st;
    p->cv_done.wait(lock, [&] {
      if (p->engine_failed) return true;
      for (Entry* e : es)
        if (e->st != St::kReady && e->st != St::kFailed) return false;
      return true;
    });
    bool ok = !p->engine_failed;
    for (Entry* e : es) ok = ok && e->st == St::kReady;
    if (!ok) {
      unhold_locked(p, es);
      return KVX_EIO;
    }
    for (int32_t i = 0; i < n; ++i) {
      const Entry* e = p->entries.at(paths[i]).get();
      images[i] = p->pool + (int64_t)e->slot * p->slot_bytes;
      sizes[i] = e->size;
    }
    return KVX_OK;
  } catch (...) {
    return KVX_EINTERNAL;
  }
}

kvx_status kvx_preload_release(kvx_preloader* p, const char* const* paths, int32_t n) {
  if (!p || !valid_paths(paths, n)) return KVX_EINVAL;
  try {
    std::lock_guard<std::mutex> lock(p->mu);
    std::vector<Entry*> es;
    for (const auto& path : distinct(paths, n)) {
      auto it = p->entries.find(path);
      if (it == p->entries.end() || it->second->claims <= 0) return KVX_EINVAL;
      es.push_back(it->second.get());
    }
    unhold_locked(p, es);
    return KVX_OK;
  } catch (...) {
    return KVX_EINTERNAL;
  }
}

kvx_status kvx_preload_stats_get(kvx_preloader* p, kvx_preload_stats* out) {
  if (!p || !out) return KVX_EINVAL;
  std::lock_guard<std::mutex> lock(p->mu);
  *out = p->stats;
  out->staged = 0;
  out->held = 0;
  for (auto& kv : p->entries) {
    if (kv.second->st == St::kReady) ++out->staged;
    if (kv.second->claims > 0) ++out->held;
  }
  return KVX_OK;
}

kvx_status kvx_preload_wait_idle(kvx_preloader* p) {
  if (!p) return KVX_EINVAL;
  std::unique_lock<std::mutex> lock(p->mu);
  p->cv_done.wait(lock, [&] {
    if (p->engine_failed) return true;
    if (!p->demand_q.empty() || !p->spec_reading.empty()) return false;
    bool queued = false;
    for (auto& kv : p->entries) {
      if (kv.second->st == St::kReading) return false;
      if (kv.second->st == St::kQueued) queued = true;
    }
    return !queued || !spec_slot_available(p);
  });
  return p->engine_failed ? KVX_EIO : KVX_OK;
}

kvx_status kvx_preload_set_test_hooks(kvx_preloader* p, int32_t delay_us) {
  if (!p || delay_us < 0 || delay_us > 1000000) return KVX_EINVAL;
  std::lock_guard<std::mutex> lock(p->mu);
  p->test_delay_us = delay_us;
  return KVX_OK;
}

kvx_status kvx_preloader_destroy(kvx_preloader* p) {
  if (!p) return KVX_OK;
  {
    std::lock_guard<std::mutex> lock(p->mu);
    p->stop = true;
  }
  p->cv_work.notify_all();
  if (p->reactor.joinable()) p->reactor.join();
  for (auto& kv : p->entries) kvx::close_tier_file(&kv.second->file);
  if (p->pinned) (void)hipHostFree(p->pool);
  else std::free(p->pool);
  delete p;
  return KVX_OK;
}

}  // extern "C"

// ---- holds for a restore that copies each image as soon as it is staged ----

namespace kvx {

bool preload_pinned(const kvx_preloader* p) { return p->pinned; }

kvx_status preload_hold(kvx_preloader* p, const std::vector<std::string>& paths,
                        std::vector<void*>* handles) {
  try {
    std::lock_guard<std::mutex> lock(p->mu);
    std::vector<Entry*> es;
    const kvx_status st = hold_locked(p, paths, &es);
    if (st != KVX_OK) return st;
    handles->assign(es.begin(), es.end());
    return KVX_OK;
  } catch (...) {
    return KVX_EINTERNAL;
  }
}

kvx_status preload_image(kvx_preloader* p, void* handle, bool wait,
                         const std::atomic<bool>* cancel, uint8_t** image, int64_t* size) {
  Entry* e = static_cast<Entry*>(handle);
  std::unique_lock<std::mutex> lock(p->mu);
  auto settled = [&] { return p->engine_failed || e->st == St::kReady || e->st == St::kFailed; };
  while (wait && !settled()) {
    if (cancel && cancel->load()) return KVX_ECLOSED;
    p->cv_done.wait_for(lock, std::chrono::milliseconds(5), settled);
  }
  if (e->st == St::kReady) {
    *image = p->pool + (int64_t)e->slot * p->slot_bytes;
    *size = e->size;
    return KVX_OK;
  }
  if (p->engine_failed || e->st == St::kFailed) return KVX_EIO;
  *image = nullptr;
  return KVX_OK;
}

void preload_discard(kvx_preloader* p, void* handle) {
  std::lock_guard<std::mutex> lock(p->mu);
  Entry* e = static_cast<Entry*>(handle);
  if (e->st == St::kReady) e->st = St::kFailed;  // read again by the next holder
}

void preload_unhold(kvx_preloader* p, const std::vector<void*>& handles) {
  std::lock_guard<std::mutex> lock(p->mu);
  std::vector<Entry*> es;
  for (void* h : handles) es.push_back(static_cast<Entry*>(h));
  unhold_locked(p, es);
}

}  // namespace kvx
