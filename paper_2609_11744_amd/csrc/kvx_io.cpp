// Storage-tier I/O engine (see kvx_io.h) and the host entry points that use
// it directly: kvx_chunk_path, kvx_read_files, kvx_write_files.
#include "kvx_io.h"

#include <errno.h>
#include <fcntl.h>
#include <linux/io_uring.h>
#include <sys/mman.h>
#include <sys/stat.h>
#include <sys/syscall.h>
#include <unistd.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>

namespace kvx {

namespace {

std::atomic<uint64_t> g_temp_counter{0};

// mkdir -p of the directory part of `path`.
bool make_parent_dirs(const std::string& path) {
  for (size_t i = 1; i < path.size(); ++i) {
    if (path[i] != '/') continue;
    const std::string dir = path.substr(0, i);
    if (mkdir(dir.c_str(), 0755) != 0 && errno != EEXIST) return false;
  }
  return true;
}

int open_maybe_direct(const char* path, int flags, bool* direct, mode_t mode = 0) {
  if (*direct) {
    const int fd = open(path, flags | O_DIRECT | O_CLOEXEC, mode);
    if (fd >= 0 || errno != EINVAL) return fd;
    *direct = false;  // the filesystem takes no O_DIRECT (e.g. tmpfs)
  }
  return open(path, flags | O_CLOEXEC, mode);
}

// At most this many bytes per submitted transfer (a read or write returns at
// most ~2 GiB at a time anyway); the rest is resubmitted.
constexpr int64_t kMaxTransfer = 1 << 30;

}  // namespace

kvx_status open_tier_file(TierFile* f, bool write) {
  if (f->fd >= 0) return KVX_OK;
  if (!write) {
    f->fd = open_maybe_direct(f->path.c_str(), O_RDONLY, &f->direct);
    return f->fd >= 0 ? KVX_OK : KVX_EIO;
  }
  if (!make_parent_dirs(f->path)) return KVX_EIO;
  char suffix[64];
  std::snprintf(suffix, sizeof suffix, ".tmp.%ld.%llu", (long)getpid(),
                (unsigned long long)g_temp_counter.fetch_add(1));
  f->temp = f->path + suffix;
  f->fd = open_maybe_direct(f->temp.c_str(), O_WRONLY | O_CREAT | O_EXCL, &f->direct, 0644);
  if (f->fd < 0) {
    f->temp.clear();
    return KVX_EIO;
  }
  f->written = 0;
  f->flushing = false;
  f->published = false;
  return KVX_OK;
}

// Reopen a file without O_DIRECT (its direct transfers failed) at the same
// name: the final name for reads, the temporary one for writes. The old
// descriptor is kept open until the file is closed: other transfers of the
// file may still be in flight on it (they fail the same way and are repeated
// on the new one).
bool reopen_buffered(TierFile* f, bool write) {
  if (f->fd >= 0) f->retired.push_back(f->fd);
  f->direct = false;
  f->fd = write ? open(f->temp.c_str(), O_WRONLY | O_CLOEXEC)
                : open(f->path.c_str(), O_RDONLY | O_CLOEXEC);
  return f->fd >= 0;
}

kvx_status publish_tier_file(TierFile* f) {
  if (f->published) return KVX_OK;
  if (f->fd >= 0) {
    if (!f->direct) posix_fadvise(f->fd, 0, 0, POSIX_FADV_DONTNEED);  // flushed: drop the pages
    close(f->fd);
  }
  f->fd = -1;
  for (int fd : f->retired) close(fd);
  f->retired.clear();
  const bool linked = link(f->temp.c_str(), f->path.c_str()) == 0 || errno == EEXIST;
  unlink(f->temp.c_str());
  f->temp.clear();
  f->published = linked;
  return linked ? KVX_OK : KVX_EIO;
}

void close_tier_file(TierFile* f) {
  if (f->fd >= 0) {
    if (!f->direct && f->temp.empty()) posix_fadvise(f->fd, 0, 0, POSIX_FADV_DONTNEED);
    close(f->fd);
  }
  f->fd = -1;
  for (int fd : f->retired) close(fd);
  f->retired.clear();
  if (!f->temp.empty() && !f->published) unlink(f->temp.c_str());
  f->temp.clear();
}

// ---- IoEngine ------------------------------------------------------------------

IoEngine::~IoEngine() {
  drain();
  if (sqe_map_) munmap(sqe_map_, sqe_map_len_);
  if (cq_map_ && cq_map_ != sq_map_) munmap(cq_map_, cq_map_len_);
  if (sq_map_) munmap(sq_map_, sq_map_len_);
  if (ring_fd_ >= 0) close(ring_fd_);
}

kvx_status IoEngine::init(int32_t depth, bool write) {
  if (depth < 1 || depth > 256 || ring_fd_ >= 0 || depth_ > 0) return KVX_EINVAL;
  write_ = write;
  depth_ = depth;
  ops_.assign((size_t)depth, Op{nullptr, nullptr, 0, 0, 0, false, -1});
  const char* off = getenv("KVX_IO_NO_URING");
  if (off && off[0] == '1') return KVX_OK;  // blocking fallback, by request
  io_uring_params p;
  std::memset(&p, 0, sizeof p);
  const int fd = (int)syscall(__NR_io_uring_setup, (unsigned)depth, &p);
  if (fd < 0) return KVX_OK;  // synchronous fallback
  sq_map_len_ = p.sq_off.array + p.sq_entries * sizeof(unsigned);
  cq_map_len_ = p.cq_off.cqes + p.cq_entries * sizeof(io_uring_cqe);
  sq_map_ = mmap(nullptr, sq_map_len_, PROT_READ | PROT_WRITE, MAP_SHARED | MAP_POPULATE, fd,
                 IORING_OFF_SQ_RING);
  cq_map_ = mmap(nullptr, cq_map_len_, PROT_READ | PROT_WRITE, MAP_SHARED | MAP_POPULATE, fd,
                 IORING_OFF_CQ_RING);
  sqe_map_len_ = p.sq_entries * sizeof(io_uring_sqe);
  sqe_map_ = mmap(nullptr, sqe_map_len_, PROT_READ | PROT_WRITE, MAP_SHARED | MAP_POPULATE, fd,
                  IORING_OFF_SQES);
  if (sq_map_ == MAP_FAILED || cq_map_ == MAP_FAILED || sqe_map_ == MAP_FAILED) {
    if (sq_map_ != MAP_FAILED) munmap(sq_map_, sq_map_len_);
    if (cq_map_ != MAP_FAILED) munmap(cq_map_, cq_map_len_);
    if (sqe_map_ != MAP_FAILED) munmap(sqe_map_, sqe_map_len_);
    sq_map_ = cq_map_ = sqe_map_ = nullptr;
    close(fd);
    return KVX_OK;  // synchronous fallback
  }
  uint8_t* sq = static_cast<uint8_t*>(sq_map_);
  uint8_t* cq = static_cast<uint8_t*>(cq_map_);
  sq_tail_ = reinterpret_cast<unsigned*>(sq + p.sq_off.tail);
  sq_mask_ = reinterpret_cast<unsigned*>(sq + p.sq_off.ring_mask);
  sq_array_ = reinterpret_cast<unsigned*>(sq + p.sq_off.array);
  cq_head_ = reinterpret_cast<unsigned*>(cq + p.cq_off.head);
  cq_tail_ = reinterpret_cast<unsigned*>(cq + p.cq_off.tail);
  cq_mask_ = reinterpret_cast<unsigned*>(cq + p.cq_off.ring_mask);
  cqes_ = cq + p.cq_off.cqes;
  sqes_ = sqe_map_;
  sq_entries_ = p.sq_entries;
  ring_fd_ = fd;
  return KVX_OK;
}

// After a failure, transfers the kernel still holds keep writing into (or
// reading from) their buffers until they complete, and closing the ring does
// not wait for them: reap completions (submitting what is queued) until none
// is in flight, for at most 30 s, so that the caller may free the buffers.
void IoEngine::drain() {
  if (ring_fd_ < 0 || inflight_ == 0) return;
  const auto deadline = std::chrono::steady_clock::now() + std::chrono::seconds(30);
  while (inflight_ > 0 && std::chrono::steady_clock::now() < deadline) {
    unsigned head = *cq_head_;
    const unsigned tail = __atomic_load_n(cq_tail_, __ATOMIC_ACQUIRE);
    for (; head != tail; ++head) {
      const io_uring_cqe* cqe = static_cast<const io_uring_cqe*>(cqes_) + (head & *cq_mask_);
      const uint64_t slot = cqe->user_data;
      if (slot < (uint64_t)depth_ && ops_[(size_t)slot].live) {
        ops_[(size_t)slot].live = false;
        --inflight_;
      }
    }
    __atomic_store_n(cq_head_, head, __ATOMIC_RELEASE);
    if (inflight_ == 0) break;
    const long n = syscall(__NR_io_uring_enter, ring_fd_, to_submit_, 1u, IORING_ENTER_GETEVENTS,
                           nullptr, 0);
    if (n >= 0) to_submit_ -= (unsigned)n < to_submit_ ? (unsigned)n : to_submit_;
    else usleep(1000);
  }
}

bool IoEngine::enter(unsigned min_complete) {
  for (;;) {
    const long n = syscall(__NR_io_uring_enter, ring_fd_, to_submit_, min_complete,
                           min_complete ? IORING_ENTER_GETEVENTS : 0u, nullptr, 0);
    if (n >= 0) {
      to_submit_ -= (unsigned)n < to_submit_ ? (unsigned)n : to_submit_;
      if (to_submit_ == 0 || min_complete) return true;
      continue;
    }
    if (errno != EINTR && errno != EAGAIN && errno != EBUSY) return false;
  }
}

kvx_status IoEngine::submit(int32_t slot) {
  Op& op = ops_[(size_t)slot];
  const unsigned tail = *sq_tail_;
  const unsigned idx = tail & *sq_mask_;
  io_uring_sqe* sqe = static_cast<io_uring_sqe*>(sqes_) + idx;
  std::memset(sqe, 0, sizeof *sqe);
  op.fd = op.f->fd;
  sqe->fd = op.fd;
  sqe->user_data = (uint64_t)slot;
  if (op.left < 0) {
    sqe->opcode = IORING_OP_FSYNC;
    sqe->fsync_flags = IORING_FSYNC_DATASYNC;
  } else {
    sqe->opcode = write_ ? IORING_OP_WRITE : IORING_OP_READ;
    sqe->off = (uint64_t)op.offset;
    sqe->addr = (uint64_t)(uintptr_t)op.buf;
    sqe->len = (uint32_t)std::min(op.left, kMaxTransfer);
  }
  sq_array_[idx] = idx;
  __atomic_store_n(sq_tail_, tail + 1, __ATOMIC_RELEASE);
  ++to_submit_;
  return enter(0) ? KVX_OK : KVX_EIO;
}

int32_t IoEngine::take_slot() {
  int32_t slot = 0;
  while (ops_[(size_t)slot].live) ++slot;  // callers keep inflight_ < depth_
  ++inflight_;
  return slot;
}

kvx_status IoEngine::start(TierFile* f, uint8_t* buf, int64_t offset, int64_t bytes,
                           uint64_t tag) {
  if (!f || f->fd < 0 || !buf || offset < 0 || bytes <= 0 || inflight_ >= depth_)
    return KVX_EINVAL;
  if (ring_fd_ < 0) {  // synchronous fallback
    while (bytes > 0) {
      const size_t len = (size_t)std::min(bytes, kMaxTransfer);
      const ssize_t n = write_ ? pwrite(f->fd, buf, len, offset) : pread(f->fd, buf, len, offset);
      if (n < 0 && errno == EINTR) continue;
      if (n < 0 && errno == EFAULT && f->direct) {
        if (!reopen_buffered(f, write_)) return KVX_EIO;
        continue;
      }
      if (n <= 0) return KVX_EIO;
      if (!write_ && !f->direct) posix_fadvise(f->fd, offset, n, POSIX_FADV_DONTNEED);
      buf += n;
      offset += n;
      bytes -= n;
      if (write_) f->written += n;
    }
    finished_.push_back(tag);
    return KVX_OK;
  }
  const int32_t slot = take_slot();
  ops_[(size_t)slot] = Op{f, buf, offset, bytes, tag, true, -1};
  return submit(slot);
}

kvx_status IoEngine::start_datasync(TierFile* f, uint64_t tag) {
  if (!write_ || !f || f->fd < 0 || inflight_ >= depth_) return KVX_EINVAL;
  if (ring_fd_ < 0) {
    if (fdatasync(f->fd) != 0) return KVX_EIO;
    finished_.push_back(tag);
    return KVX_OK;
  }
  const int32_t slot = take_slot();
  ops_[(size_t)slot] = Op{f, nullptr, 0, -1, tag, true, -1};
  return submit(slot);
}

kvx_status IoEngine::wait(std::vector<uint64_t>* done, std::vector<uint64_t>* failed) {
  const size_t before = done->size() + (failed ? failed->size() : 0);
  auto reported = [&]() { return done->size() + (failed ? failed->size() : 0) > before; };
  done->insert(done->end(), finished_.begin(), finished_.end());
  finished_.clear();
  if (ring_fd_ < 0 || reported() || inflight_ == 0) return KVX_OK;
  for (;;) {
    unsigned head = *cq_head_;
    const unsigned tail = __atomic_load_n(cq_tail_, __ATOMIC_ACQUIRE);
    kvx_status st = KVX_OK;
    while (head != tail) {
      const io_uring_cqe* cqe = static_cast<const io_uring_cqe*>(cqes_) + (head & *cq_mask_);
      const int32_t slot = (int32_t)cqe->user_data;
      const int32_t res = cqe->res;
      ++head;
      if (slot < 0 || slot >= depth_ || !ops_[(size_t)slot].live) {
        st = KVX_EINTERNAL;
        continue;
      }
      Op& op = ops_[(size_t)slot];
      if (op.left < 0) {  // an fdatasync
        op.live = false;
        --inflight_;
        if (res >= 0) done->push_back(op.tag);
        else if (failed) failed->push_back(op.tag);
        else st = KVX_EIO;
        continue;
      }
      if (res == -EFAULT && (op.f->direct || op.fd != op.f->fd)) {
        // pinned memory: repeat it buffered (the file may have been reopened
        // for another of its transfers already)
        __atomic_store_n(cq_head_, head, __ATOMIC_RELEASE);
        if ((op.f->direct && !reopen_buffered(op.f, write_)) || submit(slot) != KVX_OK) st = KVX_EIO;
        continue;
      }
      if (res <= 0) {  // an error, or end of file before the op's last byte
        op.live = false;
        --inflight_;
        if (failed) failed->push_back(op.tag);
        else st = KVX_EIO;
        continue;
      }
      if (write_) op.f->written += res;
      if (!write_ && !op.f->direct) posix_fadvise(op.f->fd, op.offset, res, POSIX_FADV_DONTNEED);
      op.buf += res;
      op.offset += res;
      op.left -= res;
      if (op.left > 0) {
        __atomic_store_n(cq_head_, head, __ATOMIC_RELEASE);
        if (submit(slot) != KVX_OK) st = KVX_EIO;
        continue;
      }
      op.live = false;
      --inflight_;
      done->push_back(op.tag);
    }
    __atomic_store_n(cq_head_, head, __ATOMIC_RELEASE);
    if (st != KVX_OK) return st;
    if (reported() || inflight_ == 0) return KVX_OK;
    if (!enter(1)) return KVX_EIO;
  }
}

}  // namespace kvx

// ---- host entry points -------------------------------------------------------------

namespace {

// Ops grouped by file path: one TierFile per distinct path, in first-use order.
struct Batch {
  std::vector<kvx::TierFile> files;
  std::vector<int32_t> file_of;  // per op
};

kvx_status group(const kvx_file_io* ops, int32_t n, Batch* b) {
  std::map<std::string, int32_t> index;
  for (int32_t i = 0; i < n; ++i) {
    const kvx_file_io& o = ops[i];
    if (!o.path || !o.path[0] || !o.buf || o.offset < 0 || o.bytes <= 0) return KVX_EINVAL;
    auto it = index.find(o.path);
    int32_t f;
    if (it == index.end()) {
      f = (int32_t)b->files.size();
      index.emplace(o.path, f);
      b->files.emplace_back();
      b->files.back().path = o.path;
    } else {
      f = it->second;
    }
    kvx::TierFile& tf = b->files[(size_t)f];
    tf.size = std::max(tf.size, o.offset + o.bytes);
    if (!kvx::io_aligned(o.buf, o.offset, o.bytes)) tf.direct = false;
    b->file_of.push_back(f);
  }
  return KVX_OK;
}

kvx_status run_batch(const kvx_file_io* ops, int32_t n, int32_t depth, bool write) {
  if (n < 0 || (n > 0 && !ops) || depth < 1 || depth > 256) return KVX_EINVAL;
  if (n == 0) return KVX_OK;
  Batch b;
  kvx_status st = group(ops, n, &b);
  if (st != KVX_OK) return st;
  if (write) {
    // Each file's ops must tile [0, size) exactly: sort by offset and check.
    std::vector<std::vector<std::pair<int64_t, int64_t>>> parts(b.files.size());
    for (int32_t i = 0; i < n; ++i)
      parts[(size_t)b.file_of[(size_t)i]].emplace_back(ops[i].offset, ops[i].bytes);
    for (auto& v : parts) {
      std::sort(v.begin(), v.end());
      int64_t at = 0;
      for (const auto& p : v) {
        if (p.first != at) return KVX_EINVAL;
        at += p.second;
      }
    }
  }
  kvx::IoEngine io;
  st = io.init(depth, write);
  std::vector<uint64_t> done;
  std::vector<int32_t> to_sync;  // buffered files fully written, to flush before publishing
  int32_t next = 0;
  while (st == KVX_OK && (next < n || io.pending() > 0 || !to_sync.empty())) {
    while (st == KVX_OK && !to_sync.empty() && io.inflight() < io.depth()) {
      const int32_t f = to_sync.back();
      to_sync.pop_back();
      st = io.start_datasync(&b.files[(size_t)f], kvx::kSyncTag | (uint64_t)f);
    }
    while (st == KVX_OK && next < n && io.inflight() < io.depth()) {
      kvx::TierFile& f = b.files[(size_t)b.file_of[(size_t)next]];
      st = kvx::open_tier_file(&f, write);
      if (st == KVX_OK)
        st = io.start(&f, static_cast<uint8_t*>(ops[next].buf), ops[next].offset,
                      ops[next].bytes, (uint64_t)next);
      ++next;
      if (!io.uring()) break;  // synchronous: report as we go
    }
    done.clear();
    if (st == KVX_OK) st = io.wait(&done);
    for (uint64_t t : done) {
      if (t & kvx::kSyncTag) {  // flushed: publish
        if (st == KVX_OK) st = kvx::publish_tier_file(&b.files[(size_t)(t & ~kvx::kSyncTag)]);
        continue;
      }
      const int32_t fi = b.file_of[(size_t)t];
      kvx::TierFile& f = b.files[(size_t)fi];
      // (several of a file's transfers can finish in one wait: act once)
      if (write && st == KVX_OK && f.written == f.size && !f.published && !f.flushing) {
        if (f.direct) {
          st = kvx::publish_tier_file(&f);
        } else {
          f.flushing = true;
          to_sync.push_back(fi);
        }
      }
    }
  }
  while (io.inflight() > 0) {  // after an error: let what is in flight land
    const int32_t before = io.inflight();
    done.clear();
    if (io.wait(&done) != KVX_OK && io.inflight() == before) break;  // no progress possible
  }
  for (auto& f : b.files) kvx::close_tier_file(&f);
  return st;
}

}  // namespace

extern "C" {

int32_t kvx_chunk_path(const char* root, const char* tag, uint64_t key, char* out, int32_t cap) {
  if (!root || !root[0] || !tag || !tag[0] || strchr(tag, '/') || !out || cap <= 0) return -1;
  const int n = std::snprintf(out, (size_t)cap, "%s/%s/%02x/%02x/%016llx.kvc", root, tag,
                              (unsigned)(key >> 56), (unsigned)((key >> 48) & 0xff),
                              (unsigned long long)key);
  return n >= 0 && n < cap ? n : -1;
}

kvx_status kvx_read_files(const kvx_file_io* ops, int32_t n, int32_t io_depth) {
  try {
    return run_batch(ops, n, io_depth, false);
  } catch (...) {
    return KVX_EINTERNAL;
  }
}

kvx_status kvx_write_files(const kvx_file_io* ops, int32_t n, int32_t io_depth) {
  try {
    return run_batch(ops, n, io_depth, true);
  } catch (...) {
    return KVX_EINTERNAL;
  }
}

}  // extern "C"
