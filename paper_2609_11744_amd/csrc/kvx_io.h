// Storage-tier I/O engine of libkvx.so (host code): one thread submits and
// reaps many outstanding file reads and writes through io_uring, so the I/O
// depth, not a thread count, sets storage concurrency (Sec. 6.4). Files are
// opened with O_DIRECT where every transfer on them is 4 KiB aligned, so
// transfers do not depend on the page cache (Sec. 6.3). Pinned (page-locked,
// driver-mapped) host memory cannot be the target of a direct transfer on
// this platform (the kernel cannot pin its pages: EFAULT), so a file whose
// direct transfer fails that way is reopened without O_DIRECT and the
// transfer repeated; such buffered files keep the page cache out of the way
// instead: a written file is flushed (fdatasync, issued through the ring)
// before it is published, and a file's pages are dropped from the cache
// after they are read or published. A chunk file is
// published by writing a uniquely named temporary file in the target
// directory and hard-linking it to its final name: the link is atomic and
// fails if the name exists, so concurrent writers of one chunk are
// first-writer-wins and a reader of the final name sees a complete file or
// none (Sec. 6.3).
#pragma once

#include <stdint.h>

#include <string>
#include <vector>

#include "kvx.h"

namespace kvx {

// A file of the tier. For writes, `size` is the complete file size: the file
// is written under a temporary name and published once `size` bytes landed.
struct TierFile {
  std::string path;
  int64_t size = 0;
  bool direct = true;     // cleared when a transfer on it is not 4 KiB aligned or cannot be direct
  int fd = -1;
  std::string temp;       // writes: the temporary name while unpublished
  int64_t written = 0;    // writes: bytes landed so far
  bool flushing = false;  // writes: complete, its fdatasync queued or running
  bool published = false;
  std::vector<int> retired;  // descriptors replaced while transfers on them may be in flight
};

inline bool io_aligned(const void* buf, int64_t offset, int64_t bytes) {
  return (((uintptr_t)buf | (uint64_t)offset | (uint64_t)bytes) & 4095) == 0;
}

// Open a file for reading, or (write) create its temporary file next to the
// final name, making missing directories. KVX_EIO on failure.
kvx_status open_tier_file(TierFile* f, bool write);

// Publish a fully written file: link the temporary name to the final one (an
// existing final name means another writer published first, which is
// success), remove the temporary name, close.
kvx_status publish_tier_file(TierFile* f);

// Close; for an unpublished write also remove its temporary file.
void close_tier_file(TierFile* f);

// Tags with this bit set name an fdatasync (the rest of the tag: a file).
constexpr uint64_t kSyncTag = (uint64_t)1 << 63;

// Reads or writes (one direction per engine) with at most `depth` transfers
// in flight: io_uring over raw system calls, or one blocking pread / pwrite at
// a time where io_uring is unavailable. A short transfer is resubmitted for
// its remainder. Not thread-safe: one thread drives an engine.
class IoEngine {
 public:
  IoEngine() = default;
  // Waits (at most 30 s) for transfers a failure left in the kernel.
  ~IoEngine();
  IoEngine(const IoEngine&) = delete;
  IoEngine& operator=(const IoEngine&) = delete;

  // depth in [1, 256].
  kvx_status init(int32_t depth, bool write);
  bool uring() const { return ring_fd_ >= 0; }
  int32_t depth() const { return depth_; }
  int32_t inflight() const { return inflight_; }
  // Transfers not yet reported by wait(): in flight, or (without io_uring)
  // already finished inside start().
  int32_t pending() const { return inflight_ + (int32_t)finished_.size(); }

  // Start a transfer of [offset, offset + bytes) of open file f from / into
  // buf; `tag` is reported by wait() when all of its bytes are done.
  kvx_status start(TierFile* f, uint8_t* buf, int64_t offset, int64_t bytes, uint64_t tag);

  // Write engines: start an fdatasync of open file f; `tag` is reported when
  // it has finished.
  kvx_status start_datasync(TierFile* f, uint64_t tag);

  // Block until at least one started transfer has finished (returns at once
  // if some already have), then append the finished tags to *done. A failed
  // transfer (an I/O error, or end of file before its last byte) makes the
  // call return KVX_EIO, or, with `failed` given, appends its tag there and
  // counts as finished.
  kvx_status wait(std::vector<uint64_t>* done, std::vector<uint64_t>* failed = nullptr);

 private:
  struct Op {
    TierFile* f;
    uint8_t* buf;
    int64_t offset;
    int64_t left;     // bytes still to transfer; -1 for an fdatasync
    uint64_t tag;
    bool live;
    int fd;           // the descriptor its last submission used
  };
  int32_t take_slot();
  kvx_status submit(int32_t slot);
  bool enter(unsigned min_complete);
  void drain();

  bool write_ = false;
  int32_t depth_ = 0, inflight_ = 0;
  std::vector<Op> ops_;
  std::vector<uint64_t> finished_;  // synchronous mode: tags finished in start()
  // io_uring state
  int ring_fd_ = -1;
  unsigned sq_entries_ = 0, to_submit_ = 0;
  void* sq_map_ = nullptr;
  size_t sq_map_len_ = 0;
  void* cq_map_ = nullptr;
  size_t cq_map_len_ = 0;
  void* sqe_map_ = nullptr;
  size_t sqe_map_len_ = 0;
  unsigned *sq_tail_ = nullptr, *sq_mask_ = nullptr, *sq_array_ = nullptr;
  unsigned *cq_head_ = nullptr, *cq_tail_ = nullptr, *cq_mask_ = nullptr;
  void* sqes_ = nullptr;
  void* cqes_ = nullptr;
};

}  // namespace kvx
