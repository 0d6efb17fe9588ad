// Internal interfaces of libkvx.so shared by the C-ABI layer, the staging ring
// and the HIP kernels.
#pragma once

#include <stdint.h>

#include <vector>

#include "kvx.h"

namespace kvx {

// Largest slab the LDS-staged (transposing) layouts accept: the padded image
// of a slab must fit the workgroup's LDS allocation.
constexpr int64_t kMaxTransposedSlab = 48 * 1024;

// Geometry of one gather / scatter call, validated on the host.
//
// Units: one unit is one slab (layer, K|V, block) of the image. Enumerating
// units chunk by chunk, then layer, then K|V, then block inside the chunk
// puts unit u at byte u * slab of the packed image, for full chunks and for
// the compact last chunk alike, so a kernel only needs the source-side
// indirection through the block table.
struct Geometry {
  int64_t slab = 0;          // bytes of one (layer, K|V, block)
  int64_t packed = 0;        // image bytes = n_units * slab
  int64_t n_units = 0;       // (l1 - l0) * 2 * n_blocks
  int32_t lr = 0;            // l1 - l0
  int32_t bpc = 0;           // blocks per chunk
  int32_t n_blocks = 0;
  int32_t num_blocks = 0;    // pool size, for the kernel's id check
};

// MI355X: 8 XCDs; a launch's workgroups are dispatched to them round-robin.
constexpr unsigned kXcds = 8;

// A dispatch's grid is counted in work-items in 32 bits, so one launch covers
// at most kMaxWorkPerLaunch workgroups (of at most 256 threads: 2^30
// work-items); larger calls are split.
constexpr uint32_t kMaxWorkPerLaunch = 1u << 22;

// Default-layout copy shape: one workgroup of kPartThreads threads moves
// kPartThreads 16-byte vectors of a slab.
constexpr uint32_t kPartThreads = 256;

// Scatters of at least this many blocks run in destination order.
constexpr int32_t kOrderedScatterMinBlocks = 1024;

// Workgroups per slab for the layout (4 KiB pieces with the default layout,
// heads with the reordering ones), and log2 of that count when it is a power
// of two (else 32: the kernels divide).
void slab_parts(int layout, uint32_t n16, uint32_t heads, uint32_t* parts, uint32_t* shift);

// How a gather or scatter walks its work items: the launcher's choice, also
// reported by kvx_copy_walk (kvx_walk.cpp).
struct Walk {
  uint32_t parts = 0, parts_shift = 32;  // workgroups per slab (slab_parts)
  uint32_t n_work = 0;                    // work items (workgroups) of the call
  uint32_t pair_shift = 32;               // ordered scatter: fronts 2^pair_shift slices apart
  uint32_t gather_pair_shift = 32;        // gather: slices paired 2^gather_pair_shift apart
  bool linear = false;                    // workgroup b moves work item b
  bool ordered = false;                   // scatter in destination order
};

// The walk of a validated gather (to_packed) or scatter: KVX_EINTERNAL when
// its work items do not fit 31 bits.
kvx_status choose_walk(bool to_packed, const kvx_cache* cache, const Geometry& g, Walk* w);


// Host-side validation shared by every entry point. `packed` may be null only
// when no copy follows (plan-only callers). Fills *g on success.
kvx_status validate(const kvx_cache* cache, int32_t l0, int32_t l1, int32_t n_blocks,
                    int32_t chunk_tokens, bool need_pointers, Geometry* g);

// Reject a packed buffer that overlaps any cache tensor in [l0, l1).
bool overlaps_cache(const kvx_cache* cache, int32_t l0, int32_t l1, const void* packed,
                    int64_t bytes);

// Enqueue the gather (to_packed = true) or scatter kernel on `stream`.
// `block_table` is a device pointer to the call's n_blocks ids; the kernels
// report bad ids in the error word err (stream_error_word). A scatter of at
// least 1,024 blocks first orders its destinations into n_blocks 8-byte
// entries: in order_scratch (device memory of the caller's) when given,
// otherwise in stream-ordered scratch allocated and freed on `stream`.
kvx_status launch_copy(bool to_packed, const kvx_cache* cache, int32_t l0, int32_t l1,
                       const int32_t* block_table, const Geometry& g, void* packed,
                       hipStream_t stream, int* err, void* order_scratch = nullptr);

// Bytes of the fixed device scratch of kvx_scatter_blocks_noalloc: one
// 8-byte order entry per block.
constexpr size_t kNoAllocScratchBytes = (size_t)KVX_NOALLOC_MAX_BLOCKS * 8;

// Enqueue the chunk-list gather (to_packed) or scatter on `stream`: refs is a
// device array of n_chunks references, validated by the kernel against
// table_len and packed_bytes. Host-checkable arguments must already be valid.
kvx_status launch_copy_chunks(bool to_packed, const kvx_cache* cache, int32_t l0, int32_t l1,
                              const int32_t* block_table, int32_t table_len,
                              const kvx_chunk_ref* refs, int32_t n_chunks, int32_t chunk_tokens,
                              void* packed, int64_t packed_bytes, hipStream_t stream,
                              int* err);

// A chunk image in host memory (restore source or offload destination) and the
// block-table slice it belongs to.
struct HostChunk {
  uint8_t* host;
  int32_t bt_offset;
  int32_t n_blocks;
};

// Host memory <-> staging-slot bytes [slot_off, slot_off + bytes).
struct Span {
  uint8_t* host;
  int64_t bytes;
  int64_t slot_off;
};

// One staging piece: a fused chunk-list copy over layers [l_begin, l_end) of
// the chunk references refs[ref_first, ref_first + ref_count) (packed offsets
// relative to the slot), filled from / drained to `spans`.
struct Piece {
  int32_t l_begin = 0, l_end = 0;
  int64_t bytes = 0;
  int32_t ref_first = 0, ref_count = 0;
  std::vector<Span> spans;
};

struct Plan {
  std::vector<Piece> pieces;
  std::vector<kvx_chunk_ref> refs;
  int32_t table_len = 0;  // block-table entries the chunks reference
};

// Where a plan's pieces ramp up to the slot size: nowhere, over the first
// pieces (the first at most 1/8 of a slot, each next at most twice the piece
// before it; a restore's first copy then starts after a small fill) or,
// mirrored, over the last pieces (an offload's last copy and drain are then
// short).
enum class Ramp { kNone, kFirst, kLast };

// Cut a chunk list into staging pieces of at most slot_bytes (see kvx_plan.cpp);
// a chunk larger than its piece's limit is cut into layer ranges.
kvx_status plan_chunks(const std::vector<HostChunk>& chunks, int32_t l0, int32_t l1, int64_t slab,
                       int32_t bpc, int64_t slot_bytes, Plan* out, Ramp ramp_at);

// The chunks of one contiguous packed image at `base` (geometry g).
std::vector<HostChunk> image_chunks(uint8_t* base, const Geometry& g);

// Device address of the sticky error word of `stream` on the calling device
// (a fixed table per device, resolved once with hipGetSymbolAddress; the null
// stream and streams beyond the table share its first word). Null on failure.
int* stream_error_word(hipStream_t stream);

}  // namespace kvx
