// Internal interfaces of libkvx.so shared by the C-ABI layer, the staging ring
// and the HIP kernels.
#pragma once

#include <stdint.h>

#include <vector>

#include "kvx.h"

namespace kvx {

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

// Host-side validation shared by every entry point. `packed` may be null only
// when no copy follows (plan-only callers). Fills *g on success.
kvx_status validate(const kvx_cache* cache, int32_t l0, int32_t l1, int32_t n_blocks,
                    int32_t chunk_tokens, bool need_pointers, Geometry* g);

// Reject a packed buffer that overlaps any cache tensor in [l0, l1).
bool overlaps_cache(const kvx_cache* cache, int32_t l0, int32_t l1, const void* packed,
                    int64_t bytes);

// Enqueue the gather (to_packed = true) or scatter kernel on `stream`.
// `block_table` is a device pointer to the call's n_blocks ids.
kvx_status launch_copy(bool to_packed, const kvx_cache* cache, int32_t l0, int32_t l1,
                       const int32_t* block_table, const Geometry& g, void* packed,
                       hipStream_t stream);

// Cut the image described by g (over layers [l0, l1)) into staging pieces of
// at most slot_bytes each (kvx_plan_pieces).
kvx_status plan_pieces(const Geometry& g, int32_t l0, int32_t l1, int32_t block_size,
                       int64_t slot_bytes, std::vector<kvx_piece>* out);

// Device address of the calling device's sticky error word (resolved once per
// device with hipGetSymbolAddress). Null on failure.
int* device_error_word();

}  // namespace kvx
