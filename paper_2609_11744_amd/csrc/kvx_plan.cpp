// Piece planner for staged transfers: cut a packed image into pieces that fit
// one staging slot. Pure host code.
//
// A staging slot carries whole storage blocks (chunks), as many as fit (Sec.
// 6.4 uses one storage block per slot; packing several small ones per slot
// keeps each host-to-device copy large). A chunk larger than a slot is cut
// into contiguous layer ranges: with the layer-major chunk layout, the layers
// [a, b) of one chunk are one contiguous byte range and are themselves the
// packed image of that chunk's blocks over [a, b). Either way every piece is
// a plain scatter (layer range, block-table slice, chunk size) of the bytes it
// carries, and the pieces tile the image exactly once, in order.
#include <cstdint>
#include <vector>

#include "kvx.h"
#include "kvx_internal.h"

namespace kvx {

kvx_status plan_pieces(const Geometry& g, int32_t l0, int32_t l1, int32_t block_size,
                       int64_t slot_bytes, std::vector<kvx_piece>* out) {
  out->clear();
  if (slot_bytes <= 0) return KVX_EINVAL;
  if (g.n_units == 0) return KVX_OK;
  const int64_t unit_bytes = g.slab;                       // one (layer, K|V, block)
  const int64_t block_bytes = (int64_t)g.lr * 2 * unit_bytes;  // one block, all layers
  const int64_t bpc = g.bpc;
  const int64_t n = g.n_blocks;
  const int64_t nchunks = (n + bpc - 1) / bpc;
  const int64_t full_chunk = bpc * block_bytes;
  const int32_t ct = (int32_t)(bpc * block_size);
  if (full_chunk <= slot_bytes) {
    const int64_t per = slot_bytes / full_chunk;  // whole chunks per piece
    for (int64_t c0 = 0; c0 < nchunks; c0 += per) {
      const int64_t first = c0 * bpc;
      const int64_t last = (c0 + per) * bpc < n ? (c0 + per) * bpc : n;
      kvx_piece p{};
      p.src_offset = first * block_bytes;
      p.bytes = (last - first) * block_bytes;
      p.bt_first = (int32_t)first;
      p.n_blocks = (int32_t)(last - first);
      p.l_begin = l0;
      p.l_end = l1;
      p.chunk_tokens = ct;
      out->push_back(p);
    }
    return KVX_OK;
  }
  for (int64_t c = 0; c < nchunks; ++c) {
    const int64_t first = c * bpc;
    const int64_t nc = n - first < bpc ? n - first : bpc;
    const int64_t layer_bytes = nc * 2 * unit_bytes;  // one layer (K and V) of this chunk
    if (layer_bytes > slot_bytes) {
      out->clear();
      return KVX_EINVAL;
    }
    const int64_t per = slot_bytes / layer_bytes;  // layers per piece
    const int64_t chunk_off = first * block_bytes;
    for (int64_t a = l0; a < l1; a += per) {
      const int64_t b = a + per < l1 ? a + per : l1;
      kvx_piece p{};
      p.src_offset = chunk_off + (a - l0) * layer_bytes;
      p.bytes = (b - a) * layer_bytes;
      p.bt_first = (int32_t)first;
      p.n_blocks = (int32_t)nc;
      p.l_begin = (int32_t)a;
      p.l_end = (int32_t)b;
      p.chunk_tokens = ct;
      out->push_back(p);
    }
  }
  return KVX_OK;
}

}  // namespace kvx

extern "C" kvx_status kvx_plan_pieces(const kvx_cache* cache, int32_t l0, int32_t l1,
                                      int32_t n_blocks, int32_t chunk_tokens, int64_t slot_bytes,
                                      kvx_piece* out, int32_t max_pieces, int32_t* n_pieces) {
  try {
    if (!n_pieces) return KVX_EINVAL;
    *n_pieces = 0;
    kvx::Geometry g;
    kvx_status st = kvx::validate(cache, l0, l1, n_blocks, chunk_tokens, false, &g);
    if (st != KVX_OK) return st;
    std::vector<kvx_piece> v;
    st = kvx::plan_pieces(g, l0, l1, cache->block_size, slot_bytes, &v);
    if (st != KVX_OK) return st;
    if (v.size() > (size_t)INT32_MAX) return KVX_EINVAL;
    *n_pieces = (int32_t)v.size();
    if (out)
      for (int32_t i = 0; i < max_pieces && (size_t)i < v.size(); ++i) out[i] = v[i];
    return KVX_OK;
  } catch (...) {
    return KVX_EINTERNAL;
  }
}
