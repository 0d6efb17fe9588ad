// Piece planner for staged transfers: cut a list of chunk images (each at its
// own host address) into pieces that fit one staging slot. Pure host code.
//
// A staging slot carries whole storage blocks (chunks), as many consecutive
// ones as fit (Sec. 6.4 uses one storage block per slot; packing several
// small ones into a slot keeps each host<->device copy large). A chunk larger
// than a slot is cut into contiguous layer ranges: with the layer-major chunk
// layout, layers [a, b) of one chunk are one contiguous byte range and are
// themselves that chunk's image over [a, b). Every piece is one fused
// chunk-list copy (one launch) of the chunk references it carries, at
// slot-relative offsets, over its layer range.
#include <algorithm>
#include <cstdint>
#include <unordered_map>
#include <vector>

#include "kvx.h"
#include "kvx_internal.h"

namespace kvx {

kvx_status plan_chunks(const std::vector<HostChunk>& chunks, int32_t l0, int32_t l1, int64_t slab,
                       int32_t bpc, int64_t slot_bytes, Plan* out, Ramp ramp_at) {
  if (ramp_at == Ramp::kLast) {
    // The same ramp at the end: plan the chunks in reverse order with the ramp
    // first, then reverse the pieces. Each piece carries its own chunk
    // references and host spans, so the pieces keep their meaning in any order.
    const std::vector<HostChunk> rev(chunks.rbegin(), chunks.rend());
    const kvx_status st = plan_chunks(rev, l0, l1, slab, bpc, slot_bytes, out, Ramp::kFirst);
    if (st == KVX_OK) std::reverse(out->pieces.begin(), out->pieces.end());
    return st;
  }
  const bool ramp = ramp_at == Ramp::kFirst;
  out->pieces.clear();
  out->refs.clear();
  out->table_len = 0;
  if (slot_bytes <= 0 || slab <= 0 || bpc <= 0 || l1 < l0) return KVX_EINVAL;
  if (l1 == l0) return KVX_OK;
  const int64_t lr = l1 - l0;
  // Size limit of the next piece: the slot, or with the ramp 1/8, 1/4 and
  // 1/2 of it for the first three pieces.
  auto cap = [&]() -> int64_t {
    const size_t k = out->pieces.size();
    if (!ramp || k >= 3) return slot_bytes;
    const int64_t c = slot_bytes >> (3 - k);
    return c > 0 ? c : slot_bytes;
  };
  Piece cur{};
  int64_t cur_cap = 0;
  bool open = false;
  auto flush = [&]() {
    if (open) out->pieces.push_back(cur);
    open = false;
  };
  for (const HostChunk& c : chunks) {
    if (!c.host || c.n_blocks < 1 || c.n_blocks > bpc || c.bt_offset < 0) return KVX_EINVAL;
    const int64_t end = (int64_t)c.bt_offset + c.n_blocks;
    if (end > INT32_MAX) return KVX_EINVAL;
    if (end > out->table_len) out->table_len = (int32_t)end;
    const int64_t layer_bytes = (int64_t)c.n_blocks * 2 * slab;  // one layer, K and V
    const int64_t chunk_bytes = lr * layer_bytes;
    if (!(open && cur.bytes + chunk_bytes <= cur_cap)) {
      flush();
      if (chunk_bytes > cap()) {
        // Too large for the next piece: contiguous layer ranges, each as many
        // layers as the piece it becomes allows (at least one).
        if (layer_bytes > slot_bytes) {
          out->pieces.clear();
          out->refs.clear();
          return KVX_EINVAL;
        }
        for (int64_t a = l0; a < l1;) {
          const int64_t fit = cap() / layer_bytes;
          const int64_t per = fit > 0 ? fit : 1;
          const int64_t b = a + per < l1 ? a + per : l1;
          Piece p{};
          p.l_begin = (int32_t)a;
          p.l_end = (int32_t)b;
          p.bytes = (b - a) * layer_bytes;
          p.ref_first = (int32_t)out->refs.size();
          p.ref_count = 1;
          p.spans.push_back(Span{c.host + (a - l0) * layer_bytes, p.bytes, 0});
          out->refs.push_back(kvx_chunk_ref{0, c.bt_offset, c.n_blocks});
          out->pieces.push_back(p);
          a = b;
        }
        continue;
      }
      cur = Piece{};
      cur.l_begin = l0;
      cur.l_end = l1;
      cur.ref_first = (int32_t)out->refs.size();
      cur_cap = cap();
      open = true;
    }
    out->refs.push_back(kvx_chunk_ref{cur.bytes, c.bt_offset, c.n_blocks});
    ++cur.ref_count;
    Span* last = cur.spans.empty() ? nullptr : &cur.spans.back();
    if (last && last->host + last->bytes == c.host)
      last->bytes += chunk_bytes;  // adjacent in host memory: one copy
    else
      cur.spans.push_back(Span{c.host, chunk_bytes, cur.bytes});
    cur.bytes += chunk_bytes;
  }
  flush();
  return KVX_OK;
}

std::vector<HostChunk> image_chunks(uint8_t* base, const Geometry& g) {
  std::vector<HostChunk> v;
  const int64_t block_bytes = (int64_t)g.lr * 2 * g.slab;
  for (int64_t first = 0; first < g.n_blocks; first += g.bpc) {
    const int64_t nc = g.n_blocks - first < g.bpc ? g.n_blocks - first : g.bpc;
    v.push_back(HostChunk{base + first * block_bytes, (int32_t)first, (int32_t)nc});
  }
  return v;
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
    if (g.n_units == 0) return KVX_OK;
    // Plan over a notional image at address 4096 (never dereferenced), then
    // report each piece as (image offset, bytes, block-table slice, layers).
    uint8_t* const base = reinterpret_cast<uint8_t*>(4096);
    kvx::Plan plan;
    st = kvx::plan_chunks(kvx::image_chunks(base, g), l0, l1, g.slab, g.bpc, slot_bytes, &plan,
                          kvx::Ramp::kNone);
    if (st != KVX_OK) return st;
    if (plan.pieces.size() > (size_t)INT32_MAX) return KVX_EINVAL;
    *n_pieces = (int32_t)plan.pieces.size();
    for (int32_t i = 0; out && i < max_pieces && (size_t)i < plan.pieces.size(); ++i) {
      const kvx::Piece& p = plan.pieces[(size_t)i];
      kvx_piece q{};
      q.src_offset = p.spans.front().host - base;
      q.bytes = p.bytes;
      q.bt_first = plan.refs[(size_t)p.ref_first].bt_offset;
      for (int32_t r = 0; r < p.ref_count; ++r) q.n_blocks += plan.refs[(size_t)(p.ref_first + r)].n_blocks;
      q.l_begin = p.l_begin;
      q.l_end = p.l_end;
      q.chunk_tokens = g.bpc * cache->block_size;
      out[i] = q;
    }
    return KVX_OK;
  } catch (...) {
    return KVX_EINTERNAL;
  }
}

// ---- step planning: prefix-hash chain and chunk dedupe ------------------------
//
// Sec. 2.1: the engine hashes each full token block together with the hash of
// the block before it, so a block's hash identifies the whole token prefix up
// to its end; lookup walks blocks until the first mismatch, and a trailing
// partial block is never cached. Sec. 6.5: identical prefixes requested by
// several requests share one read and one staging slot, so a step restores
// each distinct chunk once.

namespace {

uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

}  // namespace

extern "C" int64_t kvx_block_hashes(const int32_t* tokens, int64_t n_tokens, int32_t block_size,
                                    uint64_t parent_hash, uint64_t* out) {
  if (n_tokens < 0 || block_size <= 0 || (n_tokens > 0 && !tokens)) return -1;
  const int64_t n_blocks = n_tokens / block_size;
  if (n_blocks > 0 && !out) return -1;
  uint64_t h = parent_hash;
  for (int64_t b = 0; b < n_blocks; ++b) {
    uint64_t x = mix64(h ^ 0x6A09E667F3BCC908ULL);
    for (int32_t i = 0; i < block_size; ++i)
      x = mix64(x + (uint64_t)(uint32_t)tokens[b * block_size + i] +
                0x9E3779B97F4A7C15ULL * (uint64_t)(i + 1));
    h = x;
    out[b] = h;
  }
  return n_blocks;
}

extern "C" kvx_status kvx_dedupe_keys(const uint64_t* keys, int32_t n, int32_t* first_of) {
  if (n < 0 || (n > 0 && (!keys || !first_of))) return KVX_EINVAL;
  try {
    std::unordered_map<uint64_t, int32_t> seen;
    seen.reserve((size_t)n * 2);
    for (int32_t i = 0; i < n; ++i) first_of[i] = seen.emplace(keys[i], i).first->second;
    return KVX_OK;
  } catch (...) {
    return KVX_ENOMEM;
  }
}
