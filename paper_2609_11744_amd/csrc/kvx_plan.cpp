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

namespace {

// What one piece carries, before its chunk references and host spans are
// built: the whole chunks [first, last) of the list over the call's layers,
// or layers [l_begin, l_end) of the single chunk `first`.
struct Group {
  int32_t first, last;
  int32_t l_begin, l_end;
};

// Cut the list into groups: as many consecutive whole chunks per piece as
// fit its size limit; a chunk larger than its piece's limit is cut into
// layer ranges, each as many layers as the piece it becomes allows (at
// least one). With the ramp, the first piece holds at most 1/8 of a slot and
// each next one at most twice the piece before it, until a piece's limit
// reaches the slot; from there on every piece may fill a slot. Doubling from
// the previous piece, not from a fixed 1/8, 1/4, 1/2 of a slot, keeps the
// short tail of a chunk cut into layer ranges from being followed by a whole
// slot, whose fill the tail's copy cannot hide. Measured on the 8B shape
// (4 x 64 MiB ring, one process, alternated with the fixed ramp): restores of
// 1k, 2k, 4k and 8k tokens 3.8, 1.1, 0.2 and 1.3 % faster, 80k level.
kvx_status plan_groups(const std::vector<HostChunk>& chunks, int32_t l0, int32_t l1, int64_t slab,
                       int64_t slot_bytes, bool ramp, std::vector<Group>* out) {
  const int64_t lr = l1 - l0;
  bool ramping = ramp;
  int64_t prev = 0;  // bytes of the last group
  auto cap = [&]() -> int64_t {
    if (!ramping) return slot_bytes;
    const int64_t first = slot_bytes >> 3;
    int64_t c = out->empty() ? first : std::max(first, 2 * prev);
    if (c <= 0 || c >= slot_bytes) {
      ramping = false;
      return slot_bytes;
    }
    return c;
  };
  auto push = [&](const Group& g, int64_t bytes) {
    out->push_back(g);
    prev = bytes;
  };
  bool open = false;
  int64_t cur_bytes = 0, cur_cap = 0;
  Group cur{};
  for (int32_t i = 0; i < (int32_t)chunks.size(); ++i) {
    const int64_t layer_bytes = (int64_t)chunks[(size_t)i].n_blocks * 2 * slab;  // K and V
    const int64_t chunk_bytes = lr * layer_bytes;
    if (open && cur_bytes + chunk_bytes <= cur_cap) {
      cur.last = i + 1;
      cur_bytes += chunk_bytes;
      continue;
    }
    if (open) push(cur, cur_bytes);
    open = false;
    if (chunk_bytes > cap()) {
      if (layer_bytes > slot_bytes) return KVX_EINVAL;
      for (int64_t a = l0; a < l1;) {
        const int64_t fit = cap() / layer_bytes;
        const int64_t b = std::min<int64_t>(a + (fit > 0 ? fit : 1), l1);
        push(Group{i, i + 1, (int32_t)a, (int32_t)b}, (b - a) * layer_bytes);
        a = b;
      }
      continue;
    }
    cur = Group{i, i + 1, l0, l1};
    cur_bytes = chunk_bytes;
    cur_cap = cap();
    open = true;
  }
  if (open) push(cur, cur_bytes);
  return KVX_OK;
}

}  // namespace

kvx_status plan_chunks(const std::vector<HostChunk>& chunks, int32_t l0, int32_t l1, int64_t slab,
                       int32_t bpc, int64_t slot_bytes, Plan* out, Ramp ramp_at) {
  out->pieces.clear();
  out->refs.clear();
  out->table_len = 0;
  if (slot_bytes <= 0 || slab <= 0 || bpc <= 0 || l1 < l0) return KVX_EINVAL;
  for (const HostChunk& c : chunks) {
    if (!c.host || c.n_blocks < 1 || c.n_blocks > bpc || c.bt_offset < 0) return KVX_EINVAL;
    const int64_t end = (int64_t)c.bt_offset + c.n_blocks;
    if (end > INT32_MAX) return KVX_EINVAL;
    if (end > out->table_len) out->table_len = (int32_t)end;
  }
  if (l1 == l0) return KVX_OK;
  std::vector<Group> groups;
  kvx_status st;
  if (ramp_at == Ramp::kLast) {
    // The same ramp at the end: cut the reversed list with the ramp first,
    // then map the groups back to the list's order (whole-chunk runs stay
    // runs of consecutive chunks) and reverse their order. Each piece is
    // then built in the list's own chunk order, so chunks adjacent in host
    // memory still merge into one copy.
    const std::vector<HostChunk> rev(chunks.rbegin(), chunks.rend());
    st = plan_groups(rev, l0, l1, slab, slot_bytes, true, &groups);
    const int32_t n = (int32_t)chunks.size();
    for (Group& g : groups) g = Group{n - g.last, n - g.first, g.l_begin, g.l_end};
    std::reverse(groups.begin(), groups.end());
  } else {
    st = plan_groups(chunks, l0, l1, slab, slot_bytes, ramp_at == Ramp::kFirst, &groups);
  }
  if (st != KVX_OK) {
    out->table_len = 0;
    return st;
  }
  for (const Group& g : groups) {
    Piece p{};
    p.l_begin = g.l_begin;
    p.l_end = g.l_end;
    p.ref_first = (int32_t)out->refs.size();
    for (int32_t i = g.first; i < g.last; ++i) {
      const HostChunk& c = chunks[(size_t)i];
      const int64_t layer_bytes = (int64_t)c.n_blocks * 2 * slab;
      const int64_t bytes = (int64_t)(g.l_end - g.l_begin) * layer_bytes;
      uint8_t* host = c.host + (int64_t)(g.l_begin - l0) * layer_bytes;
      out->refs.push_back(kvx_chunk_ref{p.bytes, c.bt_offset, c.n_blocks});
      ++p.ref_count;
      Span* last = p.spans.empty() ? nullptr : &p.spans.back();
      if (last && last->host + last->bytes == host)
        last->bytes += bytes;  // adjacent in host memory: one copy
      else
        p.spans.push_back(Span{host, bytes, p.bytes});
      p.bytes += bytes;
    }
    out->pieces.push_back(std::move(p));
  }
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
                                      int32_t ramp, kvx_piece* out, int32_t max_pieces,
                                      int32_t* n_pieces) {
  try {
    if (!n_pieces) return KVX_EINVAL;
    if (ramp != KVX_RAMP_NONE && ramp != KVX_RAMP_FIRST && ramp != KVX_RAMP_LAST) {
      *n_pieces = 0;
      return KVX_EINVAL;
    }
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
                          ramp == KVX_RAMP_FIRST  ? kvx::Ramp::kFirst
                          : ramp == KVX_RAMP_LAST ? kvx::Ramp::kLast
                                                  : kvx::Ramp::kNone);
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
      q.n_spans = (int32_t)p.spans.size();
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

// ---- step plan: the restore and offload chunk lists of one batched step ------
//
// Every chunk of every request is keyed by the hash of its last full block
// (Sec. 2.1: that hash covers the whole prefix through it, so a child that
// extends a parent's partial last chunk gets a different chunk). A chunk's
// residency is that of its first occurrence. The gate (Sec. 6.6) compares the
// tokens a request would load with the tier's threshold; a missing chunk is
// restored once, the first time a loading request needs it (Sec. 6.5), and
// recomputed for every request that needs it otherwise. New blocks are cut
// into chunks for the store path (Sec. 6.4).

namespace {

struct StepChunk {
  uint64_t key;
  int32_t request, chunk, n_blocks, first;  // first: index of the key's first occurrence
};

}  // namespace

extern "C" kvx_status kvx_plan_step(const kvx_step_request* reqs, int32_t n_requests,
                                    int32_t block_size, int32_t chunk_tokens, int64_t gate_tokens,
                                    kvx_step_plan* plan) {
  if (!plan || n_requests < 0 || (n_requests > 0 && !reqs) || block_size <= 0 ||
      chunk_tokens <= 0 || chunk_tokens % block_size != 0 || gate_tokens < 0)
    return KVX_EINVAL;
  try {
    const int32_t bpc = chunk_tokens / block_size;
    std::vector<StepChunk> ch;
    int64_t n_offload = 0;
    for (int32_t r = 0; r < n_requests; ++r) {
      const kvx_step_request& q = reqs[r];
      if (q.n_blocks < 0 || q.new_blocks < 0 || (q.n_blocks > 0 && !q.block_hashes)) return KVX_EINVAL;
      const int32_t nch = (int32_t)(((int64_t)q.n_blocks + bpc - 1) / bpc);
      if (q.n_resident != nch || (nch > 0 && !q.resident)) return KVX_EINVAL;
      for (int32_t k = 0; k < nch; ++k) {
        const int32_t first = k * bpc;
        const int32_t last = std::min(first + bpc, q.n_blocks) - 1;
        ch.push_back(StepChunk{q.block_hashes[last], r, k, last - first + 1, 0});
      }
      n_offload += ((int64_t)q.new_blocks + bpc - 1) / bpc;
    }
    if ((int64_t)ch.size() > INT32_MAX || n_offload > INT32_MAX) return KVX_EINVAL;
    std::unordered_map<uint64_t, int32_t> seen;
    seen.reserve(ch.size() * 2);
    for (size_t i = 0; i < ch.size(); ++i) ch[i].first = seen.emplace(ch[i].key, (int32_t)i).first->second;
    auto resident = [&](const StepChunk& c) {
      const StepChunk& f = ch[(size_t)c.first];
      return reqs[f.request].resident[f.chunk] != 0;
    };
    std::vector<int64_t> load((size_t)n_requests, 0);  // blocks each request would load
    for (const StepChunk& c : ch)
      if (!resident(c)) load[(size_t)c.request] += c.n_blocks;
    // a request with nothing to load counts as loading
    auto loads = [&](int32_t r) {
      return load[(size_t)r] == 0 || load[(size_t)r] * block_size >= gate_tokens;
    };
    // first pass: sizes and the restore order
    std::vector<int32_t> restore_of(ch.size(), -1);  // by first occurrence: restore index
    std::vector<int32_t> restore_src;                // restore index -> chunk that defines it
    int32_t hits = 0;
    for (size_t i = 0; i < ch.size(); ++i) {
      const StepChunk& c = ch[i];
      if (c.first == (int32_t)i && resident(c)) ++hits;
      if (resident(c) || restore_of[(size_t)c.first] >= 0 || !loads(c.request)) continue;
      restore_of[(size_t)c.first] = (int32_t)restore_src.size();
      restore_src.push_back((int32_t)i);
    }
    int32_t n_declined = 0;
    for (int32_t r = 0; r < n_requests; ++r)
      if (!loads(r)) ++n_declined;
    plan->n_restore = (int32_t)restore_src.size();
    plan->n_offload = (int32_t)n_offload;
    plan->n_chunk_states = (int32_t)ch.size();
    plan->n_declined = n_declined;
    plan->resident_hits = hits;
    plan->restore_blocks = 0;
    for (int32_t idx : restore_src) plan->restore_blocks += ch[(size_t)idx].n_blocks;
    plan->offload_blocks = 0;
    for (int32_t r = 0; r < n_requests; ++r) plan->offload_blocks += reqs[r].new_blocks;
    plan->recompute_blocks = 0;
    for (const StepChunk& c : ch)
      if (!resident(c) && restore_of[(size_t)c.first] < 0) plan->recompute_blocks += c.n_blocks;
    if (plan->restore_blocks > INT32_MAX || plan->offload_blocks > INT32_MAX) return KVX_EINVAL;
    // second pass: the lists, if the caller gave room for them
    if (!plan->restore && !plan->offload && !plan->chunk_states && !plan->declined) return KVX_OK;
    if (!plan->restore || !plan->offload || !plan->chunk_states || !plan->declined ||
        plan->restore_cap < plan->n_restore || plan->offload_cap < plan->n_offload ||
        plan->chunk_states_cap < plan->n_chunk_states || plan->declined_cap < plan->n_declined)
      return KVX_EINVAL;
    int32_t bt = 0;
    for (int32_t k = 0; k < plan->n_restore; ++k) {
      const StepChunk& c = ch[(size_t)restore_src[(size_t)k]];
      plan->restore[k] = kvx_step_restore{c.key, c.n_blocks, c.request, c.chunk, bt};
      bt += c.n_blocks;
    }
    for (size_t i = 0; i < ch.size(); ++i) {
      const StepChunk& c = ch[i];
      plan->chunk_states[i] = resident(c) ? KVX_CHUNK_RESIDENT
                              : restore_of[(size_t)c.first] >= 0 ? restore_of[(size_t)c.first]
                                                                   : KVX_CHUNK_RECOMPUTE;
    }
    int32_t o = 0, obt = 0;
    for (int32_t r = 0; r < n_requests; ++r)
      for (int32_t first = 0, k = 0; first < reqs[r].new_blocks; first += bpc, ++k) {
        const int32_t nb = std::min(bpc, reqs[r].new_blocks - first);
        plan->offload[o++] = kvx_step_offload{r, k, nb, obt, first};
        obt += nb;
      }
    int32_t d = 0;
    for (int32_t r = 0; r < n_requests; ++r)
      if (!loads(r)) plan->declined[d++] = r;
    return KVX_OK;
  } catch (...) {
    return KVX_ENOMEM;
  }
}
