// Walk selection for the gather and scatter kernels (host code): how a call's
// work items are laid out over the chip's XCDs, whether a scatter visits its
// destinations in ascending order, and which slices move together. The launcher
// (kvx_kernels.hip) and kvx_copy_walk share it.
#include <cstdint>

#include "kvx.h"
#include "kvx_internal.h"

namespace kvx {

void slab_parts(int layout, uint32_t n16, uint32_t heads, uint32_t* parts, uint32_t* shift) {
  *parts = layout == KVX_LAYOUT_NHD ? (n16 + kPartThreads - 1) / kPartThreads : heads;
  *shift = (*parts & (*parts - 1)) == 0 ? (uint32_t)__builtin_ctz(*parts) : 32u;
}

namespace {

// Whether a large scatter of small slabs walks the image in order with no
// XCD ranges (workgroup b moves work item b: the whole chip reads the packed
// image front to back). Compared over 9-16 (cache, packed buffer) allocation
// pairs in one process at the tensor-parallel shard shapes of the 8B cache
// (80k prefix, 16-block chunks, default layout), against the destination-
// ordered walk: 4 KiB slabs 71.6-72.1 % of peak against 68.0-68.3 %, 8 KiB
// 70.8 against 69.3-69.8 %, 16 KiB level (73.7 / 73.6 %, a wider spread), and
// 32 KiB 71.1 against 75.3 % (image order with XCD ranges: 69.3 / 69.1 % at 4
// and 8 KiB). An HND cache with one KV head is the default layout byte for
// byte, and measured the same way (4 KiB slabs: 73.7 against 70.4 %); with
// two heads in 8 KiB it lost 1.8 points (1.4 on the current kernels, over 18
// pairs), so it keeps destination order. The paged-attention layout with one
// head takes the linear walk too, with its heads on 256 threads
// (kvx_kernels.hip): over 18 allocation pairs 73.2 % against 68.3 % for
// destination order on 128 threads, and about 1 point with either change
// alone; with two heads the linear walk lost 0.2 points.
bool scatter_linear(int64_t n_blocks, int64_t slab, int layout, int32_t heads) {
  const bool rows = layout == KVX_LAYOUT_NHD ||
                    ((layout == KVX_LAYOUT_HND || layout == KVX_LAYOUT_PAGED_ATTN) && heads == 1);
  return rows && n_blocks >= kOrderedScatterMinBlocks && slab <= 8192;
}

// Whether a scatter of n_blocks in chunks of bpc blocks runs in destination
// order. The rate of one walk over the same ids moves by up to 8 points of
// peak with where the cache and the packed buffer land in physical memory,
// so the walks were compared over 12 placements (4 caches x 3 packed buffers
// allocated in one process, each walk on each pair, alternated; 8B-shaped
// cache, 20,000-block pool, mean % of 8 TB/s). With one-block chunks image
// order averaged 76.8 against 73.6 in destination order at 2,048 blocks (at
// least as fast on 11 of the 12 pairs) and 76.3 against 76.1 at 5,000; with
// 4-block chunks the two were level (73.6 / 73.6), and destination order led
// with 16 and 64 (74.6 against 71.8 and 75.0 against 70.8 at 2,048 blocks,
// 76.9 against 71.9 at 5,000 with 16).
bool scatter_in_destination_order(int64_t n_blocks, int64_t bpc, int64_t slab, int layout,
                                  int32_t heads) {
  return n_blocks >= kOrderedScatterMinBlocks && bpc > 1 &&
         !scatter_linear(n_blocks, slab, layout, heads);
}

// Pairing for the ordered scatter of n_work work items (one launch) over
// n_slices layer|K|V slices: log2 of the distance D in slices between the two
// slices its fronts move together, or 32 for one front per XCD. Two fronts
// pay, as measured, where the paired slabs sit 2 MiB apart in the packed
// chunk (D chunk layers apart) and D <= 4: on the 80k scatter pattern
// (standalone probe, one allocation for the pool, two processes) pairs 2 MiB
// apart beat one front by 2.2-2.3 points with 16-block chunks (D = 4) and by
// 0.9-2.0 with 64-block chunks (D = 1), and lost 0.6-1.1 with 4-block chunks
// (D = 16); pairs at any other distance (32 KiB to 64 MiB) lost 0.5-2 points
// to one front in all but one process. In the library, alternated on three
// machines: the 80k scatter (D = 4) 75.1-75.6 % of peak against 72.7-72.9 %,
// 80.5-83.0 % against 78.9-80.5 % on two faster machines; the 32k scatter with
// 256-token chunks 72.6-72.8 % against 69.5-70.5 %. Why 2 MiB is the
// distance that pays is not established: it depends on how the chip maps
// physical addresses to memory channels, which these kernels do not see.
// log2 of D, the distance in slices at which two slices' runs in a packed
// chunk sit 2 MiB apart, where D is a power of two of at most 2^max_ds and
// the slice count a multiple of 2 D; else 32.
uint32_t pairing_2mib(uint32_t parts_shift, uint32_t n_slices, uint32_t bpc, uint64_t slab,
                      uint32_t max_ds) {
  constexpr uint64_t kPairBytes = 2u << 20;
  if (parts_shift >= 32) return 32;
  const uint64_t run = (uint64_t)bpc * slab;  // one slice's run in a chunk
  if (run == 0 || kPairBytes % run) return 32;
  const uint64_t d = kPairBytes / run;
  if ((d & (d - 1)) || d > (1ull << max_ds) || n_slices % (2 * d)) return 32;
  return (uint32_t)__builtin_ctzll(d);
}

// Farther apart (D = 8, 16) the fronts paid with slabs above 8 KiB, compared
// over 9-12 (cache, packed buffer) allocation pairs in one process: 32 KiB
// slabs in 8-block chunks (D = 8) 77.0 % of peak against 76.0 % for one front
// at 5,000 blocks and 74.6 against 73.8 % at 2,048, in 4-block chunks (D = 16)
// 76.6 against 76.0 % and 74.4 against 73.7 %; 16 KiB slabs in 16-block chunks
// (D = 8) 74.4 against 73.3 %. With 4 and 8 KiB slabs (D = 32, 16) they lost
// 1.3-1.4 points, so smaller slabs keep D <= 4.
uint32_t scatter_pairing(uint32_t n_work, uint32_t parts_shift, uint32_t n_slices, uint32_t bpc,
                         uint64_t slab) {
  if (n_work > kMaxWorkPerLaunch || n_slices % (2 * kXcds)) return 32;
  return pairing_2mib(parts_shift, n_slices, bpc, slab, slab > 8192 ? 4 : 2);
}

// Pairing for the gather: each chunk's slices walked in pairs 2 MiB apart in
// the chunk, D <= 32 slices (the packed-side writes then alternate between two
// runs 2 MiB apart). On the 80k gather pattern (standalone probe, two
// processes each) this measured 0.3-0.8 points above the plain walk with 16-
// and 64-block chunks (D = 4, 1); pairs at other distances (512 KiB to 32 MiB)
// were 0.5-4 points slower. Farther apart in slices, compared over 12 (cache,
// packed buffer) allocation pairs in one process (8B shape, 20,000-block
// pool; the rate of one walk moves by several points with where the
// allocations land): with 4- and 8-block chunks of 32 KiB slabs (D = 16, 8)
// 80.8 / 80.6 % of peak against 79.6 / 79.3 % for the plain walk at 2,048
// blocks, 81.2 / 81.1 against 80.7 / 80.5 at 5,000; at the tensor-parallel
// shard shapes (4 and 8 KiB slabs, 16-block chunks: D = 32, 16) 77.3 / 77.4
// against 75.5 / 75.6 over 16 pairs, faster on every pair.
uint32_t gather_pairing(uint32_t parts_shift, uint32_t n_slices, uint32_t bpc, uint64_t slab) {
  return pairing_2mib(parts_shift, n_slices, bpc, slab, 5);
}

}  // namespace

kvx_status choose_walk(bool to_packed, const kvx_cache* cache, const Geometry& g, Walk* w) {
  *w = Walk();
  if (g.n_units == 0) return KVX_OK;
  const uint32_t n16 = (uint32_t)(g.slab / 16);
  slab_parts(cache->layout, n16, (uint32_t)cache->num_kv_heads, &w->parts, &w->parts_shift);
  if ((uint64_t)g.n_units * w->parts > 0x7FFFFFFF) return KVX_EINTERNAL;
  w->n_work = (uint32_t)g.n_units * w->parts;
  const uint32_t n_slices = (uint32_t)(2 * g.lr);
  if (to_packed) {
    w->gather_pair_shift = gather_pairing(w->parts_shift, n_slices, (uint32_t)g.bpc,
                                          (uint64_t)g.slab);
    return KVX_OK;
  }
  w->linear = scatter_linear(g.n_blocks, g.slab, cache->layout, cache->num_kv_heads);
  w->ordered = scatter_in_destination_order(g.n_blocks, g.bpc, g.slab, cache->layout,
                                            cache->num_kv_heads);
  if (w->ordered)
    w->pair_shift = scatter_pairing(w->n_work, w->parts_shift, n_slices, (uint32_t)g.bpc,
                                    (uint64_t)g.slab);
  return KVX_OK;
}

}  // namespace kvx

// ---- the walk a copy takes -----------------------------------------------------

extern "C" kvx_status kvx_copy_walk(const kvx_cache* cache, int32_t l0, int32_t l1,
                                    int32_t n_blocks, int32_t chunk_tokens, int32_t to_packed,
                                    kvx_walk* out) {
  if (!out || (to_packed != 0 && to_packed != 1)) return KVX_EINVAL;
  try {
    *out = kvx_walk{};
    kvx::Geometry g;
    kvx_status st = kvx::validate(cache, l0, l1, n_blocks, chunk_tokens, false, &g);
    if (st != KVX_OK) return st;
    kvx::Walk w;
    st = kvx::choose_walk(to_packed == 1, cache, g, &w);
    if (st != KVX_OK || w.n_work == 0) return st;
    const uint32_t ps = to_packed ? w.gather_pair_shift : w.pair_shift;
    out->work_items = w.n_work;
    out->parts = (int32_t)w.parts;
    out->ordered = w.ordered ? 1 : 0;
    out->linear = w.linear ? 1 : 0;
    out->pair_slices = ps < 32 ? (int32_t)(1u << ps) : 0;
    out->fronts = w.ordered && w.pair_shift < 32 ? 2 : 1;
    return KVX_OK;
  } catch (...) {
    return KVX_EINTERNAL;
  }
}
