// HIP kernels for gfx950: paged-KV gather (paged slabs -> packed image) and
// scatter (packed image -> paged slabs).
//
// The work is pure data movement, bound by HBM bandwidth, so the kernels use
// no MFMA. With the default cache layout every slab is contiguous and in the
// same order on both sides, so nothing is transposed and no LDS is used; the
// other cache layouts stage each slab through LDS (see move_slab_transposed).
// One workgroup moves one unit, a whole slab (layer, K|V, block) of `slab`
// bytes:
//   * the unit's decode (chunk, layer, K|V, block) and its block-table read
//     depend on blockIdx only, so they run on the scalar unit once per
//     workgroup;
//   * the slab moves as 16-byte vectors, consecutive lanes on consecutive
//     addresses, so every wave instruction reads or writes 1 KiB contiguous;
//   * each thread issues all of its loads before its stores, so a workgroup
//     has its whole slab in flight (32 KiB slabs: 1024 threads x 2 vectors);
//   * both streams are touched once, so loads and stores are non-temporal;
//   * workgroups are dispatched round-robin over the 8 XCDs, so workgroup b
//     is mapped to a unit such that each XCD walks one contiguous range of
//     units. The packed side of an XCD's work is then one sequential stream,
//     which HBM serves measurably better than 8 interleaved ones (the write
//     side of a copy is what bounds it).
// The packed-side address of unit u is u * slab (see Geometry), so only the
// paged side goes through the block table.
//
// Large scatters write to caller-chosen (typically random) blocks. HBM takes
// writes faster when each XCD's write stream ascends through memory, so a
// large scatter first buckets the destination ids (order_kernel, into
// stream-ordered scratch) and then visits units layer by layer in ascending
// destination order; the packed side is then read out of order, which costs
// less than unordered writes.
#include <hip/hip_runtime.h>

#include <mutex>

#include "kvx_internal.h"

namespace kvx {
namespace {

typedef unsigned int v4u __attribute__((ext_vector_type(4)));

constexpr int kErrBadBlock = 1;
constexpr int kErrBadChunk = 2;
constexpr unsigned kXcds = 8;  // MI355X: 8 XCDs, workgroups dispatched round-robin

// Device pointers of the call's layers, in image order: p[2 * (l - l0) + kv].
// Passed by value as a kernel argument (2 KiB for KVX_MAX_LAYERS = 128).
struct LayerPtrs {
  char* p[2 * KVX_MAX_LAYERS];
};

// Shape of one slab, for the transposing layouts.
struct SlabGeom {
  uint32_t bs;   // tokens per block
  uint32_t h;    // KV heads
  uint32_t d;    // head dim (elements)
  uint32_t v16;  // 16-byte vectors per (token, head) row: d * elem_bytes / 16
  uint32_t x;    // elements per 16-byte vector: 16 / elem_bytes
  uint32_t pad;
};

struct UnitGeom {
  uint32_t units_per_chunk;  // (l1 - l0) * 2 * bpc
  uint32_t bpc;
  uint32_t n_blocks;
  uint32_t num_blocks;       // pool size
  uint32_t n16;              // 16-byte vectors per slab
  uint32_t pad;
  uint64_t slab;
  SlabGeom sg;
};

// Sticky error word, one per device. Host code reaches it only through the
// address that hipGetSymbolAddress returns (device_error_word()).
__device__ int g_error_word;

// Workgroup b of a launch over n units -> unit index. XCD x = b % kXcds runs
// the workgroups b = x, x + kXcds, ...; they get the contiguous range
// [x*q + min(x, r), ...) of q or q + 1 units (q = n / kXcds, r = n % kXcds).
// A bijection on [0, n) for every n.
__device__ __forceinline__ uint32_t xcd_contiguous(uint32_t b, uint32_t n) {
  const uint32_t q = n / kXcds, r = n % kXcds, x = b % kXcds, k = b / kXcds;
  return x * q + (x < r ? x : r) + k;
}

template <int T, int V>
__device__ __forceinline__ void move_slab(const v4u* __restrict__ s, v4u* __restrict__ d,
                                          uint32_t n16) {
  uint32_t i = threadIdx.x;
  // Main body: V vectors per thread per pass, loads first.
  for (; i + (V - 1) * T < n16; i += V * T) {
    v4u r[V];
#pragma unroll
    for (int q = 0; q < V; ++q) r[q] = __builtin_nontemporal_load(s + i + q * T);
#pragma unroll
    for (int q = 0; q < V; ++q) __builtin_nontemporal_store(r[q], d + i + q * T);
  }
  for (; i < n16; i += T) __builtin_nontemporal_store(__builtin_nontemporal_load(s + i), d + i);
}

// ---- cache layouts that reorder a slab ---------------------------------------
//
// The packed side is always [token][head][dim]. The cache side may be
//   KVX_LAYOUT_HND         [head][token][dim] rows (K and V);
//   KVX_LAYOUT_PAGED_ATTN  K [head][dim / x][token][x] (x = 16 / elem_bytes: the
//                          16-byte vectors of a row are re-strided), V
//                          [head][dim][token] (an element transpose).
// Such a slab is staged through LDS: the workgroup loads it in source order
// (16-byte vectors, consecutive lanes on consecutive addresses), then writes
// it in destination order, each lane fetching what its output vector needs
// from LDS. Both global sides stay coalesced; only LDS sees the transpose.
// One pad vector after every 16 spreads strided LDS reads over the banks.

extern __shared__ __attribute__((aligned(16))) unsigned char kvx_lds[];

__device__ __forceinline__ uint32_t lds_slot(uint32_t v) { return v + (v >> 4); }

// Source vector index of destination vector w for a vector permutation
// (HND K/V, paged-attention K). Gather: destination = packed, source = cache.
template <bool kToPacked, int kLayout>
__device__ __forceinline__ uint32_t src_vector(uint32_t w, const SlabGeom& g) {
  uint32_t t, h, dv;
  if (kToPacked) {  // w = (t * h + hh) * v16 + dv in packed order
    dv = w % g.v16;
    const uint32_t th = w / g.v16;
    h = th % g.h;
    t = th / g.h;
    return kLayout == KVX_LAYOUT_HND ? (h * g.bs + t) * g.v16 + dv : (h * g.v16 + dv) * g.bs + t;
  }
  if (kLayout == KVX_LAYOUT_HND) {  // w = (h * bs + t) * v16 + dv in cache order
    dv = w % g.v16;
    const uint32_t r = w / g.v16;
    t = r % g.bs;
    h = r / g.bs;
  } else {  // w = (h * v16 + dv) * bs + t in cache order
    t = w % g.bs;
    const uint32_t r = w / g.bs;
    dv = r % g.v16;
    h = r / g.v16;
  }
  return (t * g.h + h) * g.v16 + dv;
}

// Destination vector w of a paged-attention V slab move, assembled element by
// element from the LDS image of the source (Elem = the element type).
template <bool kToPacked, typename Elem>
__device__ __forceinline__ v4u gather_elements(uint32_t w, const SlabGeom& g) {
  constexpr uint32_t kX = 16 / sizeof(Elem);
  Elem out[kX];
#pragma unroll
  for (uint32_t i = 0; i < kX; ++i) {
    const uint32_t e = w * kX + i;
    uint32_t se;
    if (kToPacked) {  // packed element (t, h, d) <- cache element (h, d, t)
      const uint32_t d = e % g.d, th = e / g.d, h = th % g.h, t = th / g.h;
      se = (h * g.d + d) * g.bs + t;
    } else {          // cache element (h, d, t) <- packed element (t, h, d)
      const uint32_t t = e % g.bs, r = e / g.bs, d = r % g.d, h = r / g.d;
      se = (t * g.h + h) * g.d + d;
    }
    const uint32_t v = se / kX, lane = se % kX;
    out[i] = reinterpret_cast<const Elem*>(kvx_lds + 16u * lds_slot(v))[lane];
  }
  return __builtin_bit_cast(v4u, out);
}

template <bool kToPacked, int kLayout, int kElem, int T>
__device__ __forceinline__ void move_slab_transposed(const v4u* __restrict__ src,
                                                     v4u* __restrict__ dst, uint32_t n16,
                                                     const SlabGeom& g, uint32_t kv) {
  v4u* lds = reinterpret_cast<v4u*>(kvx_lds);
  for (uint32_t v = threadIdx.x; v < n16; v += T) lds[lds_slot(v)] = __builtin_nontemporal_load(src + v);
  __syncthreads();
  if (kLayout == KVX_LAYOUT_PAGED_ATTN && kv == 1) {
    for (uint32_t w = threadIdx.x; w < n16; w += T) {
      v4u val;
      if (kElem == 1) val = gather_elements<kToPacked, uint8_t>(w, g);
      else if (kElem == 2) val = gather_elements<kToPacked, uint16_t>(w, g);
      else if (kElem == 4) val = gather_elements<kToPacked, uint32_t>(w, g);
      else val = gather_elements<kToPacked, uint64_t>(w, g);
      __builtin_nontemporal_store(val, dst + w);
    }
  } else {
    for (uint32_t w = threadIdx.x; w < n16; w += T)
      __builtin_nontemporal_store(lds[lds_slot(src_vector<kToPacked, kLayout>(w, g))], dst + w);
  }
}

// Move one slab in the direction and layout of the kernel.
template <bool kToPacked, int kLayout, int kElem, int T, int V>
__device__ __forceinline__ void move_unit(char* paged, char* pk, uint32_t n16, const SlabGeom& g,
                                          uint32_t kv) {
  const v4u* s = reinterpret_cast<const v4u*>(kToPacked ? paged : pk);
  v4u* d = reinterpret_cast<v4u*>(kToPacked ? pk : paged);
  if (kLayout == KVX_LAYOUT_NHD)
    move_slab<T, V>(s, d, n16);
  else
    move_slab_transposed<kToPacked, kLayout, kElem, T>(s, d, n16, g, kv);
}

// kOrdered = false: units in image order (u -> chunk, layer|K|V, block).
// kOrdered = true: unit v -> lk = v / n_blocks, k = v % n_blocks, block index
// i = order[k] (destinations ascending by bucket); the image position u of
// (chunk i / bpc, lk, block i % bpc) follows.
template <bool kToPacked, bool kOrdered, int kLayout, int kElem, int T, int V>
__global__ void __launch_bounds__(T)
    copy_units_kernel(LayerPtrs layers, const int32_t* __restrict__ block_table, UnitGeom g,
                      uint32_t unit_base, uint32_t unit_count,
                      const uint32_t* __restrict__ order, char* __restrict__ packed,
                      int* __restrict__ err) {
  uint32_t u = unit_base + xcd_contiguous(blockIdx.x, unit_count);
  uint32_t c, first, nc, lk, j;
  if (kOrdered) {
    lk = u / g.n_blocks;
    const uint32_t i = order[u - lk * g.n_blocks];  // < n_blocks (a permutation)
    c = i / g.bpc;
    first = c * g.bpc;
    j = i - first;
    const uint32_t left = g.n_blocks - first;
    nc = left < g.bpc ? left : g.bpc;
    u = c * g.units_per_chunk + lk * nc + j;
  } else {
    c = u / g.units_per_chunk;
    const uint32_t r = u - c * g.units_per_chunk;
    first = c * g.bpc;
    const uint32_t left = g.n_blocks - first;
    nc = left < g.bpc ? left : g.bpc;  // blocks in this chunk
    lk = r / nc;                       // 2 * (l - l0) + kv
    j = r - lk * nc;
  }
  const int32_t id = block_table[first + j];
  if ((uint32_t)id >= g.num_blocks) {
    if (threadIdx.x == 0) atomicOr(err, kErrBadBlock);
    return;
  }
  char* paged = layers.p[lk] + (uint64_t)(uint32_t)id * g.slab;
  char* pk = packed + (uint64_t)u * g.slab;
  move_unit<kToPacked, kLayout, kElem, T, V>(paged, pk, g.n16, g.sg, lk & 1);
}

// Chunk-list copy: a batch of chunks, each with its own block-table slice and
// its own place in the packed buffer (the fused block copy of several
// requests' chunks in one launch). Unit space is padded: chunk c owns units
// [c * upc, (c + 1) * upc) with upc = (l1 - l0) * 2 * bpc, unit r of a chunk
// is (lk = r / bpc, j = r % bpc), and units with j >= the chunk's n_blocks
// exit at once. So a workgroup finds its chunk by one division, with no
// search. Each reference is validated here (it lives in device memory): a bad
// one sets kErrBadChunk and its units are skipped.
struct ChunkGeom {
  uint32_t upc;          // (l1 - l0) * 2 * bpc
  uint32_t bpc;
  uint32_t lr2;          // (l1 - l0) * 2
  uint32_t num_blocks;   // pool size
  uint32_t n16;
  int32_t table_len;
  uint64_t slab;
  int64_t packed_bytes;
  SlabGeom sg;
};

template <bool kToPacked, int kLayout, int kElem, int T, int V>
__global__ void __launch_bounds__(T)
    copy_chunks_kernel(LayerPtrs layers, const int32_t* __restrict__ block_table,
                       const kvx_chunk_ref* __restrict__ refs, ChunkGeom g, uint32_t unit_base,
                       uint32_t unit_count, char* __restrict__ packed, int* __restrict__ err) {
  const uint32_t u = unit_base + xcd_contiguous(blockIdx.x, unit_count);
  const uint32_t c = u / g.upc;
  const uint32_t r = u - c * g.upc;
  const uint32_t lk = r / g.bpc;
  const uint32_t j = r - lk * g.bpc;
  const kvx_chunk_ref ref = refs[c];
  const bool ok = ref.n_blocks >= 1 && (uint32_t)ref.n_blocks <= g.bpc && ref.bt_offset >= 0 &&
                  (int64_t)ref.bt_offset + ref.n_blocks <= (int64_t)g.table_len &&
                  ref.packed_offset >= 0 && (ref.packed_offset & 15) == 0 &&
                  ref.packed_offset + (int64_t)g.lr2 * ref.n_blocks * (int64_t)g.slab <=
                      g.packed_bytes;
  if (!ok) {
    if (r == 0 && threadIdx.x == 0) atomicOr(err, kErrBadChunk);
    return;
  }
  const uint32_t nc = (uint32_t)ref.n_blocks;
  if (j >= nc) return;  // padding unit
  const int32_t id = block_table[ref.bt_offset + j];
  if ((uint32_t)id >= g.num_blocks) {
    if (threadIdx.x == 0) atomicOr(err, kErrBadBlock);
    return;
  }
  char* paged = layers.p[lk] + (uint64_t)(uint32_t)id * g.slab;
  char* pk = packed + ref.packed_offset + (uint64_t)(lk * nc + j) * g.slab;
  move_unit<kToPacked, kLayout, kElem, T, V>(paged, pk, g.n16, g.sg, lk & 1);
}

// Destination order for a scatter: order[] lists the block-table indexes
// bucketed by destination id, buckets ascending. The id range [0, num_blocks)
// is cut into kBins equal bins (ids outside it go to the last bin; the copy
// kernel skips them). One workgroup counts bin sizes in LDS, scans them into
// bin starts and places each index with an LDS atomic, so order[] is a
// permutation of [0, n) for any table (within a bin the order is
// unspecified, which only matters if destinations repeat, and a scatter's
// destinations must be distinct).
constexpr int kOrderThreads = 1024;
constexpr uint32_t kBins = 4096;  // 4 bins per thread

__device__ __forceinline__ uint32_t bin_of(int32_t id, uint32_t num_blocks, uint32_t bins) {
  const uint32_t u = (uint32_t)id;
  return u >= num_blocks ? bins - 1 : (uint32_t)(((uint64_t)u * bins) / num_blocks);
}

__global__ void __launch_bounds__(kOrderThreads)
    order_kernel(const int32_t* __restrict__ block_table, uint32_t n, uint32_t num_blocks,
                 uint32_t* __restrict__ order) {
  __shared__ uint32_t cnt[kBins];
  __shared__ uint32_t wave_total[kOrderThreads / 64];
  const uint32_t t = threadIdx.x, lane = t % 64, wave = t / 64;
  const uint32_t bins = num_blocks < kBins ? num_blocks : kBins;
  for (uint32_t b = t; b < kBins; b += kOrderThreads) cnt[b] = 0;
  __syncthreads();
  for (uint32_t i = t; i < n; i += kOrderThreads)
    atomicAdd(&cnt[bin_of(block_table[i], num_blocks, bins)], 1u);
  __syncthreads();
  // exclusive scan of the kBins counts: 4 per thread, then waves, then workgroup
  const uint32_t c0 = cnt[4 * t], c1 = cnt[4 * t + 1], c2 = cnt[4 * t + 2], c3 = cnt[4 * t + 3];
  const uint32_t mine = c0 + c1 + c2 + c3;
  uint32_t incl = mine;
  for (uint32_t off = 1; off < 64; off <<= 1) {
    const uint32_t y = __shfl_up(incl, off, 64);
    if (lane >= off) incl += y;
  }
  if (lane == 63) wave_total[wave] = incl;
  __syncthreads();
  if (wave == 0) {
    uint32_t w = lane < kOrderThreads / 64 ? wave_total[lane] : 0;
    for (uint32_t off = 1; off < kOrderThreads / 64; off <<= 1) {
      const uint32_t y = __shfl_up(w, off, 64);
      if (lane >= off) w += y;
    }
    if (lane < kOrderThreads / 64) wave_total[lane] = w;  // inclusive over waves
  }
  __syncthreads();
  const uint32_t base = (wave > 0 ? wave_total[wave - 1] : 0u) + incl - mine;
  cnt[4 * t] = base;
  cnt[4 * t + 1] = base + c0;
  cnt[4 * t + 2] = base + c0 + c1;
  cnt[4 * t + 3] = base + c0 + c1 + c2;
  __syncthreads();
  for (uint32_t i = t; i < n; i += kOrderThreads)
    order[atomicAdd(&cnt[bin_of(block_table[i], num_blocks, bins)], 1u)] = i;
}

// A dispatch's grid is counted in work-items in 32 bits, so one launch covers
// at most kMaxUnitsPerLaunch workgroups; larger calls are split.
constexpr uint32_t kMaxUnitsPerLaunch = 1u << 22;

// Scatters of at least this many blocks run in destination order.
constexpr int32_t kOrderedScatterMinBlocks = 1024;

// Dynamic LDS bytes for a transposing layout: the padded slab image.
inline size_t lds_bytes(uint32_t n16) { return 16u * (size_t)(n16 + n16 / 16 + 1); }

// Launch `cnt` workgroups of kernel K<..., layout, elem, T, V> for the slab
// shape: the default layout picks the copy shape by slab size; the others use
// 256 threads and the LDS-staged mover.
#define KVX_DISPATCH(KERNEL, PREFIX, ...)                                                      \
  do {                                                                                     \
    if (layout == KVX_LAYOUT_NHD) {                                                        \
      if (n16 % (2 * 1024) == 0)                                                           \
        hipLaunchKernelGGL((KERNEL<PREFIX, KVX_LAYOUT_NHD, 0, 1024, 2>), grid, dim3(1024), 0, \
                           stream, __VA_ARGS__);                                           \
      else if (n16 % (4 * 256) == 0)                                                       \
        hipLaunchKernelGGL((KERNEL<PREFIX, KVX_LAYOUT_NHD, 0, 256, 4>), grid, dim3(256), 0,   \
                           stream, __VA_ARGS__);                                           \
      else                                                                                 \
        hipLaunchKernelGGL((KERNEL<PREFIX, KVX_LAYOUT_NHD, 0, 256, 1>), grid, dim3(256), 0,   \
                           stream, __VA_ARGS__);                                           \
    } else if (layout == KVX_LAYOUT_HND) {                                                 \
      hipLaunchKernelGGL((KERNEL<PREFIX, KVX_LAYOUT_HND, 0, 256, 1>), grid, dim3(256),        \
                         lds_bytes(n16), stream, __VA_ARGS__);                             \
    } else if (elem == 1) {                                                                \
      hipLaunchKernelGGL((KERNEL<PREFIX, KVX_LAYOUT_PAGED_ATTN, 1, 256, 1>), grid, dim3(256), \
                         lds_bytes(n16), stream, __VA_ARGS__);                             \
    } else if (elem == 2) {                                                                \
      hipLaunchKernelGGL((KERNEL<PREFIX, KVX_LAYOUT_PAGED_ATTN, 2, 256, 1>), grid, dim3(256), \
                         lds_bytes(n16), stream, __VA_ARGS__);                             \
    } else if (elem == 4) {                                                                \
      hipLaunchKernelGGL((KERNEL<PREFIX, KVX_LAYOUT_PAGED_ATTN, 4, 256, 1>), grid, dim3(256), \
                         lds_bytes(n16), stream, __VA_ARGS__);                             \
    } else {                                                                               \
      hipLaunchKernelGGL((KERNEL<PREFIX, KVX_LAYOUT_PAGED_ATTN, 8, 256, 1>), grid, dim3(256), \
                         lds_bytes(n16), stream, __VA_ARGS__);                             \
    }                                                                                      \
  } while (0)

#define KVX_DIR_ORDER(D, O) D, O

template <bool kToPacked, bool kOrdered>
hipError_t launch(const LayerPtrs& lp, const int32_t* bt, const UnitGeom& ug, uint32_t n_units,
                  const uint32_t* order, char* packed, int* err, int layout, int elem,
                  hipStream_t stream) {
  const uint32_t n16 = ug.n16;
  for (uint32_t base = 0; base < n_units; base += kMaxUnitsPerLaunch) {
    const uint32_t cnt = n_units - base < kMaxUnitsPerLaunch ? n_units - base : kMaxUnitsPerLaunch;
    const dim3 grid(cnt);
    KVX_DISPATCH(copy_units_kernel, KVX_DIR_ORDER(kToPacked, kOrdered), lp, bt, ug, base, cnt,
                 order, packed, err);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <bool kToPacked>
hipError_t launch_chunks(const LayerPtrs& lp, const int32_t* bt, const kvx_chunk_ref* refs,
                         const ChunkGeom& cg, uint32_t n_units, char* packed, int* err,
                         int layout, int elem, hipStream_t stream) {
  const uint32_t n16 = cg.n16;
  for (uint32_t base = 0; base < n_units; base += kMaxUnitsPerLaunch) {
    const uint32_t cnt = n_units - base < kMaxUnitsPerLaunch ? n_units - base : kMaxUnitsPerLaunch;
    const dim3 grid(cnt);
    KVX_DISPATCH(copy_chunks_kernel, kToPacked, lp, bt, refs, cg, base, cnt, packed, err);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

SlabGeom slab_geom(const kvx_cache* c) {
  SlabGeom sg;
  sg.bs = (uint32_t)c->block_size;
  sg.h = (uint32_t)c->num_kv_heads;
  sg.d = (uint32_t)c->head_dim;
  sg.v16 = (uint32_t)((int64_t)c->head_dim * c->elem_bytes / 16);
  sg.x = (uint32_t)(16 / c->elem_bytes);
  sg.pad = 0;
  return sg;
}

}  // namespace

int* device_error_word() {
  static std::mutex mu;
  static int* addr[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(g_error_word)) == hipSuccess) addr[dev] = (int*)p;
  }
  return addr[dev];
}

kvx_status launch_copy(bool to_packed, const kvx_cache* cache, int32_t l0, int32_t l1,
                       const int32_t* block_table, const Geometry& g, void* packed,
                       hipStream_t stream) {
  if (g.n_units == 0) return KVX_OK;
  if (g.n_units > 0x7FFFFFFF || g.slab % 16 != 0) return KVX_EINTERNAL;
  int* err = device_error_word();
  if (!err) return KVX_EHIP;
  LayerPtrs lp = {};
  for (int32_t l = l0; l < l1; ++l) {
    lp.p[2 * (l - l0)] = static_cast<char*>(cache->k[l]);
    lp.p[2 * (l - l0) + 1] = static_cast<char*>(cache->v[l]);
  }
  UnitGeom ug;
  ug.units_per_chunk = (uint32_t)(2 * g.lr * g.bpc);
  ug.bpc = (uint32_t)g.bpc;
  ug.n_blocks = (uint32_t)g.n_blocks;
  ug.num_blocks = (uint32_t)g.num_blocks;
  ug.n16 = (uint32_t)(g.slab / 16);
  ug.pad = 0;
  ug.slab = (uint64_t)g.slab;
  ug.sg = slab_geom(cache);
  const int layout = cache->layout, elem = cache->elem_bytes;
  const uint32_t n_units = (uint32_t)g.n_units;
  if (to_packed) {
    hipError_t e = launch<true, false>(lp, block_table, ug, n_units, nullptr, (char*)packed, err,
                                       layout, elem, stream);
    return e == hipSuccess ? KVX_OK : KVX_EHIP;
  }
  // Destination-ordered scatter for large calls; the order lives in
  // stream-ordered scratch. If that allocation fails, fall back to image
  // order (same result, slower).
  uint32_t* order = nullptr;
  if (g.n_blocks >= kOrderedScatterMinBlocks &&
      hipMallocAsync((void**)&order, (size_t)g.n_blocks * sizeof(uint32_t), stream) != hipSuccess)
    order = nullptr;
  (void)hipGetLastError();
  hipError_t e;
  if (order) {
    hipLaunchKernelGGL(order_kernel, dim3(1), dim3(kOrderThreads), 0, stream, block_table,
                       (uint32_t)g.n_blocks, (uint32_t)g.num_blocks, order);
    e = hipGetLastError();
    if (e == hipSuccess)
      e = launch<false, true>(lp, block_table, ug, n_units, order, (char*)packed, err, layout,
                              elem, stream);
    const hipError_t ef = hipFreeAsync(order, stream);
    if (e == hipSuccess) e = ef;
  } else {
    e = launch<false, false>(lp, block_table, ug, n_units, nullptr, (char*)packed, err, layout,
                             elem, stream);
  }
  return e == hipSuccess ? KVX_OK : KVX_EHIP;
}

kvx_status launch_copy_chunks(bool to_packed, const kvx_cache* cache, int32_t l0, int32_t l1,
                              const int32_t* block_table, int32_t table_len,
                              const kvx_chunk_ref* refs, int32_t n_chunks, int32_t chunk_tokens,
                              void* packed, int64_t packed_bytes, hipStream_t stream) {
  if (n_chunks <= 0 || l1 <= l0) return KVX_OK;
  int* err = device_error_word();
  if (!err) return KVX_EHIP;
  const int64_t slab = (int64_t)cache->block_size * cache->num_kv_heads * cache->head_dim *
                       cache->elem_bytes;
  const int64_t bpc = chunk_tokens / cache->block_size;
  const int64_t upc = (int64_t)(l1 - l0) * 2 * bpc;
  const int64_t n_units = upc * n_chunks;
  if (bpc <= 0 || n_units > 0x7FFFFFFF || slab % 16 != 0) return KVX_EINTERNAL;
  LayerPtrs lp = {};
  for (int32_t l = l0; l < l1; ++l) {
    lp.p[2 * (l - l0)] = static_cast<char*>(cache->k[l]);
    lp.p[2 * (l - l0) + 1] = static_cast<char*>(cache->v[l]);
  }
  ChunkGeom cg;
  cg.upc = (uint32_t)upc;
  cg.bpc = (uint32_t)bpc;
  cg.lr2 = (uint32_t)(2 * (l1 - l0));
  cg.num_blocks = (uint32_t)cache->num_blocks;
  cg.n16 = (uint32_t)(slab / 16);
  cg.table_len = table_len;
  cg.slab = (uint64_t)slab;
  cg.packed_bytes = packed_bytes;
  cg.sg = slab_geom(cache);
  const int layout = cache->layout, elem = cache->elem_bytes;
  hipError_t e = to_packed ? launch_chunks<true>(lp, block_table, refs, cg, (uint32_t)n_units,
                                                 (char*)packed, err, layout, elem, stream)
                           : launch_chunks<false>(lp, block_table, refs, cg, (uint32_t)n_units,
                                                  (char*)packed, err, layout, elem, stream);
  return e == hipSuccess ? KVX_OK : KVX_EHIP;
}

}  // namespace kvx
