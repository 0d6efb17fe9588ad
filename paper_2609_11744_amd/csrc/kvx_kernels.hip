// HIP kernels for gfx950: paged-KV gather (paged slabs -> packed image) and
// scatter (packed image -> paged slabs).
//
// The work is pure data movement, bound by HBM bandwidth, so the kernels use
// no MFMA. With the default cache layout every slab is contiguous and in the
// same order on both sides, so nothing is transposed and no LDS is used; the
// other cache layouts move a slab head by head (see move_head).
// A unit is a slab (layer, K|V, block) of `slab` bytes. With the default
// layout one workgroup moves one part of a unit: 256 threads, one 16-byte
// vector each, so a part is 4 KiB (a 32 KiB slab is 8 parts; the last part of
// a slab may be short). On this chip a copy moves measurably more bytes per
// second with one load and one store per thread in many short workgroups than
// with several vectors per thread in fewer, longer ones (contiguous 4 GiB:
// 83 % of peak against 77.5 % at 1024 threads x 2 vectors; the 80k gather
// pattern 76.7 % against 73.6 %); persistent grids that loop over units
// measured lower still. The other layouts move a whole slab per workgroup.
//   * the unit's decode (chunk, layer, K|V, block, part) and its block-table
//     read depend on blockIdx only, so they run on the scalar unit once per
//     workgroup;
//   * the slab moves as 16-byte vectors, consecutive lanes on consecutive
//     addresses, so every wave instruction reads or writes 1 KiB contiguous;
//   * both streams are touched once, so loads are non-temporal and stores
//     stream to memory at device scope (kvx_store.h);
//   * workgroups are dispatched round-robin over the 8 XCDs, so workgroup b
//     is mapped to a (unit, part) such that each XCD walks one contiguous
//     range of them. The packed side of an XCD's work is then one sequential
//     stream, which HBM serves measurably better than 8 interleaved ones (the
//     write side of a copy is what bounds it).
// The packed-side address of unit u is u * slab (see Geometry), so only the
// paged side goes through the block table.
//
// Large scatters write to caller-chosen (typically random) blocks. HBM takes
// writes faster when each XCD's write stream ascends through memory, so a
// large scatter first buckets the destination ids (order_kernel, into
// stream-ordered scratch) and then visits units layer by layer in ascending
// destination order; the packed side is then read out of order, which costs
// less than unordered writes. The exceptions measured faster in image order:
// a chunk of one block (each chunk is then one sequential read, and the
// writes go to one destination block of every layer in turn;
// scatter_in_destination_order in kvx_walk.cpp), and slabs of at most 8 KiB,
// walked with no XCD ranges so that the whole chip reads the packed image
// front to back (scatter_linear).
//
// Pairing at 2 MiB. Where a layer|K|V slice's run in a packed chunk (blocks
// per chunk x slab) times a power of two D is 2 MiB, both directions can move
// two slices D apart together: the gather walks each chunk's slices in such
// pairs (its packed-side writes alternate between two runs 2 MiB apart; D up
// to 32), and the ordered scatter walks each XCD's range as two fronts that
// move the same destination block of two such slices (D up to 16 for slabs
// above 8 KiB, else 4). Both
// measured faster than the plain walks on this chip, and pairs at other
// distances slower (scatter_pairing, gather_pairing in kvx_walk.cpp).
#include <hip/hip_runtime.h>

#include <mutex>
#include <type_traits>

#include "kvx_internal.h"
#include "kvx_store.h"

namespace kvx {
namespace {

using kvx_dev::store_stream;
using kvx_dev::stream_dst;
using kvx_dev::v4u;

constexpr int kErrBadBlock = 1;
constexpr int kErrBadChunk = 2;
constexpr int kErrorWords = 1024;  // word 0: the null stream, and streams beyond the table

// One entry of a scatter's destination order: a block-table index and the
// block id found there (read once by the ordering kernel).
struct OrderEntry {
  uint32_t index;
  int32_t id;
};

// Device pointers of the call's layers, in image order: p[2 * (l - l0) + kv].
// Passed by value as a kernel argument (2 KiB for KVX_MAX_LAYERS = 128).
struct LayerPtrs {
  char* p[2 * KVX_MAX_LAYERS];
};

// Division by a divisor known only at run time, as a multiply: for d >= 2,
// m = ceil(2^32 / d) and n / d = umulhi(n, m) whenever n * d < 2^32 (the
// rounding error of m, below d, then moves n * m / 2^32 by less than 1/d);
// m = 0 stands for d = 1. Every numerator here is an element or vector index
// inside one head's part of a slab and every divisor a slab dimension; a
// transposed slab is at most kMaxTransposedSlab (48 KiB) bytes, so both are
// below 2^16.
struct FastDiv {
  uint32_t d;
  uint32_t m;
};

__device__ __forceinline__ uint32_t fdiv(uint32_t n, FastDiv f) {
  return f.m ? __umulhi(n, f.m) : n;
}

// Shape of one head's part of a slab, for the reordering layouts.
struct SlabGeom {
  FastDiv bs;      // tokens per block
  FastDiv d;       // head dim (elements)
  FastDiv v16;     // 16-byte vectors per (token, head) row: d * elem_bytes / 16
  uint32_t x;      // elements per 16-byte vector: 16 / elem_bytes
  uint32_t nh;     // vectors of one head: bs * v16
  uint32_t prow;   // packed row stride in vectors: heads * v16
  FastDiv pad;       // scatter: LDS pad period (see lds_slot)
  uint32_t v_pairs;  // paged-attention V of 2-byte words gathered as row pairs (v_pairs_gather)
  uint32_t swz;      // gather: LDS swizzle shift (see lds_slot)
};

// Division of any 32-bit numerator by a divisor fixed for the launch, as a
// multiply (Granlund and Montgomery, "Division by invariant integers using
// multiplication", 1994): with l = ceil(log2 d), m = floor(2^32 (2^l - d) / d)
// + 1 and t = umulhi(n, m), n / d = (t + ((n - t) >> 1)) >> (l - 1) for d >= 2;
// m = 0 stands for d = 1. The workgroup index decode divides unit indexes (up
// to 2^31) by slab and chunk counts, so the narrower FastDiv does not apply.
struct DivU32 {
  uint32_t d;
  uint32_t m;
  uint32_t s;
};

__device__ __forceinline__ uint32_t divu(uint32_t n, DivU32 f) {
  if (f.m == 0) return n;
  const uint32_t t = __umulhi(n, f.m);
  return (t + ((n - t) >> 1)) >> f.s;
}

struct UnitGeom {
  uint32_t units_per_chunk;  // (l1 - l0) * 2 * bpc
  uint32_t bpc;
  uint32_t n_blocks;
  uint32_t num_blocks;       // pool size
  uint32_t n16;              // 16-byte vectors per slab
  uint32_t parts;            // workgroups per slab (parts_shift: log2 of a power of two, else 32)
  uint32_t parts_shift;
  // Ordered scatter walked as two fronts per XCD (xcd_two_fronts) whose
  // slices are paired D = 2^pair_shift apart (paired_slice); pair_shift = 32
  // for one front per XCD. Gather: each chunk's slices walked in pairs
  // 2^gather_pair_shift apart (see the unit decode), or 32 for the plain walk.
  uint32_t pair_shift;
  uint32_t gather_pair_shift;
  uint32_t half_slices;      // slices per half of an XCD's range
  uint32_t linear_walk;      // 1: workgroup b moves work item b (no XCD ranges)
  DivU32 xcd_slices_div;     // by slices per XCD range
  DivU32 parts_div;
  DivU32 upc_div;            // by units_per_chunk
  DivU32 bpc_div;            // by bpc
  DivU32 last_div;           // by the last chunk's block count
  DivU32 nb_div;             // by n_blocks
  uint64_t slab;
  SlabGeom sg;
};

// Sticky error words, a table per device: each stream that launches copies
// gets a word of its own (stream_error_word), so that a check of one stream
// neither reports nor clears another stream's error. Host code reaches the
// table only through the address that hipGetSymbolAddress returns.
__device__ int g_error_words[kErrorWords];

// Workgroup b of a launch over n units -> unit index. XCD x = b % kXcds runs
// the workgroups b = x, x + kXcds, ...; they get the contiguous range
// [x*q + min(x, r), ...) of q or q + 1 units (q = n / kXcds, r = n % kXcds).
// A bijection on [0, n) for every n.
__device__ __forceinline__ uint32_t xcd_contiguous(uint32_t b, uint32_t n) {
  const uint32_t q = n / kXcds, r = n % kXcds, x = b % kXcds, k = b / kXcds;
  return x * q + (x < r ? x : r) + k;
}

// The same ranges for the destination-ordered scatter, walked as two fronts:
// XCD x's range is cut into halves (the first a whole number of slabs,
// `parts` work items each, parts a power of two, 2^shift) and its workgroups
// alternate between them, one work item at a time (items past twice the
// first half follow in order). A bijection on [0, n). The launcher uses it
// only where each XCD's range is a whole, even number of layer|K|V slices,
// so that the two fronts move the same destination block of two slices
// together (its writes in two cache tensors, its reads from one packed
// chunk), and paired_slice chooses which two (scatter_pairing, kvx_walk.cpp).
__device__ __forceinline__ uint32_t xcd_two_fronts(uint32_t b, uint32_t n, uint32_t shift) {
  const uint32_t q = n / kXcds, r = n % kXcds, x = b % kXcds, k = b / kXcds;
  const uint32_t len = q + (x < r ? 1u : 0u), start = x * q + (x < r ? x : r);
  const uint32_t half = ((len >> 1) >> shift) << shift;
  if (k >= 2 * half) return start + k;
  const uint32_t pair = k >> (shift + 1), i = k & ((2u << shift) - 1);
  return start + (i & 1) * half + (pair << shift) + (i >> 1);
}

// The layer|K|V slice moved at slice r of the ordered walk (XCD x's range is
// walk slices [x S, (x + 1) S), halves of H = S / 2): slice t of the first
// half of XCD x's range and slice t of its second half are pair j = H x + t,
// which moves slices a_j and a_j + D (a_j: the j-th slice whose index has bit
// log2 D clear, D = 2^ds). A bijection on the slices when their count is a
// multiple of 2 D.
__device__ __forceinline__ uint32_t paired_slice(uint32_t r, DivU32 sx, uint32_t half,
                                                 uint32_t ds) {
  const uint32_t x = divu(r, sx), rem = r - x * sx.d;
  const uint32_t h = rem >= half ? 1u : 0u, jj = half * x + rem - h * half;
  return ((jj >> ds) << (ds + 1)) + (jj & ((1u << ds) - 1)) + (h << ds);
}

template <int T, int V>
__device__ __forceinline__ void move_slab(const v4u* __restrict__ s, v4u* __restrict__ d,
                                          uint32_t n16) {
  const auto out = stream_dst(d, n16 * 16u);
  uint32_t i = threadIdx.x;
  // Main body: V vectors per thread per pass, loads first.
  for (; i + (V - 1) * T < n16; i += V * T) {
    v4u r[V];
#pragma unroll
    for (int q = 0; q < V; ++q) r[q] = __builtin_nontemporal_load(s + i + q * T);
#pragma unroll
    for (int q = 0; q < V; ++q) store_stream(out, i + q * T, r[q]);
  }
  for (; i < n16; i += T) store_stream(out, i, __builtin_nontemporal_load(s + i));
}

// ---- cache layouts that reorder a slab ---------------------------------------
//
// The packed side is always [token][head][dim]. The cache side may be
//   KVX_LAYOUT_HND         [head][token][dim] rows (K and V);
//   KVX_LAYOUT_PAGED_ATTN  K [head][dim / x][token][x] (x = 16 / elem_bytes: the
//                          16-byte vectors of a row are re-strided), V
//                          [head][dim][token] (an element transpose).
// In every one of them a head's data is contiguous on the cache side (nh =
// bs * v16 vectors), and on the packed side it is one v16-vector row per token
// at stride prow = heads * v16. So a workgroup moves one head (the slab's
// parts are its heads), one vector per thread for the usual shapes; inside a
// head, local packed vector w = t * v16 + dv sits at packed_at(w).
//   * HND: the head's cache rows are its packed rows in the same order, so
//     vectors move directly (no LDS); the packed side is 16 * v16-byte runs.
//   * paged-attention K: a vector permutation. The head is loaded in source
//     order into LDS, then written in destination order, each lane fetching
//     the source vector its output vector is. (Moving each vector straight
//     from its source to its destination, the packed side then in 64-byte
//     runs, measured 2.3 points slower both ways on the 80k workload: the
//     wave-contiguous runs on both sides are worth more than the LDS pass.)
//   * paged-attention V: an element transpose. The head is loaded in source
//     order into LDS, then each output vector is assembled element by element
//     from it.
// Both global sides stay coalesced (consecutive lanes on consecutive 16-byte
// vectors, or whole packed rows) and only LDS sees the reordering; the LDS
// image is swizzled so that a wave's strided reads land on distinct banks. A
// thread holds V vectors of the head, all of its loads issued before it waits
// for any of them: V = 1 when a head fits one vector per thread (the usual
// shapes: few registers, full occupancy), else kVecPerThread, enough for the
// largest head (kMaxSlabVectors).

constexpr int kTransposeThreads = 256;
constexpr uint32_t kMaxSlabVectors = 48 * 1024 / 16;
constexpr int kVecPerThread = (int)(kMaxSlabVectors / kTransposeThreads);  // 12

extern __shared__ __attribute__((aligned(16))) unsigned char kvx_lds[];

// LDS slot of vector v in the head's image; the layout differs by direction.
// Gather (kToPacked): inside each aligned group of 16 vectors (256 bytes, one
// pass over the 64 banks) the position is XORed with h(r), r = bits swz ..
// swz + 3 of v, which the XOR leaves alone, so the map is a permutation of
// every group. h(r) = r ^ (bit 3 of r moved to bit 1) is itself a permutation
// of 0 .. 15, so a wave walking the image at a stride of 2^swz vectors (the
// head's read stride, chosen on the host) meets 16 different positions per
// group, and consecutive vectors stay in one group; moving bit 3 to bit 1
// also keeps rows r and r + 8 apart modulo 8 positions (32 banks), where the
// 32-bit reads of a half-wave meet (see lane_perm). Scatter: one pad vector
// after every `pad` vectors (the read stride). Measured on gfx950 with the LDS
// bank-conflict counter, a 16 x 16 transposed read of 16-byte vectors costs
// no conflict cycles through an XOR swizzle, 4 per wave instruction with the
// pad and 28 with neither, and linear 16-byte writes cost none either way.
// The 80k paged-attention gather ran 1 to 2 points faster with the swizzle
// (no conflicts left) than with the pad; the scatter ran 2 points slower
// with it (also with no conflicts left): it is not bound by the LDS, and the
// swizzle's extra arithmetic in its element-by-element loop costs more than
// the conflicts it removes.
template <bool kToPacked>
__device__ __forceinline__ uint32_t lds_slot(uint32_t v, const SlabGeom& g) {
  if (kToPacked) {
    const uint32_t r = (v >> g.swz) & 15u;
    return v ^ (r ^ ((r >> 2) & 2u));
  }
  return v + fdiv(v, g.pad);
}

// Quotient and remainder.
__device__ __forceinline__ uint32_t divmod(uint32_t n, FastDiv f, uint32_t& rem) {
  const uint32_t q = fdiv(n, f);
  rem = n - q * f.d;
  return q;
}

// Bytes a head's moves write from the destination's first vector: the head's
// packed rows (a gather) or its nh contiguous cache vectors (a scatter).
template <bool kToPacked>
__device__ __forceinline__ uint32_t head_dst_bytes(const SlabGeom& g) {
  return (kToPacked ? (g.bs.d - 1) * g.prow + g.v16.d : g.nh) * 16u;
}

// Packed-side offset (in vectors, from the head's first row) of local packed
// vector w = t * v16 + dv.
__device__ __forceinline__ uint32_t packed_at(uint32_t w, const SlabGeom& g) {
  uint32_t dv;
  const uint32_t t = divmod(w, g.v16, dv);
  return t * g.prow + dv;
}

// HND: local vector w is cache vector w and local packed vector w.
template <bool kToPacked, int T, int V>
__device__ __forceinline__ void move_head_rows(const v4u* __restrict__ src, v4u* __restrict__ dst,
                                               const SlabGeom& g) {
  v4u r[V];
#pragma unroll
  for (int q = 0; q < V; ++q) {
    const uint32_t w = threadIdx.x + q * T;
    if (w < g.nh) r[q] = __builtin_nontemporal_load(src + (kToPacked ? w : packed_at(w, g)));
  }
  const auto out = stream_dst(dst, head_dst_bytes<kToPacked>(g));
#pragma unroll
  for (int q = 0; q < V; ++q) {
    const uint32_t w = threadIdx.x + q * T;
    if (w < g.nh) store_stream(out, kToPacked ? packed_at(w, g) : w, r[q]);
  }
}

// Load the head's nh source vectors, in source order, into the padded LDS
// image. A gather reads the cache (contiguous), a scatter the packed rows.
template <bool kToPacked, int T, int V>
__device__ __forceinline__ void stage_in(const v4u* __restrict__ src, const SlabGeom& g) {
  v4u* lds = reinterpret_cast<v4u*>(kvx_lds);
  v4u r[V];
#pragma unroll
  for (int q = 0; q < V; ++q) {
    const uint32_t v = threadIdx.x + q * T;
    if (v < g.nh) r[q] = __builtin_nontemporal_load(src + (kToPacked ? v : packed_at(v, g)));
  }
#pragma unroll
  for (int q = 0; q < V; ++q) {
    const uint32_t v = threadIdx.x + q * T;
    if (v < g.nh) lds[lds_slot<kToPacked>(v, g)] = r[q];
  }
}

// The LDS serves 32-bit and narrower reads a half-wave (32 lanes) at a time
// over 32 banks (measured: two extra cycles per such read when a half-wave
// puts two words on one bank). The paired V gather below therefore lets lane
// L of a wave handle pair lane_perm(L) of the wave's 64 pairs, a permutation
// of the lane bits (b5 b4 b3 b2 b1 b0 -> b4 b3 b5 b2 b1 b0) that gives each
// half-wave 4 token pairs x 8 dim groups instead of 2 x 16; the 64 pairs of a
// wave, and so the bytes each store instruction writes, are the same as in
// lane order. (The scatter keeps lane order: permuting which lane stores
// which cache vector measured a point slower, the stores of a wave no longer
// running in address order; its reads are kept apart by the swizzle.)
__device__ __forceinline__ uint32_t lane_perm(uint32_t i) {
  const uint32_t l = i & 63u;
  return (i & ~63u) | (((l >> 3) & 3u) << 4) | (((l >> 5) & 1u) << 3) | (l & 7u);
}

// Write the head's nh destination vectors, in destination order, each
// produced by f(w). A gather writes the packed rows, a scatter the cache.
template <bool kToPacked, int T, int V, typename F>
__device__ __forceinline__ void stage_out(v4u* __restrict__ dst, const SlabGeom& g, F f) {
  v4u r[V];
#pragma unroll
  for (int q = 0; q < V; ++q) {
    const uint32_t w = threadIdx.x + q * T;
    if (w < g.nh) r[q] = f(w);
  }
  const auto out = stream_dst(dst, head_dst_bytes<kToPacked>(g));
#pragma unroll
  for (int q = 0; q < V; ++q) {
    const uint32_t w = threadIdx.x + q * T;
    if (w < g.nh) store_stream(out, kToPacked ? packed_at(w, g) : w, r[q]);
  }
}

// Paged-attention K: source vector (in the LDS image) of destination vector w.
// Cache order inside a head is w = dv * bs + t, packed order w = t * v16 + dv.
template <bool kToPacked>
__device__ __forceinline__ uint32_t k_source(uint32_t w, const SlabGeom& g) {
  uint32_t lo;
  if (kToPacked) {
    const uint32_t t = divmod(w, g.v16, lo);  // lo = dv
    return lo * g.bs.d + t;
  }
  const uint32_t dv = divmod(w, g.bs, lo);    // lo = t
  return lo * g.v16.d + dv;
}

template <typename E>
struct ElemRow {
  E e[16 / sizeof(E)];
};

// Paged-attention V: destination vector w assembled element by element from
// the LDS image of the source. Cache elements inside a head are (dim, t) at
// dim * bs + t; packed elements (t, dim) at t * d + dim.
template <bool kToPacked, typename E>
__device__ __forceinline__ v4u v_elements(uint32_t w, const SlabGeom& g) {
  constexpr uint32_t kX = 16 / sizeof(E);
  ElemRow<E> out;
  if (kToPacked) {  // packed (t, dv * x + i) <- cache element (dv * x + i, t): stride bs
    uint32_t dv;
    const uint32_t t = divmod(w, g.v16, dv);
    const uint32_t e0 = dv * kX * g.bs.d + t;
#pragma unroll
    for (uint32_t i = 0; i < kX; ++i) {
      const uint32_t e = e0 + i * g.bs.d;
      out.e[i] = reinterpret_cast<const E*>(kvx_lds + 16u * lds_slot<kToPacked>(e / kX, g))[e % kX];
    }
  } else {  // cache (dim, t .. t + x - 1) <- packed elements (t + i, dim); t wraps to dim + 1
    uint32_t t;
    uint32_t dim = divmod(w * kX, g.bs, t);
#pragma unroll
    for (uint32_t i = 0; i < kX; ++i) {
      const uint32_t e = t * g.d.d + dim;
      out.e[i] = reinterpret_cast<const E*>(kvx_lds + 16u * lds_slot<kToPacked>(e / kX, g))[e % kX];
      if (++t == g.bs.d) {
        t = 0;
        ++dim;
      }
    }
  }
  return __builtin_bit_cast(v4u, out);
}

// Paged-attention V of 2-byte words in a gather, two packed rows per thread:
// the rows of tokens t and t + 1 (t even) at one group of dims, whose
// elements come from cache words (dim, t) and (dim, t + 1), adjacent in one
// dword. Each 32-bit LDS read yields one element of each vector, so no two
// lanes share a dword, and for the usual shapes (block size 16, 16 vectors
// per row) a wave's reads of one element land on 64 distinct banks; the two
// stores of a lane write whole token rows. A scatter does not pair its
// vectors this way: paired dims d, d + 1 would make each store instruction
// write every other 32-byte run of the cache lines (the 80k scatter ran at
// half speed that way).
template <int T, int V>
__device__ __forceinline__ void v_pairs_gather(v4u* __restrict__ dst, const SlabGeom& g) {
  typedef ElemRow<uint16_t> Row;
  const uint32_t np = g.nh >> 1;
  Row r0[V], r1[V];
  uint32_t w0[V];
#pragma unroll
  for (int q = 0; q < V; ++q) {
    // a half-wave takes 4 token pairs x 8 dim groups (16 vectors per row)
    const uint32_t p = lane_perm(threadIdx.x + q * T);
    if (p >= np) continue;
    uint32_t dv;
    const uint32_t tp = divmod(p, g.v16, dv);  // tokens 2 tp, 2 tp + 1
    w0[q] = 2 * tp * g.v16.d + dv;
    const uint32_t e0 = dv * 8 * g.bs.d + 2 * tp;
#pragma unroll
    for (uint32_t i = 0; i < 8; ++i) {
      const uint32_t e = e0 + i * g.bs.d;
      const uint32_t w = *reinterpret_cast<const uint32_t*>(kvx_lds + 16u * lds_slot<true>(e >> 3, g) +
                                                            2u * (e & 7u));
      r0[q].e[i] = (uint16_t)w;
      r1[q].e[i] = (uint16_t)(w >> 16);
    }
  }
  const auto out = stream_dst(dst, head_dst_bytes<true>(g));
#pragma unroll
  for (int q = 0; q < V; ++q) {
    const uint32_t p = lane_perm(threadIdx.x + q * T);
    if (p >= np) continue;
    store_stream(out, packed_at(w0[q], g), __builtin_bit_cast(v4u, r0[q]));
    store_stream(out, packed_at(w0[q] + g.v16.d, g), __builtin_bit_cast(v4u, r1[q]));
  }
}

// One head of a slab in a reordering layout (src / dst: the head's cache
// vectors and its first packed row, in the kernel's direction).
template <bool kToPacked, int kLayout, int kElem, int T, int V>
__device__ __forceinline__ void move_head(const v4u* __restrict__ src, v4u* __restrict__ dst,
                                          const SlabGeom& g, uint32_t kv) {
  typedef typename std::conditional<
      kElem == 1, uint8_t,
      typename std::conditional<kElem == 2, uint16_t,
                                typename std::conditional<kElem == 4, uint32_t,
                                                          uint64_t>::type>::type>::type E;
  if (kLayout == KVX_LAYOUT_HND) {
    move_head_rows<kToPacked, T, V>(src, dst, g);
    return;
  }
  stage_in<kToPacked, T, V>(src, g);
  __syncthreads();
  const v4u* lds = reinterpret_cast<const v4u*>(kvx_lds);
  if (kv == 0)
    stage_out<kToPacked, T, V>(
        dst, g, [&](uint32_t w) { return lds[lds_slot<kToPacked>(k_source<kToPacked>(w, g), g)]; });
  else if (kToPacked && kElem == 2 && g.v_pairs)
    v_pairs_gather<T, V>(dst, g);
  else
    stage_out<kToPacked, T, V>(dst, g,
                               [&](uint32_t w) { return v_elements<kToPacked, E>(w, g); });
}

// Move part `part` of one slab in the direction and layout of the kernel: a
// 4 KiB piece with the default layout, one head with the reordering ones.
template <bool kToPacked, int kLayout, int kElem, int T, int V>
__device__ __forceinline__ void move_unit(char* paged, char* pk, uint32_t n16, const SlabGeom& g,
                                          uint32_t kv, uint32_t part) {
  v4u* pv = reinterpret_cast<v4u*>(paged);
  v4u* kv4 = reinterpret_cast<v4u*>(pk);
  if (kLayout == KVX_LAYOUT_NHD) {
    const uint32_t off = part * (uint32_t)(T * V);  // < n16: part < ceil(n16 / (T * V))
    const uint32_t left = n16 - off;
    const uint32_t n = left < (uint32_t)(T * V) ? left : (uint32_t)(T * V);
    if (kToPacked)
      move_slab<T, V>(pv + off, kv4 + off, n);
    else
      move_slab<T, V>(kv4 + off, pv + off, n);
  } else {
    v4u* cache_head = pv + part * g.nh;       // head `part`: nh contiguous cache vectors
    v4u* packed_head = kv4 + part * g.v16.d;  // its first packed row
    if (kToPacked)
      move_head<true, kLayout, kElem, T, V>(cache_head, packed_head, g, kv);
    else
      move_head<false, kLayout, kElem, T, V>(packed_head, cache_head, g, kv);
  }
}

// Work item w of a launch -> (unit, part of the unit).
__device__ __forceinline__ uint32_t split_work(uint32_t w, uint32_t parts, uint32_t shift,
                                               DivU32 parts_div, uint32_t* part) {
  const uint32_t u = shift < 32 ? w >> shift : divu(w, parts_div);
  *part = w - u * parts;
  return u;
}

// Work item w = unit * parts + part.
// kOrdered = false: units in image order (u -> chunk, layer|K|V, block).
// kOrdered = true: unit v -> lk = v / n_blocks, k = v % n_blocks, (block index
// i, its block id) = order[k] (destinations ascending by bucket); the image
// position u of (chunk i / bpc, lk, block i % bpc) follows.
// A workgroup moves only 4 KiB, so the scalar loads before its first data
// load matter: the block id and the layer pointer (or, ordered, the order
// entry, which carries the id, and the layer pointer) are issued together
// and waited for once. The empty asm statements take the loaded values,
// which keeps the compiler from moving the layer pointer's load past the
// block-id check.
template <bool kToPacked, bool kOrdered, int kLayout, int kElem, int T, int V>
__global__ void __launch_bounds__(T)
    copy_units_kernel(LayerPtrs layers, const int32_t* __restrict__ block_table, UnitGeom g,
                      uint32_t work_base, uint32_t work_count,
                      const OrderEntry* __restrict__ order, char* __restrict__ packed,
                      int* __restrict__ err) {
  uint32_t part;
  const uint32_t w = g.linear_walk                  ? blockIdx.x
                     : kOrdered && g.pair_shift < 32 ? xcd_two_fronts(blockIdx.x, work_count,
                                                                      g.parts_shift)
                                                     : xcd_contiguous(blockIdx.x, work_count);
  uint32_t u = split_work(work_base + w, g.parts, g.parts_shift, g.parts_div, &part);
  uint32_t c, first, nc, lk, j;
  int32_t id;
  char* layer;
  if (kOrdered) {
    const uint32_t walk = divu(u, g.nb_div);  // slice in walk order
    const OrderEntry e = order[u - walk * g.n_blocks];  // e.index < n_blocks (a permutation)
    lk = g.pair_shift < 32 ? paired_slice(walk, g.xcd_slices_div, g.half_slices, g.pair_shift)
                           : walk;
    layer = layers.p[lk];
    __asm__ volatile("" : : "s"(e.index), "s"(e.id), "s"(layer));
    const uint32_t i = e.index;
    id = e.id;
    c = divu(i, g.bpc_div);
    first = c * g.bpc;
    j = i - first;
    const uint32_t left = g.n_blocks - first;
    nc = left < g.bpc ? left : g.bpc;
    u = c * g.units_per_chunk + lk * nc + j;
  } else {
    c = divu(u, g.upc_div);
    const uint32_t r = u - c * g.units_per_chunk;
    first = c * g.bpc;
    const uint32_t left = g.n_blocks - first;
    nc = left < g.bpc ? left : g.bpc;  // blocks in this chunk
    const DivU32 ncd = nc == g.bpc ? g.bpc_div : g.last_div;
    if (g.gather_pair_shift < 32) {
      // Paired walk of the chunk: its work items in walk order are pair p of
      // slices (a_p, a_p + D) (a_p: the p-th slice whose index has bit log2 D
      // clear, D = 2^ds), then block j, then the two slices' part `part`
      // alternately. A bijection on the chunk's items.
      const uint32_t ps = g.parts_shift + 1, ds = g.gather_pair_shift;
      const uint32_t wi = (r << g.parts_shift) + part;  // walk position within the chunk
      const uint32_t p = divu(wi >> ps, ncd);            // 2 * nc * parts items per pair
      const uint32_t r2 = wi - ((p * nc) << ps);
      const uint32_t r3 = r2 & ((1u << ps) - 1);
      j = r2 >> ps;
      part = r3 >> 1;
      lk = ((p >> ds) << (ds + 1)) + (p & ((1u << ds) - 1)) + ((r3 & 1) << ds);
      u = c * g.units_per_chunk + lk * nc + j;  // image position of (lk, j)
    } else {
      lk = divu(r, ncd);  // 2 * (l - l0) + kv
      j = r - lk * nc;
    }
    id = block_table[first + j];
    layer = layers.p[lk];
    __asm__ volatile("" : : "s"(id), "s"(layer));
  }
  if ((uint32_t)id >= g.num_blocks) {
    if (threadIdx.x == 0) atomicOr(err, kErrBadBlock);
    return;
  }
  char* paged = layer + (uint64_t)(uint32_t)id * g.slab;
  char* pk = packed + (uint64_t)u * g.slab;
  move_unit<kToPacked, kLayout, kElem, T, V>(paged, pk, g.n16, g.sg, lk & 1, part);
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
  uint32_t parts;        // workgroups per slab, as in UnitGeom
  uint32_t parts_shift;
  DivU32 parts_div;
  DivU32 upc_div;
  DivU32 bpc_div;
  int32_t table_len;
  uint64_t slab;
  int64_t packed_bytes;
  SlabGeom sg;
};

template <bool kToPacked, int kLayout, int kElem, int T, int V>
__global__ void __launch_bounds__(T)
    copy_chunks_kernel(LayerPtrs layers, const int32_t* __restrict__ block_table,
                       const kvx_chunk_ref* __restrict__ refs, ChunkGeom g, uint32_t work_base,
                       uint32_t work_count, char* __restrict__ packed, int* __restrict__ err) {
  uint32_t part;
  const uint32_t u = split_work(work_base + xcd_contiguous(blockIdx.x, work_count), g.parts,
                                g.parts_shift, g.parts_div, &part);
  const uint32_t c = divu(u, g.upc_div);
  const uint32_t r = u - c * g.upc;
  const uint32_t lk = divu(r, g.bpc_div);
  const uint32_t j = r - lk * g.bpc;
  const kvx_chunk_ref ref = refs[c];
  const bool ok = ref.n_blocks >= 1 && (uint32_t)ref.n_blocks <= g.bpc && ref.bt_offset >= 0 &&
                  (int64_t)ref.bt_offset + ref.n_blocks <= (int64_t)g.table_len &&
                  ref.packed_offset >= 0 && (ref.packed_offset & 15) == 0 &&
                  ref.packed_offset + (int64_t)g.lr2 * ref.n_blocks * (int64_t)g.slab <=
                      g.packed_bytes;
  if (!ok) {
    if (r == 0 && part == 0 && threadIdx.x == 0) atomicOr(err, kErrBadChunk);
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
  move_unit<kToPacked, kLayout, kElem, T, V>(paged, pk, g.n16, g.sg, lk & 1, part);
}

// Destination order for a scatter: order[] lists the block-table indexes,
// each with the id it holds, bucketed by destination id, buckets ascending. The id range [0, num_blocks)
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
                 OrderEntry* __restrict__ order) {
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
  for (uint32_t i = t; i < n; i += kOrderThreads) {
    const int32_t id = block_table[i];
    order[atomicAdd(&cnt[bin_of(id, num_blocks, bins)], 1u)] = OrderEntry{i, id};
  }
}

// Dynamic LDS bytes for a reordering layout: the image of one head, rounded
// up to whole swizzle groups of 16 vectors (gather) or with its pad vectors
// (scatter); none for HND, which moves rows directly.
inline size_t lds_bytes(int layout, const SlabGeom& sg, bool to_packed) {
  if (layout != KVX_LAYOUT_PAGED_ATTN) return 0;
  if (to_packed) return 16u * (size_t)((sg.nh + 15u) & ~15u);
  return 16u * (size_t)(sg.nh + sg.nh / sg.pad.d + 1);
}

// Launch `cnt` workgroups of kernel K<..., layout, elem, T, V>: the default
// layout moves 4 KiB parts (kPartThreads threads x 1 vector); the others move
// one head per workgroup of 256 threads (paged attention through LDS).
#define KVX_UNPAREN(...) __VA_ARGS__

// Whether a paged-attention scatter of heads that fit one vector per thread
// runs them on half as many threads with two vectors each. Twice as many of
// its workgroups then fit a compute unit, which keeps more loads in flight
// across its LDS phases. Measured over 12-18 (cache, packed buffer)
// allocation pairs in one process at the 80k prefix of the 8B shape, against
// one vector on each of 256 threads: 81.2 against 78.9 % of peak with 8
// heads, level with 4 (75.3 / 75.2 %), 69.4 against 69.9 % with 2 and, with
// the linear walk a one-head scatter takes (kvx_walk.cpp), 69.6 against
// 73.2 % with 1. So only slabs of four heads or more take it.
inline bool pa_scatter_on_half_threads(const SlabGeom& sg) {
  return sg.nh <= (uint32_t)kTransposeThreads && sg.prow >= 4u * sg.v16.d;
}

// One head per workgroup of kTransposeThreads: one vector per thread when the
// head fits, else kVecPerThread; a paged-attention scatter of four or more
// such heads per slab on half the threads (pa_scatter_on_half_threads; the
// gather and the HND layout were no faster that way). PREFIX is the kernel's
// parenthesized leading template arguments; kToPacked is the enclosing
// launcher's direction.
#define KVX_LAUNCH_HEADS(KERNEL, PREFIX, LAYOUT, ELEM, ...)                                 \
  do {                                                                                 \
    const dim3 tb(kTransposeThreads);                                                  \
    if constexpr (LAYOUT == KVX_LAYOUT_PAGED_ATTN && !kToPacked) {                     \
      if (pa_scatter_on_half_threads(sg)) {                                            \
        hipLaunchKernelGGL(                                                            \
            (KERNEL<KVX_UNPAREN PREFIX, LAYOUT, ELEM, kTransposeThreads / 2, 2>), grid, \
            dim3(kTransposeThreads / 2), lds_bytes(layout, sg, kToPacked), stream, __VA_ARGS__);  \
        break;                                                                         \
      }                                                                                \
    }                                                                                  \
    if (sg.nh <= (uint32_t)kTransposeThreads)                                          \
      hipLaunchKernelGGL((KERNEL<KVX_UNPAREN PREFIX, LAYOUT, ELEM, kTransposeThreads, 1>), \
                         grid, tb, lds_bytes(layout, sg, kToPacked), stream, __VA_ARGS__);        \
    else                                                                               \
      hipLaunchKernelGGL(                                                              \
          (KERNEL<KVX_UNPAREN PREFIX, LAYOUT, ELEM, kTransposeThreads, kVecPerThread>), \
          grid, tb, lds_bytes(layout, sg, kToPacked), stream, __VA_ARGS__);                       \
  } while (0)

#define KVX_DISPATCH(KERNEL, PREFIX, ...)                                                   \
  do {                                                                                 \
    if (layout == KVX_LAYOUT_NHD)                                                      \
      hipLaunchKernelGGL((KERNEL<KVX_UNPAREN PREFIX, KVX_LAYOUT_NHD, 0, kPartThreads, 1>), \
                         grid, dim3(kPartThreads), 0, stream, __VA_ARGS__);            \
    else if (layout == KVX_LAYOUT_HND)                                                 \
      KVX_LAUNCH_HEADS(KERNEL, PREFIX, KVX_LAYOUT_HND, 0, __VA_ARGS__);                 \
    else if (elem == 1)                                                                \
      KVX_LAUNCH_HEADS(KERNEL, PREFIX, KVX_LAYOUT_PAGED_ATTN, 1, __VA_ARGS__);          \
    else if (elem == 2)                                                                \
      KVX_LAUNCH_HEADS(KERNEL, PREFIX, KVX_LAYOUT_PAGED_ATTN, 2, __VA_ARGS__);          \
    else if (elem == 4)                                                                \
      KVX_LAUNCH_HEADS(KERNEL, PREFIX, KVX_LAYOUT_PAGED_ATTN, 4, __VA_ARGS__);          \
    else                                                                               \
      KVX_LAUNCH_HEADS(KERNEL, PREFIX, KVX_LAYOUT_PAGED_ATTN, 8, __VA_ARGS__);          \
  } while (0)

template <bool kToPacked, bool kOrdered>
hipError_t launch(const LayerPtrs& lp, const int32_t* bt, const UnitGeom& ug, uint32_t n_work,
                  const OrderEntry* order, char* packed, int* err, int layout, int elem,
                  hipStream_t stream) {
  const SlabGeom& sg = ug.sg;
  for (uint32_t base = 0; base < n_work; base += kMaxWorkPerLaunch) {
    const uint32_t cnt = n_work - base < kMaxWorkPerLaunch ? n_work - base : kMaxWorkPerLaunch;
    const dim3 grid(cnt);
    KVX_DISPATCH(copy_units_kernel, (kToPacked, kOrdered), lp, bt, ug, base, cnt,
                 order, packed, err);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <bool kToPacked>
hipError_t launch_chunks(const LayerPtrs& lp, const int32_t* bt, const kvx_chunk_ref* refs,
                         const ChunkGeom& cg, uint32_t n_work, char* packed, int* err,
                         int layout, int elem, hipStream_t stream) {
  const SlabGeom& sg = cg.sg;
  for (uint32_t base = 0; base < n_work; base += kMaxWorkPerLaunch) {
    const uint32_t cnt = n_work - base < kMaxWorkPerLaunch ? n_work - base : kMaxWorkPerLaunch;
    const dim3 grid(cnt);
    KVX_DISPATCH(copy_chunks_kernel, (kToPacked), lp, bt, refs, cg, base, cnt, packed, err);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

DivU32 div_u32(uint32_t d) {
  DivU32 f{d, 0u, 0u};
  if (d <= 1) return f;
  uint32_t l = 0;
  while (l < 32 && (1ull << l) < d) ++l;  // ceil(log2 d)
  f.m = (uint32_t)(((1ull << 32) * ((1ull << l) - d)) / d + 1);
  f.s = l - 1;
  return f;
}

FastDiv fast_div(uint32_t d) {
  FastDiv f;
  f.d = d;
  f.m = d == 1 ? 0u : (uint32_t)(((1ull << 32) + d - 1) / d);
  return f;
}

// Head shape and LDS layout for a reordering layout, from the stride (in
// vectors) of the head's strided LDS reads: a gather (cache image in LDS)
// reads paged-attention K vectors and V elements of consecutive dims at
// stride bs, and swizzles with shift log2 of that stride (at least 16)
// rounded up to a power of two; a scatter (packed image in LDS) reads them at
// stride v16 (K: consecutive tokens; V: the x tokens of one output vector)
// and pads every v16 (at least 8) vectors. HND uses no LDS.
SlabGeom slab_geom(const kvx_cache* c, bool to_packed) {
  const uint32_t bs = (uint32_t)c->block_size, h = (uint32_t)c->num_kv_heads,
                 d = (uint32_t)c->head_dim, x = (uint32_t)(16 / c->elem_bytes),
                 v16 = (uint32_t)((int64_t)c->head_dim * c->elem_bytes / 16);
  SlabGeom sg;
  sg.bs = fast_div(bs);
  sg.d = fast_div(d);
  sg.v16 = fast_div(v16 ? v16 : 1);
  sg.x = x;
  sg.nh = bs * v16;
  sg.prow = h * v16;
  // V of 2-byte words as row pairs in a gather: token pairs, so an even
  // block size (v_pairs_gather says why not in a scatter)
  sg.v_pairs = c->elem_bytes == 2 && to_packed && bs % 2 == 0 ? 1u : 0u;
  const uint32_t stride = to_packed ? bs : v16;
  sg.swz = 4;
  while ((1u << sg.swz) < stride) ++sg.swz;
  sg.pad = fast_div(stride < 8 ? 8 : stride);
  return sg;
}

}  // namespace

namespace {

// Per device: the table's device address and which stream owns each word.
// Fixed-size (no allocation), open addressing on the stream handle.
constexpr int kMaxDevices = 64;
struct ErrorTable {
  int* base = nullptr;
  hipStream_t owner[kErrorWords] = {};
  bool used[kErrorWords] = {};
};
ErrorTable g_tables[kMaxDevices];
std::mutex g_tables_mu;

}  // namespace

int* stream_error_word(hipStream_t stream) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_tables_mu);
  ErrorTable& t = g_tables[dev];
  if (!t.base) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(g_error_words)) != hipSuccess) return nullptr;
    t.base = (int*)p;
  }
  if (!stream) return t.base;
  const uint64_t h = (uint64_t)(uintptr_t)stream * 0x9E3779B97F4A7C15ull;
  uint32_t w = 1 + (uint32_t)(h >> 40) % (kErrorWords - 1);
  for (int probe = 0; probe < kErrorWords - 1; ++probe) {
    if (!t.used[w]) {
      t.used[w] = true;
      t.owner[w] = stream;
      return t.base + w;
    }
    if (t.owner[w] == stream) return t.base + w;
    w = w + 1 == (uint32_t)kErrorWords ? 1u : w + 1;
  }
  return t.base;  // table full: the shared word
}

kvx_status launch_copy(bool to_packed, const kvx_cache* cache, int32_t l0, int32_t l1,
                       const int32_t* block_table, const Geometry& g, void* packed,
                       hipStream_t stream, int* err, void* order_scratch) {
  if (g.n_units == 0) return KVX_OK;
  if (g.n_units > 0x7FFFFFFF || g.slab % 16 != 0) return KVX_EINTERNAL;
  if (!err) return KVX_EHIP;
  LayerPtrs lp = {};
  for (int32_t l = l0; l < l1; ++l) {
    lp.p[2 * (l - l0)] = static_cast<char*>(cache->k[l]);
    lp.p[2 * (l - l0) + 1] = static_cast<char*>(cache->v[l]);
  }
  Walk walk;
  const kvx_status ws = choose_walk(to_packed, cache, g, &walk);
  if (ws != KVX_OK) return ws;
  UnitGeom ug;
  ug.units_per_chunk = (uint32_t)(2 * g.lr * g.bpc);
  ug.bpc = (uint32_t)g.bpc;
  ug.n_blocks = (uint32_t)g.n_blocks;
  ug.num_blocks = (uint32_t)g.num_blocks;
  ug.n16 = (uint32_t)(g.slab / 16);
  const int layout = cache->layout, elem = cache->elem_bytes;
  ug.parts = walk.parts;
  ug.parts_shift = walk.parts_shift;
  ug.parts_div = div_u32(ug.parts);
  ug.upc_div = div_u32(ug.units_per_chunk);
  ug.bpc_div = div_u32(ug.bpc);
  ug.last_div = div_u32((uint32_t)(g.n_blocks - (g.n_blocks - 1) / g.bpc * g.bpc));
  ug.nb_div = div_u32(ug.n_blocks);
  ug.slab = (uint64_t)g.slab;
  ug.sg = slab_geom(cache, to_packed);
  const uint32_t n_work = walk.n_work;
  const uint32_t n_slices = (uint32_t)(2 * g.lr);
  ug.pair_shift = walk.pair_shift;
  ug.gather_pair_shift = walk.gather_pair_shift;
  ug.half_slices = n_slices / kXcds / 2;
  ug.linear_walk = walk.linear ? 1u : 0u;
  ug.xcd_slices_div = div_u32(n_slices / kXcds ? n_slices / kXcds : 1);
  if (to_packed) {
    hipError_t e = launch<true, false>(lp, block_table, ug, n_work, nullptr, (char*)packed, err,
                                       layout, elem, stream);
    return e == hipSuccess ? KVX_OK : KVX_EHIP;
  }
  // Destination-ordered scatter for large calls of multi-block chunks; the
  // order lives in the caller's scratch (order_scratch, n_blocks entries) or
  // else in stream-ordered scratch allocated here. If that allocation fails,
  // fall back to image order (same result, slower).
  OrderEntry* order = nullptr;
  const bool own = order_scratch == nullptr;
  if (walk.ordered) {
    if (!own)
      order = static_cast<OrderEntry*>(order_scratch);
    else if (hipMallocAsync((void**)&order, (size_t)g.n_blocks * sizeof(OrderEntry), stream) !=
             hipSuccess)
      order = nullptr;
  }
  (void)hipGetLastError();
  hipError_t e;
  if (order) {
    hipLaunchKernelGGL(order_kernel, dim3(1), dim3(kOrderThreads), 0, stream, block_table,
                       (uint32_t)g.n_blocks, (uint32_t)g.num_blocks, order);
    e = hipGetLastError();
    if (e == hipSuccess)
      e = launch<false, true>(lp, block_table, ug, n_work, order, (char*)packed, err, layout,
                              elem, stream);
    if (own) {
      const hipError_t ef = hipFreeAsync(order, stream);
      if (e == hipSuccess) e = ef;
    }
  } else {
    e = launch<false, false>(lp, block_table, ug, n_work, nullptr, (char*)packed, err, layout,
                             elem, stream);
  }
  return e == hipSuccess ? KVX_OK : KVX_EHIP;
}

kvx_status launch_copy_chunks(bool to_packed, const kvx_cache* cache, int32_t l0, int32_t l1,
                              const int32_t* block_table, int32_t table_len,
                              const kvx_chunk_ref* refs, int32_t n_chunks, int32_t chunk_tokens,
                              void* packed, int64_t packed_bytes, hipStream_t stream,
                              int* err) {
  if (n_chunks <= 0 || l1 <= l0) return KVX_OK;
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
  const int layout = cache->layout, elem = cache->elem_bytes;
  slab_parts(layout, cg.n16, (uint32_t)cache->num_kv_heads, &cg.parts, &cg.parts_shift);
  cg.parts_div = div_u32(cg.parts);
  cg.upc_div = div_u32(cg.upc);
  cg.bpc_div = div_u32(cg.bpc);
  cg.table_len = table_len;
  cg.slab = (uint64_t)slab;
  cg.packed_bytes = packed_bytes;
  cg.sg = slab_geom(cache, to_packed);
  if ((uint64_t)n_units * cg.parts > 0x7FFFFFFF) return KVX_EINTERNAL;
  const uint32_t n_work = (uint32_t)n_units * cg.parts;
  hipError_t e = to_packed ? launch_chunks<true>(lp, block_table, refs, cg, n_work,
                                                 (char*)packed, err, layout, elem, stream)
                           : launch_chunks<false>(lp, block_table, refs, cg, n_work,
                                                  (char*)packed, err, layout, elem, stream);
  return e == hipSuccess ? KVX_OK : KVX_EHIP;
}

}  // namespace kvx

// ---- scatter for callers that cannot allocate --------------------------------
//
// The order entries of a destination-ordered scatter live in this fixed array
// instead of stream-ordered scratch: each GPU the library runs on holds one
// copy (kvx::kNoAllocScratchBytes) until the process ends. Host code reaches a
// device's copy only through the address hipGetSymbolAddress returns for that
// device (resolved once per device, with the device current); the array's
// name on the host is not a device address.
static __device__ __align__(256) unsigned char scratch[kvx::kNoAllocScratchBytes];

namespace {

constexpr int kScratchDevices = 64;
void* g_scratch_ptr[kScratchDevices] = {};
std::mutex g_scratch_mu;

// The calling device's copy of `scratch`, or null.
void* device_scratch() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kScratchDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    g_scratch_ptr[dev] = p;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" kvx_status kvx_scatter_blocks_noalloc(const kvx_cache* cache, int32_t l0, int32_t l1,
                                                 const int32_t* block_table, int32_t n_blocks,
                                                 int32_t chunk_tokens, const void* src,
                                                 hipStream_t stream) {
  try {
    kvx::Geometry g;
    kvx_status st = kvx::validate(cache, l0, l1, n_blocks, chunk_tokens, true, &g);
    if (st != KVX_OK) return st;
    if (n_blocks > KVX_NOALLOC_MAX_BLOCKS) return KVX_EINVAL;
    if (g.n_units == 0) return KVX_OK;
    if (!block_table || !src || ((uintptr_t)src & 15)) return KVX_EINVAL;
    if (kvx::overlaps_cache(cache, l0, l1, src, g.packed)) return KVX_EINVAL;
    void* order = device_scratch();
    int* err = kvx::stream_error_word(stream);
    if (!order || !err) return KVX_EHIP;
    return kvx::launch_copy(false, cache, l0, l1, block_table, g, const_cast<void*>(src), stream,
                            err, order);
  } catch (...) {
    return KVX_EINTERNAL;
  }
}

