/*
 * kvx.h -- C ABI of libkvx.so: moving prefix KV state between a paged GPU KV
 * cache and contiguous transfer chunks on one MI355X (gfx950).
 *
 * What the operations are (from the paper's statement of the problem):
 *   - The serving engine keeps KV in fixed-size token blocks; the blocks of
 *     one prompt are not adjacent in memory (Sec. 2.1, "KV Cache in LLM
 *     Serving"). Size model: bytes per token = layers x 2 x KV heads x head
 *     dim x dtype size (Sec. 2.1).
 *   - The external cache transfers "storage blocks" that each group several
 *     GPU blocks (Sec. 6.4); a batched block copy moves data between the GPU
 *     KV tensors and contiguous staging slots (Secs. 6.2, 6.4). Here that copy
 *     is a gather (paged -> packed chunks, for offload) and a scatter (packed
 *     chunks -> paged, for load).
 *   - Staging is one contiguous, aligned, pinned host allocation cut into
 *     fixed slots; a transfer larger than the pool goes through it piece by
 *     piece, and a slot is reused only after the GPU copy that read it has
 *     completed, as reported by a device event (Sec. 6.4). That is
 *     kvx_restore_from_staging.
 *
 * Layouts (the paper gives none; these are this library's definitions):
 *   Cache   per layer l, separate K and V device tensors, each contiguous
 *           [num_blocks][block_size][num_kv_heads][head_dim] of elem_bytes-byte
 *           words. A slab is one (layer, K|V, block):
 *           slab = block_size * num_kv_heads * head_dim * elem_bytes bytes.
 *   Chunk   chunk_tokens must be a positive multiple of block_size; a chunk
 *           holds bpc = chunk_tokens / block_size consecutive entries of the
 *           block table. Inside a chunk the order is [layer l0..l1-1][K, V]
 *           [token][head][dim]: for each (layer, K|V) the chunk's slabs are
 *           adjacent, in block-table order.
 *   Image   the packed image of n blocks over layers [l0, l1) is the chunks
 *           back to back. The last chunk may hold fewer than bpc blocks and
 *           is compact, so the image is exactly
 *           n * (l1 - l0) * 2 * slab bytes with no padding.
 *
 * Asynchrony: gather and scatter validate, enqueue on the caller's stream and
 * return; results are defined once that stream has completed. Block ids live
 * in device memory and are checked by the kernels: a unit whose id is outside
 * [0, num_blocks) is skipped (nothing is written for it) and a sticky error
 * word of the stream the call was given is set, which kvx_check() on that
 * stream reports as KVX_EBADBLOCK.
 * Scatter destinations must be distinct; duplicates make the result depend
 * on execution order (not checked).
 *
 * Ownership: the caller owns every cache tensor, block table, packed buffer,
 * landing buffer, host source and stream passed in. The library never frees
 * caller memory and keeps no pointer to kvx_cache's arrays after a call
 * returns (kvx_ring_bind copies what it needs). A ring owns its pinned slot
 * allocation, its side stream, its events and its fill threads.
 *
 * Threading: gather, scatter and kvx_check may be called from any thread. A
 * ring is used by one thread at a time.
 *
 * No C++ exception crosses this interface.
 */
#ifndef KVX_H_
#define KVX_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum kvx_status {
  KVX_OK = 0,
  KVX_EINVAL = -1,     /* bad argument (detected on the host, nothing enqueued) */
  KVX_ENOMEM = -2,     /* a host or device allocation failed */
  KVX_EHIP = -3,       /* a HIP runtime call failed */
  KVX_EBADBLOCK = -4,  /* a kernel met a block id outside [0, num_blocks) */
  KVX_ECLOSED = -5,    /* the ring was aborted while a restore was running */
  KVX_EINTERNAL = -6,  /* invariant violated inside the library */
  KVX_EIO = -7,        /* a storage-tier file could not be opened, read, written or published */
  KVX_EBUSY = -8       /* the ring is running a transfer started by kvx_offload_begin or
                          kvx_restore_begin */
} kvx_status;

/* Largest layer range a single call may cover. */
#define KVX_MAX_LAYERS 128

/* Cache tensor layouts (per layer; the packed chunk layout is the same for
 * all of them, [token][head][dim] inside each (layer, K|V)):
 *   KVX_LAYOUT_NHD         K and V [num_blocks][block_size][num_kv_heads][head_dim]
 *   KVX_LAYOUT_HND         K and V [num_blocks][num_kv_heads][block_size][head_dim]
 *   KVX_LAYOUT_PAGED_ATTN  K [num_blocks][num_kv_heads][head_dim / x][block_size][x]
 *                          with x = 16 / elem_bytes, V [num_blocks][num_kv_heads]
 *                          [head_dim][block_size] (the paged-attention kernel layout)
 * The two reordering layouts move a slab head by head (paged attention through
 * LDS) and need head_dim * elem_bytes to be a multiple of 16 and a slab of at
 * most 48 KiB. */
#define KVX_LAYOUT_NHD 0
#define KVX_LAYOUT_HND 1
#define KVX_LAYOUT_PAGED_ATTN 2

/* Description of a paged cache. k and v are host arrays of num_layers device
 * pointers (16-byte aligned); they are read during the call only. */
typedef struct kvx_cache {
  void* const* k;
  void* const* v;
  int32_t num_layers;
  int32_t num_blocks;
  int32_t block_size;    /* tokens per GPU block */
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t elem_bytes;    /* 1, 2, 4 or 8; the path copies raw words */
  int32_t layout;        /* KVX_LAYOUT_*; 0 is the default */
} kvx_cache;

/* Size model of Sec. 2.1: layers * 2 * kv_heads * head_dim * elem_bytes.
 * Returns -1 if any argument is not positive. */
int64_t kvx_bytes_per_token(int32_t layers, int32_t kv_heads, int32_t head_dim,
                            int32_t elem_bytes);

/* Bytes of the packed image of n_blocks blocks over layers [l0, l1):
 * n_blocks * (l1 - l0) * 2 * slab. Returns -1 on an invalid shape or range. */
int64_t kvx_packed_bytes(const kvx_cache* cache, int32_t l0, int32_t l1, int32_t n_blocks);

/* Byte distance between the starts of consecutive chunks of a packed image:
 * the size of a full chunk, (l1 - l0) * 2 * chunk_tokens * row bytes with
 * row = num_kv_heads * head_dim * elem_bytes (Sec. 6.4: a storage block
 * groups chunk_tokens / block_size GPU blocks). Chunk c starts at c times
 * this; only the last chunk of an image may be shorter. Returns -1 on an
 * invalid shape or range, or chunk_tokens not a positive multiple of
 * block_size. Cache pointers are not read. */
int64_t kvx_chunk_stride(const kvx_cache* cache, int32_t l0, int32_t l1, int32_t chunk_tokens);

/* Gather (offload side): for every chunk c, layer l in [l0, l1), K|V and block
 * j of the chunk, copy slab cache[l][K|V][block_table[c*bpc + j]] to its place
 * in the packed image at dst (layout above).
 *   block_table  device int32[n_blocks]; ids may repeat (read-only side)
 *   dst          device, 16-byte aligned, kvx_packed_bytes(...) bytes; must
 *                not overlap any cache tensor
 *   stream       HIP stream to enqueue on (0 = the null stream)
 * n_blocks == 0 or l0 == l1 is a no-op returning KVX_OK.
 * Errors: KVX_EINVAL for a null or misaligned pointer, l0 < 0, l1 < l0,
 * l1 > num_layers, l1 - l0 > KVX_MAX_LAYERS, chunk_tokens not a positive
 * multiple of block_size, slab not a multiple of 16 bytes, dst overlapping
 * the cache, or a call of more than 2^31 - 1 slabs or workgroups (slabs x
 * parts per slab: its 4 KiB pieces with the default layout, its heads with
 * the others); KVX_EHIP if the launch fails. Bad block ids: see kvx_check. */
kvx_status kvx_gather_blocks(const kvx_cache* cache, int32_t l0, int32_t l1,
                             const int32_t* block_table, int32_t n_blocks, int32_t chunk_tokens,
                             void* dst, hipStream_t stream);

/* Scatter (load side): the inverse of kvx_gather_blocks. Every slab the image
 * names is written; no other cache byte changes. block_table holds distinct
 * destination ids. Arguments and errors as for kvx_gather_blocks, with src
 * (device, 16-byte aligned, kvx_packed_bytes(...) bytes) read instead of dst
 * written. */
kvx_status kvx_scatter_blocks(const kvx_cache* cache, int32_t l0, int32_t l1,
                              const int32_t* block_table, int32_t n_blocks, int32_t chunk_tokens,
                              const void* src, hipStream_t stream);

/* How kvx_gather_blocks (to_packed = 1) or kvx_scatter_blocks (0) with these
 * arguments walks its work: the launcher's own choice, reported for tests and
 * measurement records. Pure host code: the cache's tensor pointers may be
 * NULL. A call moves work_items workgroups; each moves one part of a slab
 * (parts per slab: 4 KiB pieces with the default layout, heads with the
 * others). A scatter of 1,024 blocks or more in chunks of more than one block
 * runs in ascending destination order (ordered = 1; block ids bucketed by a
 * small kernel first), except with slabs of at most 8 KiB in the default
 * layout (or a reordering layout with one KV head): those, like every smaller
 * scatter, walk
 * the packed image in order, with linear = 1 when workgroup b moves work item
 * b rather than each XCD taking one contiguous range. pair_slices = D > 0:
 * slices D apart, whose runs sit 2 MiB apart in a packed chunk, are moved
 * together (the gather's paired walk, or an ordered scatter's two fronts per
 * XCD: fronts = 2). For an empty call every field is 0. KVX_EINVAL for the
 * arguments the copy calls reject on the host (except pointers). */
typedef struct kvx_walk {
  int64_t work_items;
  int32_t parts;
  int32_t ordered;
  int32_t linear;
  int32_t pair_slices;
  int32_t fronts;
  int32_t reserved;
} kvx_walk;

kvx_status kvx_copy_walk(const kvx_cache* cache, int32_t l0, int32_t l1, int32_t n_blocks,
                         int32_t chunk_tokens, int32_t to_packed, kvx_walk* out);

/* Largest n_blocks of kvx_scatter_blocks_noalloc. */
#define KVX_NOALLOC_MAX_BLOCKS 65536

/* kvx_scatter_blocks for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same arguments, validation, kernels and result, but the
 * destination order that a scatter of 1,024 blocks or more computes first (in
 * chunks of more than one block, and with the default layout, or a
 * reordering layout with one KV head, only for slabs above 8 KiB) lives in
 * a fixed device array of the library's (512 KiB, KVX_NOALLOC_MAX_BLOCKS
 * 8-byte entries; each GPU the library runs on holds one until the process
 * ends) instead of stream-ordered scratch. The call allocates nothing.
 * n_blocks above KVX_NOALLOC_MAX_BLOCKS returns KVX_EINVAL before anything is
 * enqueued. Every call on one GPU shares that GPU's array, and each call
 * rewrites the entries it uses before reading them: calls that may overlap on
 * one GPU (other streams, or other threads) race on it and must be ordered by
 * the caller. */
kvx_status kvx_scatter_blocks_noalloc(const kvx_cache* cache, int32_t l0, int32_t l1,
                                      const int32_t* block_table, int32_t n_blocks,
                                      int32_t chunk_tokens, const void* src, hipStream_t stream);

/* ---- batched chunk lists (several requests in one launch) ------------------ */

/* One chunk of a batch: the packed image of blocks block_table[bt_offset ..
 * bt_offset + n_blocks) over the call's layer range, laid out as one chunk
 * (1 <= n_blocks <= chunk_tokens / block_size), at byte packed_offset of the
 * packed buffer (16-byte aligned). Chunks may come from different requests
 * and sit anywhere in the packed buffer; they must not overlap there. */
typedef struct kvx_chunk_ref {
  int64_t packed_offset;
  int32_t bt_offset;
  int32_t n_blocks;
} kvx_chunk_ref;

/* Batched gather: every chunk of `chunks` (a device array of n_chunks refs) is
 * gathered into the packed buffer in one launch. This is the paper's fused
 * batched block copy: the ready mappings of several requests moved by a single
 * launch (Sec. 6.4).
 *   block_table  device int32[table_len]
 *   packed       device, 16-byte aligned, packed_bytes bytes; must not
 *                overlap any cache tensor
 * Host-checkable errors as for kvx_gather_blocks (KVX_EINVAL), plus a launch
 * too large for 32-bit unit indexes (n_chunks * (l1 - l0) * 2 * blocks per
 * chunk >= 2^31). The refs live on the device and are checked by the kernel:
 * a ref with n_blocks out of range, a block-table slice past table_len, or an
 * image that is misaligned or does not fit in packed_bytes is skipped and
 * makes kvx_check return KVX_EINVAL. Bad block ids: KVX_EBADBLOCK. */
kvx_status kvx_gather_chunks(const kvx_cache* cache, int32_t l0, int32_t l1,
                             const int32_t* block_table, int32_t table_len,
                             const kvx_chunk_ref* chunks, int32_t n_chunks, int32_t chunk_tokens,
                             void* packed, int64_t packed_bytes, hipStream_t stream);

/* Batched scatter: the inverse of kvx_gather_chunks. Destinations of all
 * chunks must be distinct. */
kvx_status kvx_scatter_chunks(const kvx_cache* cache, int32_t l0, int32_t l1,
                              const int32_t* block_table, int32_t table_len,
                              const kvx_chunk_ref* chunks, int32_t n_chunks, int32_t chunk_tokens,
                              const void* packed, int64_t packed_bytes, hipStream_t stream);

/* Wait for `stream`, then read and clear its sticky error word on the calling
 * device: KVX_EINVAL if a kernel of a call given this stream met an invalid
 * device-resident chunk reference, else KVX_EBADBLOCK if one met a bad block
 * id, KVX_EHIP if the stream reported an error, else KVX_OK. Each stream has a
 * word of its own (errors on one stream are never reported to, or cleared by,
 * a check of another), kept in a fixed table of 1,024 words per device: the
 * null stream and streams beyond the first 1,023 distinct handles seen on a
 * device share the table's first word. Work a ring or a deferred call runs on
 * a stream of its own reports to the stream the caller passed. An error left
 * unchecked when a stream is destroyed is reported to a later stream that
 * receives the same handle. */
kvx_status kvx_check(hipStream_t stream);

const char* kvx_strerror(kvx_status status);

/* ---- staging ring (Sec. 6.4) ---------------------------------------------- */

/* One piece of a staged transfer: the image bytes [src_offset, src_offset +
 * bytes) hold the packed image of blocks block_table[bt_first ..
 * bt_first + n_blocks) over layers [l_begin, l_end) with chunk size
 * chunk_tokens (a piece is either a run of whole chunks or a layer range of
 * one chunk). chunk_tokens is the call's, or the prefix's length where the
 * prefix is shorter than one chunk (the two images are the same bytes). */
typedef struct kvx_piece {
  int64_t src_offset;
  int64_t bytes;
  int32_t bt_first;
  int32_t n_blocks;
  int32_t l_begin;
  int32_t l_end;
  int32_t chunk_tokens;
  int32_t n_spans;  /* host-link copies the piece takes (runs of chunks adjacent in the image) */
} kvx_piece;

/* Where a plan's piece sizes ramp up to the slot size. */
#define KVX_RAMP_NONE 0   /* every piece up to slot_bytes */
#define KVX_RAMP_FIRST 1  /* the first piece at most 1/8 of a slot, each next one at
                             most twice the piece before it, until a piece may fill a
                             slot (a restore: its first copy starts after a small
                             fill, and each fill finishes while the copy before it
                             still runs) */
#define KVX_RAMP_LAST 2   /* the same ramp from the last piece backwards (an offload:
                             its last copy and drain are short); the pieces of the
                             first-ramp plan of the reversed chunk list, in reverse
                             order, each carrying its chunks in image order */

/* Split the packed image of (cache shape, [l0, l1), n_blocks, chunk_tokens)
 * into pieces: as many consecutive whole chunks per piece as fit its size
 * limit (slot_bytes, or less under the ramp); a chunk larger than its piece's
 * limit is split into contiguous layer ranges, as many layers per piece as its
 * limit allows (at least one), and the next chunk starts a new piece. So a
 * ramped piece may hold less than its limit. This is the planner the ring
 * runs (kvx_ring_bind: KVX_RAMP_FIRST for restores, KVX_RAMP_LAST for
 * offloads). Pure host computation (no HIP call). Writes at most max_pieces
 * entries to out (out may be NULL to count) and the total count to *n_pieces.
 * KVX_EINVAL if a single layer of a chunk exceeds slot_bytes, ramp is not a
 * KVX_RAMP_* value or the arguments are invalid (cache pointers are not
 * read). */
kvx_status kvx_plan_pieces(const kvx_cache* cache, int32_t l0, int32_t l1, int32_t n_blocks,
                           int32_t chunk_tokens, int64_t slot_bytes, int32_t ramp, kvx_piece* out,
                           int32_t max_pieces, int32_t* n_pieces);

typedef struct kvx_ring kvx_ring;

/* Create a ring on `device` with n_slots (>= 1) slots of slot_bytes (a
 * positive multiple of 4096): one hipHostMalloc allocation of
 * n_slots * slot_bytes pinned bytes, one non-blocking side stream at default
 * priority, per-slot events and, where the HSA runtime exposes the GPU's DMA
 * engines, per-slot completion signals. The first ring created on a device in
 * the process also times the engines (about 0.2 s where all 16 engines are
 * candidates, on 32 MiB device and 32 MiB pinned buffers of its own, freed
 * afterwards). device_landing is the
 * device buffer that H2D copies land in (n_slots * slot_bytes bytes, 16-byte
 * aligned, owned by the caller); NULL makes the ring allocate its own. The
 * ring's fill (restore) or drain (offload) threads are started by the first
 * transfer that needs them and kept, parked between transfers, until
 * kvx_ring_destroy (a bind that changes their direction or count replaces
 * them at the next transfer). */
kvx_status kvx_ring_create(int device, int32_t n_slots, int64_t slot_bytes, void* device_landing,
                           kvx_ring** out);

/* Bind the next restores to a transfer: cache (pointers copied), layer
 * range, prefix length, chunk size, the host image (packed layout,
 * kvx_packed_bytes(...) bytes; it stands in for the storage tier and is read
 * only) and the number of host fill threads (1..64) that copy image pieces
 * into staging slots. fill_threads == 0 skips staging: the H2D copies then
 * read the image directly, which must be pinned (the preloaded case, where
 * the data already sits in pinned memory). Plans the pieces as
 * kvx_plan_pieces does with KVX_RAMP_FIRST: a restore's first piece holds at
 * most 1/8 of a slot and each next one at most twice the piece before it
 * (larger chunks cut into layer ranges) until a piece may fill a slot, so its
 * first host-to-device copy starts after a small first fill;
 * offloads (kvx_ring_bind_offload) plan with KVX_RAMP_LAST. */
kvx_status kvx_ring_bind(kvx_ring* ring, const kvx_cache* cache, int32_t l0, int32_t l1,
                         int32_t n_blocks, int32_t chunk_tokens, const void* host_source,
                         int32_t fill_threads);

/* Restore the bound image into the blocks named by block_table (device
 * int32[n_blocks], distinct destination ids). For piece i on slot s = i mod
 * n_slots: fill threads copy the piece into host slot s once the H2D copy of
 * piece i - n_slots has completed; once the scatter of piece i - n_slots has
 * finished reading device slot s, host slot s is copied to device slot s by a
 * DMA engine; once the host has seen that copy complete, `stream` runs the
 * scatter of the piece (the copy of piece i + 1 is issued before that wait,
 * so the engine never idles). Returns once every piece's scatter is enqueued
 * (the host thread waits for fill threads and for the copies, not for the
 * scatters); all scatters are ordered on `stream`. Without DMA engines (see
 * kvx_ring_stats.dma) the copies go through the HIP runtime on the side
 * stream, ordered by events, and the call returns once every piece is
 * enqueued without waiting for the device. The cache equals the scatter of
 * the whole image once `stream` completes. KVX_ECLOSED if kvx_ring_abort was
 * called; scatters already enqueued still complete. */
kvx_status kvx_restore_from_staging(kvx_ring* ring, const int32_t* block_table,
                                    hipStream_t stream);

/* A chunk image in host memory: the packed image of one chunk (layout above,
 * over the binding's layer range) of the blocks block_table[bt_offset ..
 * bt_offset + n_blocks), 1 <= n_blocks <= chunk_tokens / block_size. For a
 * restore, host is the source (stands in for the storage read); for an
 * offload, the destination (stands in for the storage write). */
typedef struct kvx_host_chunk {
  void* host;
  int32_t bt_offset;
  int32_t n_blocks;
} kvx_host_chunk;

/* Bind the next restores to a list of chunk images, each at its own host
 * address (the deduplicated chunks of several requests, Sec. 6.5: identical
 * prefixes share one read). Pieces pack consecutive chunks into slots; every
 * piece is scattered by one fused chunk-list launch. The block table passed to
 * kvx_restore_from_staging must hold at least max(bt_offset + n_blocks)
 * entries. fill_threads as for kvx_ring_bind (0: the chunk images must be
 * pinned). Waits until the ring's previous transfer has finished on the
 * device (its chunk table is replaced). */
kvx_status kvx_ring_bind_chunks(kvx_ring* ring, const kvx_cache* cache, int32_t l0, int32_t l1,
                                int32_t chunk_tokens, const kvx_host_chunk* chunks,
                                int32_t n_chunks, int32_t fill_threads);

/* Bind the next offloads: the store path, the mirror of a restore (Sec. 6.4,
 * stores use the reverse pipeline). Each chunk's blocks are gathered and its
 * image written to the chunk's host address. drain_threads (1..64) copy
 * staging slots to the destinations; 0 copies device slots straight into the
 * destinations, which must then be pinned. */
kvx_status kvx_ring_bind_offload(kvx_ring* ring, const kvx_cache* cache, int32_t l0, int32_t l1,
                                 int32_t chunk_tokens, const kvx_host_chunk* chunks,
                                 int32_t n_chunks, int32_t drain_threads);

/* Offload the bound chunks, reading the blocks named by block_table (device).
 * For piece i on slot s = i mod n_slots: once the copy of piece i - n_slots
 * has left device slot s, `stream` gathers the piece into it (one fused
 * launch) and records an event; once that event has completed and the drain
 * threads have emptied host slot s, device slot s is copied to host slot s by
 * a DMA engine (without DMA engines: by the HIP runtime on the side stream);
 * drain threads copy host slot s to the chunks' destinations once that copy
 * has completed. Returns when every destination holds its image (it waits for
 * the device). KVX_ECLOSED after kvx_ring_abort. */
kvx_status kvx_offload_to_staging(kvx_ring* ring, const int32_t* block_table, hipStream_t stream);

/* Deferred store (Secs. 2.3, 5.1: the offload API defers the store work of
 * engine iteration N to iteration N + 1, so the copies to the host overlap
 * the next forward pass): start the offload of the bound chunks on a thread
 * the ring owns and return at once. The gathers run after the work already
 * enqueued on `stream`, on a stream the ring owns with a hardware queue of
 * its own (created with a compute-unit mask covering every compute unit: the
 * runtime shares a few hardware queues round-robin among streams, and a store
 * whose stream shared the forward pass's queue waited behind all of it).
 * Like any stream created without the non-blocking flag it is ordered
 * against the legacy default stream, so the forward pass it should overlap
 * must run on another stream. The copies to the host run on the DMA engine
 * and the drains on the drain threads, as in kvx_offload_to_staging. Until
 * kvx_offload_wait has returned, every other call on the ring except
 * kvx_ring_abort and kvx_ring_destroy returns KVX_EBUSY, and block_table and
 * the destinations must stay valid. Argument errors found before the start
 * are returned here; errors of the transfer by kvx_offload_wait. */
kvx_status kvx_offload_begin(kvx_ring* ring, const int32_t* block_table, hipStream_t stream);

/* Wait for the offload started by kvx_offload_begin and return its status
 * (KVX_OK at once if none was started). On return every destination holds
 * its image, as after kvx_offload_to_staging. Bad block ids met by its
 * gathers are reported by kvx_check on the stream given to kvx_offload_begin. */
kvx_status kvx_offload_wait(kvx_ring* ring);

/* Asynchronous restore (Sec. 6.4: the worker turns load plans into transfers
 * without blocking the engine; Sec. 6.2): start the restore of the bound
 * transfer into the blocks named by block_table on a thread the ring owns
 * (started by the first begin on the ring and kept until kvx_ring_destroy),
 * and return at once. Its scatters run after the work already enqueued on
 * `stream`, on a stream the ring owns; fills, host-link copies and slot reuse
 * are those of kvx_restore_from_staging. Until kvx_restore_wait has returned,
 * every other call on the ring except kvx_ring_abort and kvx_ring_destroy
 * returns KVX_EBUSY, and block_table and the bound sources must stay valid.
 * Argument errors found before the start are returned here; errors of the
 * transfer by kvx_restore_wait; bad block ids by kvx_check on `stream`. */
kvx_status kvx_restore_begin(kvx_ring* ring, const int32_t* block_table, hipStream_t stream);

/* Wait until the restore started by kvx_restore_begin has enqueued every
 * scatter, then order `stream` after all of them (no host wait for the
 * device): work enqueued on `stream` after this call sees the restored
 * blocks. Returns the transfer's status (KVX_OK at once if none was started;
 * KVX_ECLOSED after kvx_ring_abort). */
kvx_status kvx_restore_wait(kvx_ring* ring, hipStream_t stream);

typedef struct kvx_ring_stats {
  int64_t pieces;         /* pieces moved by the last restore or offload */
  int64_t bytes;          /* image bytes moved by it */
  double fill_ms;         /* summed fill (restore) or drain (offload) thread copy time */
  double wait_fill_ms;    /* time the enqueuing thread waited for fill or drain threads */
  double enqueue_ms;      /* wall time of the last restore or offload call */
  int32_t dma;            /* 1: the last transfer's host-link copies were issued to the GPU's
                             DMA engines directly; 0: through the HIP runtime on the side
                             stream (which may run a device-to-host copy as a copy kernel on
                             compute units) */
  int32_t dma_engine;     /* with dma: the engine id bit of that direction (restore: H2D,
                             offload: D2H). The device's pair is timed by the first ring
                             created on it in the process: of the runtime's preferred (else
                             available) engines, those fast alone in each direction, and of
                             those the D2H / H2D pair fastest running at once. 0 = the
                             runtime's own choice */
} kvx_ring_stats;

kvx_status kvx_ring_stats_get(const kvx_ring* ring, kvx_ring_stats* out);

/* ---- transfer timeline ---------------------------------------------------------- *
 *
 * The paper traces its connector with a profiler whose timeline shows storage
 * reads interleaved with GPU transfers (Sec. 4.1, the trace sample). A ring
 * with tracing on records, for its transfers, one interval per:
 *   KVX_TRACE_FILL     a fill thread copying its share of a piece into the
 *                      piece's pinned slot (restore; lane = the thread);
 *   KVX_TRACE_DRAIN    a drain thread copying its share out of the slot
 *                      (offload; lane = the thread);
 *   KVX_TRACE_WAIT     the enqueuing thread waiting for a piece's fill or
 *                      drain threads;
 *   KVX_TRACE_H2D      a piece's host-to-device copy (restore);
 *   KVX_TRACE_D2H      a piece's device-to-host copy (offload);
 *   KVX_TRACE_SCATTER  a piece's fused scatter launch (restore);
 *   KVX_TRACE_GATHER   a piece's fused gather launch (offload).
 * Times are nanoseconds of the host's monotonic clock (CLOCK_MONOTONIC, the
 * clock of std::chrono::steady_clock and Python's time.monotonic_ns), so host
 * events of the caller line up with them. Copies on the DMA engines carry the
 * engine's own start and end (HSA async-copy timestamps, converted from the
 * HSA system clock sampled at the transfer's start); copies through the HIP
 * runtime and the launches carry timing events, placed on the host clock by a
 * reference event that the transfer records and waits for before its first
 * piece (so a traced transfer first waits for work already queued on its
 * stream, and device intervals may be off by the few microseconds between
 * that event completing and the host seeing it). A DMA copy issued as several
 * copies (a piece of several host spans, no fill or drain threads) has no
 * H2D / D2H interval. Transfers bound to chunk files record no fill or drain
 * intervals (the reactor's reads and writes are not traced). */
#define KVX_TRACE_FILL 1
#define KVX_TRACE_DRAIN 2
#define KVX_TRACE_WAIT 3
#define KVX_TRACE_H2D 4
#define KVX_TRACE_D2H 5
#define KVX_TRACE_SCATTER 6
#define KVX_TRACE_GATHER 7

typedef struct kvx_trace_event {
  int32_t kind;    /* KVX_TRACE_* */
  int32_t piece;   /* piece index within the transfer */
  int32_t lane;    /* fill / drain thread; 0 for the others */
  int32_t slot;    /* staging slot of the piece */
  int64_t bytes;   /* bytes the interval moved (0 for KVX_TRACE_WAIT) */
  int64_t t0_ns;   /* start and end, host monotonic clock */
  int64_t t1_ns;
} kvx_trace_event;

/* Turn recording of the timeline on (enable = 1) or off (0) for this ring's
 * next transfers; each transfer replaces the previous one's record. While any
 * ring in the process traces, copies on the DMA engines are profiled (HSA
 * async-copy profiling, process-wide). KVX_EBUSY during an asynchronous
 * transfer. */
kvx_status kvx_ring_set_trace(kvx_ring* ring, int32_t enable);

/* The last traced transfer's intervals, ordered by start: up to cap of them
 * into out (caller-owned; out may be null with cap 0), their total count into
 * *n. Waits until that transfer's traced launches and copies have finished.
 * KVX_EBUSY during an asynchronous transfer; *n = 0 if the last transfer was
 * not traced or failed. */
kvx_status kvx_ring_trace_get(kvx_ring* ring, kvx_trace_event* out, int32_t cap, int32_t* n);

/* Make a running or later restore on this ring return KVX_ECLOSED. Safe to
 * call from another thread. */
kvx_status kvx_ring_abort(kvx_ring* ring);

/* ---- storage tier (files) ------------------------------------------------------ *
 *
 * One file per chunk (storage block, Sec. 6.4) holding the chunk's packed
 * image. Files are read and written by one reactor thread through io_uring
 * with at most io_depth transfers in flight (Sec. 6.4: the I/O depth, not a
 * thread count, sets storage concurrency), with O_DIRECT wherever every
 * transfer on a file is 4 KiB aligned (Sec. 6.3). A written file is published
 * by hard-linking a uniquely named temporary file in the same directory to the
 * final name and removing the temporary name: atomic, and first-writer-wins if
 * the name already exists (then the existing file is kept and the call still
 * succeeds), so a reader of a final name sees a whole file or none (Sec. 6.3).
 * Files are not fsync'ed. Where io_uring is unavailable, or KVX_IO_NO_URING=1
 * is set in the environment, the same calls run one blocking pread / pwrite at
 * a time. */

typedef struct {
  const char* path;   /* the chunk's file (copied at bind) */
  int32_t bt_offset;  /* first entry of the chunk in the transfer's block table */
  int32_t n_blocks;   /* 1 .. chunk_tokens / block_size */
} kvx_file_chunk;

/* Bind the next restores to chunk files: as kvx_ring_bind_chunks, with each
 * chunk's image read from its file (its whole size: (l1 - l0) * 2 * n_blocks
 * * slab bytes) into the staging slots by the reactor instead of fill
 * threads; a slot is read into only after its previous H2D copy completed.
 * io_depth 1..256. A missing or short file makes the restore return KVX_EIO
 * (slots already scattered stay scattered). */
kvx_status kvx_ring_bind_files(kvx_ring* ring, const kvx_cache* cache, int32_t l0, int32_t l1,
                               int32_t chunk_tokens, const kvx_file_chunk* chunks,
                               int32_t n_chunks, int32_t io_depth);

/* Bind the next offloads to chunk files: as kvx_ring_bind_offload, with each
 * chunk's image written from the staging slots to its file and published once
 * complete (missing directories are created). io_depth 1..256. */
kvx_status kvx_ring_bind_offload_files(kvx_ring* ring, const kvx_cache* cache, int32_t l0,
                                       int32_t l1, int32_t chunk_tokens,
                                       const kvx_file_chunk* chunks, int32_t n_chunks,
                                       int32_t io_depth);

/* Hash-addressed chunk path (Sec. 6.3: the path follows from the model
 * configuration and the prefix hash, intermediate directories spread the
 * entries): "<root>/<tag>/<k0>/<k1>/<key>.kvc" with k0, k1 the top two bytes of
 * key in hex and key as 16 hex digits; tag names the model configuration and
 * holds no '/'. Writes the NUL-terminated path to out[cap] and returns its
 * length, or -1 on a bad argument or a path longer than cap - 1. */
int32_t kvx_chunk_path(const char* root, const char* tag, uint64_t key, char* out, int32_t cap);

/* One host-side transfer of the storage tier: bytes [offset, offset + bytes)
 * of the file at path from / into buf (caller-owned host memory). */
typedef struct {
  const char* path;
  void* buf;
  int64_t offset;
  int64_t bytes;
} kvx_file_io;

/* Read every op's byte range of its file into its buffer (ops naming one path
 * share one open file), io_depth 1..256 in flight; returns when all are done.
 * KVX_EIO if a file is missing or shorter than an op needs. */
kvx_status kvx_read_files(const kvx_file_io* ops, int32_t n, int32_t io_depth);

/* Write and publish whole files: the ops naming one path must tile [0, size)
 * of that file exactly (KVX_EINVAL otherwise); each file is published as
 * above once all of its bytes are written. */
kvx_status kvx_write_files(const kvx_file_io* ops, int32_t n, int32_t io_depth);

/* ---- preloading (Sec. 6.5) ------------------------------------------------------ *
 *
 * Chunk files of requests that are still waiting are read ahead of time into a
 * bounded pool of host slots (one chunk file per slot), so that when such a
 * request runs only the host-to-device copy is left on its path: its demand
 * fetch claims the staged images, which a ring restores straight from the pool
 * (kvx_ring_bind_chunks with fill_threads 0). One reactor thread reads files
 * in 32 MiB pieces through io_uring, at most io_depth in flight, and always
 * serves demand before speculation: speculative pieces are issued only while
 * no demand file has pieces left to issue; one preload runs at a time (the
 * files of one kvx_preload_hint call, read concurrently; the next call's
 * files start when none of them is left), and speculative reads take only
 * slots beyond the `reserve` free ones. A file is
 * read at most once while staged: hints for a known file are dropped, and a
 * fetch claims its image or joins its read. Released images stay staged, so
 * the pool also caches chunk images: a speculative read may take the slot of
 * a cached image nobody holds (least recently used first) but never that of a
 * preloaded image not yet fetched; a demand fetch may take either, cached
 * images first. Files are read
 * buffered into a pinned pool (pinned memory cannot take direct transfers on
 * this platform) and their pages dropped from the page cache after reading.
 * The calls are thread-safe; kvx_preloader_destroy must not run concurrently
 * with another call on the same preloader. */
typedef struct kvx_preloader kvx_preloader;

typedef struct kvx_preload_stats {
  int64_t hints;           /* files queued by kvx_preload_hint */
  int64_t spec_deduped;    /* hints for a file already staged, being read or queued */
  int64_t spec_dropped;    /* hints refused: n_slots files already queued */
  int64_t spec_reads;      /* files read speculatively to completion */
  int64_t demand_fetches;  /* distinct files requested by kvx_preload_fetch */
  int64_t hits_ready;      /* of those, already staged */
  int64_t hits_inflight;   /* of those, joined a speculative read in progress */
  int64_t demand_reads;    /* files whose read completed as demand work */
  int64_t evictions;       /* staged files whose slot was taken for another file */
  int64_t spec_preempted;  /* speculative reads stopped to give their slot to a demand file
                              (the file is queued to be read again) */
  int64_t bytes_read;      /* file bytes read into the pool */
  int64_t staged;          /* files staged now */
  int64_t held;            /* files held by fetches now */
} kvx_preload_stats;

/* n_slots slots of slot_bytes (a positive multiple of 4096; a chunk file must
 * fit one slot), io_depth 1..256 pieces in flight, reserve 0..n_slots-1 slots
 * kept free of speculative reads; pinned 1 allocates the pool with
 * hipHostMalloc (needed to restore from it), 0 with plain aligned memory
 * (host-only use). Touches every page of the pool (pages are otherwise
 * mapped on first use, on the request path) and starts the reactor thread. */
kvx_status kvx_preloader_create(int32_t n_slots, int64_t slot_bytes, int32_t io_depth,
                                int32_t reserve, int32_t pinned, kvx_preloader** out);

/* Queue the chunk files (paths copied) of one waiting request for
 * speculative reading: one preload, started after the preloads queued
 * before it. Returns at once. */
kvx_status kvx_preload_hint(kvx_preloader* p, const char* const* paths, int32_t n);

/* Demand: make every named file staged (claiming staged images, joining reads
 * in progress, reading the rest before any speculative work; a file that
 * finds no slot takes that of a staged image nobody holds, else stops a
 * speculative read and takes its slot) and hold it:
 * images[i] / sizes[i] receive the host address and byte size of paths[i]'s
 * image, valid until kvx_preload_release. Blocks until all are staged.
 * KVX_ENOMEM if the files held after the call would exceed n_slots (nothing is
 * held then); KVX_EIO if a file is missing, empty, larger than a slot or
 * unreadable (nothing is held then). */
kvx_status kvx_preload_fetch(kvx_preloader* p, const char* const* paths, int32_t n, void** images,
                             int64_t* sizes);

/* Drop one hold of each named file (KVX_EINVAL, changing nothing, if one is
 * not held). Released images stay staged until their slot is needed. */
kvx_status kvx_preload_release(kvx_preloader* p, const char* const* paths, int32_t n);

/* Bind the next restores of `ring` to chunk files held in preloader p's pool
 * (pinned; else KVX_EINVAL), with the chunk list of kvx_ring_bind_files
 * (paths copied; a path may name several chunks of one size). Each
 * kvx_restore_from_staging then holds every named file as kvx_preload_fetch
 * does (claiming staged images, joining reads in progress, reading the rest
 * as demand work in chunk order; KVX_ENOMEM as for the fetch, nothing held)
 * but does not wait for all of them: a piece's host-to-device copies run
 * straight out of the pool as soon as its files are staged, while the later
 * files are still being read (Sec. 6.5: the demand load claims what the
 * preload staged and joins what it is reading). The restore returns once
 * every copy out of the pool has landed and drops its holds (the images stay
 * staged as cached images). A file that cannot be read, or whose size is not
 * its chunk's image size ((l1 - l0) * 2 * n_blocks * slab bytes), makes the
 * restore return KVX_EIO (pieces already scattered stay scattered). p must
 * outlive the binding. */
kvx_status kvx_ring_bind_preloaded(kvx_ring* ring, const kvx_cache* cache, int32_t l0, int32_t l1,
                                   int32_t chunk_tokens, kvx_preloader* p,
                                   const kvx_file_chunk* chunks, int32_t n_chunks);

/* Block until no read is in progress and no queued hint can start. */
kvx_status kvx_preload_wait_idle(kvx_preloader* p);

kvx_status kvx_preload_stats_get(kvx_preloader* p, kvx_preload_stats* out);

/* Stop the reactor (reads in flight complete first) and free the pool. */
kvx_status kvx_preloader_destroy(kvx_preloader* p);

/* Testing hook: the reactor pauses delay_us (0 .. 1000000; else KVX_EINVAL)
 * after each batch of completed pieces, which holds reads in progress long
 * enough for a test to act in the middle of one. Off (0) by default. */
kvx_status kvx_preload_set_test_hooks(kvx_preloader* p, int32_t delay_us);

/* Fault-injection hooks for testing the slot-reuse protocol from the host.
 * max_delay_us > 0: each fill or drain thread pauses a pseudo-random 0 ..
 * max_delay_us microseconds before every piece (varies the interleavings).
 * flags bit 0: a restore's fill threads overwrite their share of a released
 * host slot with 0xA5 bytes (then pause) before refilling it, so a copy that
 * still read a released slot would deliver the poison.
 * flags bit 1: the host-link copies (both directions) go through the HIP
 * runtime on the side stream even when the DMA engines are set up (exercises
 * that path); changing it first waits for the ring's copies in flight.
 * Other bits: KVX_EINVAL. Off by default; call between transfers. */
kvx_status kvx_ring_set_test_hooks(kvx_ring* ring, int32_t max_delay_us, int32_t flags);

/* Wait for an offload started by kvx_offload_begin (after kvx_ring_abort it
 * stops early), the ring's side stream and last restore, then free everything
 * the ring owns. */
kvx_status kvx_ring_destroy(kvx_ring* ring);

/* ---- step planning (host) ---------------------------------------------------- */

/* Prefix-hash chain (Sec. 2.1): out[b] = hash of full block b of `tokens`,
 * covering that block's block_size tokens and the hash of block b - 1
 * (parent_hash for block 0, e.g. 0 at the start of a prompt). Equal hashes mean
 * equal token prefixes through that block, so the hash of a chunk's last block
 * identifies the chunk. A trailing partial block gets no hash (partial blocks
 * are never cached). Returns the number of full blocks (n_tokens / block_size)
 * written to out, or -1 on a bad argument. Pure host code. */
int64_t kvx_block_hashes(const int32_t* tokens, int64_t n_tokens, int32_t block_size,
                         uint64_t parent_hash, uint64_t* out);

/* Chunk dedupe (Sec. 6.5: identical prefixes share one read): first_of[i] =
 * the smallest j with keys[j] == keys[i]; chunk i is restored itself iff
 * first_of[i] == i. Pure host code. */
kvx_status kvx_dedupe_keys(const uint64_t* keys, int32_t n, int32_t* first_of);

/* One request of a batched engine step (caller-owned arrays, read during the
 * call only). */
typedef struct kvx_step_request {
  const uint64_t* block_hashes;  /* n_blocks hashes of the prompt's full blocks, as
                                    kvx_block_hashes computes them */
  const uint8_t* resident;       /* one flag per chunk of the prompt: nonzero if the GPU
                                    holds that chunk (the engine's prefix lookup) */
  int32_t n_blocks;
  int32_t n_resident;            /* ceil(n_blocks / (chunk_tokens / block_size)) */
  int32_t new_blocks;            /* newly computed blocks to offload */
  int32_t reserved;
} kvx_step_request;

/* A chunk the step restores: its key (the hash of its last block), its
 * blocks, its origin (the first request, in order, that loads and needs it,
 * and the chunk's index in that request's prompt) and its slice of the
 * restore block table. */
typedef struct kvx_step_restore {
  uint64_t key;
  int32_t n_blocks;
  int32_t request;
  int32_t chunk;
  int32_t bt_offset;
} kvx_step_restore;

/* A chunk of one request's newly computed blocks (the store path): chunk
 * index among that request's new-block chunks, its blocks, its slice of the
 * offload block table and the request's first new block in it. */
typedef struct kvx_step_offload {
  int32_t request;
  int32_t chunk;
  int32_t n_blocks;
  int32_t bt_offset;
  int32_t new_first;
} kvx_step_offload;

/* chunk_states entries: >= 0 is an index into the restore list. */
#define KVX_CHUNK_RESIDENT (-1)
#define KVX_CHUNK_RECOMPUTE (-2)

/* Output of kvx_plan_step: caller-owned arrays with their capacities
 * (entries), then the counts and sums the call writes. */
typedef struct kvx_step_plan {
  kvx_step_restore* restore;
  kvx_step_offload* offload;
  int32_t* chunk_states;      /* per (request, chunk of its prompt), in order */
  int32_t* declined;          /* requests under the gate that had something to load */
  int32_t restore_cap, offload_cap, chunk_states_cap, declined_cap;
  int32_t n_restore, n_offload, n_chunk_states, n_declined;
  int32_t resident_hits;      /* distinct chunks the GPU already holds */
  int32_t reserved;
  int64_t restore_blocks, offload_blocks;
  int64_t recompute_blocks;   /* blocks of needed chunks nobody restores, per request */
} kvx_step_plan;

/* Plan one batched step (Secs. 6.2, 6.4-6.6): every chunk of every prompt
 * (chunk_tokens / block_size blocks; a prompt's last chunk may be shorter) is
 * keyed by the hash of its last full block, so a chunk that extends another
 * prompt's partial last chunk is a different chunk; a chunk's residency is
 * that of its first occurrence. A request loads when the tokens of its chunks
 * the GPU does not hold reach gate_tokens (the tier's break-even threshold,
 * Sec. 6.6; 0 loads everything; a request with nothing to load counts as
 * loading). A missing chunk is restored once, the first time a loading
 * request needs it (identical prefixes share one read, Sec. 6.5), and is
 * recomputed for each request that needs it otherwise. Each request's new
 * blocks are cut into chunks, in request order, for the store path. Restore
 * and offload block-table slices follow list order from 0.
 * With all four arrays NULL only the counts and sums are written (size query);
 * otherwise every array must hold its count (else KVX_EINVAL). KVX_EINVAL also
 * for a bad argument, a residency count other than the prompt's chunk count,
 * or a total over INT32_MAX blocks. Pure host code. */
kvx_status kvx_plan_step(const kvx_step_request* reqs, int32_t n_requests, int32_t block_size,
                         int32_t chunk_tokens, int64_t gate_tokens, kvx_step_plan* plan);

/* ---- break-even gate (host) --------------------------------------------------- */

/* A timing curve from an offline calibration sweep (Sec. 4.1, Pareto capture):
 * seconds[i] measured at a document (or prefix) of tokens[i] tokens. tokens
 * strictly ascending, n >= 2, every value finite; the caller owns both arrays.
 * Between points the curve is linear; beyond either end it continues the end
 * segment's line. Any invalid curve makes the calls below return KVX_EINVAL. */
typedef struct {
  const double* tokens;
  const double* seconds;
  int32_t n;
} kvx_curve;

/* *out = the curve at `tokens`. */
kvx_status kvx_curve_eval(const kvx_curve* c, double tokens, double* out);

/* *out = 1 when loading a cached prefix of prefix_tokens of a doc_tokens
 * document beats recomputing it (Sec. 4.1): hit(P) + cold(D - P) < cold(D),
 * with cold the full-prefill TTFT curve and hit the cache-hit TTFT curve;
 * else 0. Requires 0 <= prefix_tokens <= doc_tokens. */
kvx_status kvx_load_beats_recompute(const kvx_curve* cold, const kvx_curve* hit,
                                    int64_t doc_tokens, int64_t prefix_tokens, int32_t* out);

/* The break-even frontier at one document size (Sec. 5.2): *out = the
 * smallest P in {g, 2g, ...} (g = granularity, e.g. the chunk size), P <=
 * doc_tokens, for which loading beats recomputing; -1 if none does. */
kvx_status kvx_break_even_prefix(const kvx_curve* cold, const kvx_curve* hit, int64_t doc_tokens,
                                 int32_t granularity, int64_t* out);

/* The gate's threshold for one source tier (Sec. 6.6): *out = the smallest x
 * in {g, 2g, ...}, x <= max_tokens, such that a fully cached prompt of every
 * grid size from x through max_tokens loads faster than it recomputes
 * (hit(y) < cold(y)); -1 if even max_tokens does not. A reusable prefix below
 * the threshold is recomputed instead of loaded. */
kvx_status kvx_break_even_tokens(const kvx_curve* cold, const kvx_curve* hit, int64_t max_tokens,
                                 int32_t granularity, int64_t* out);

/* The transfer budget of a fully cached document (Sec. 5.2): *out_seconds =
 * cold(D) - (hit(D) - copy(D)), copy being the measured KV transfer time of
 * the hit path. Its KV bytes divided by this budget is the bandwidth a cache
 * path must sustain to match recomputation. */
kvx_status kvx_max_io(const kvx_curve* cold, const kvx_curve* hit, const kvx_curve* copy,
                      int64_t doc_tokens, double* out_seconds);

/* The hit curve of a tier from a measured restore rate (Secs. 5.2, 6.6: the
 * hit path's time is its non-transfer part plus the KV transfer):
 * out_seconds[i] = non_transfer.seconds[i] + non_transfer.tokens[i] *
 * bytes_per_token / (restore_GBps * 1e9), for the n knots of non_transfer
 * (out_seconds holds n doubles, caller-owned). The added term is linear in
 * tokens, so the curve through these knots is exact between and beyond them.
 * KVX_EINVAL for an invalid curve, bytes_per_token <= 0 or a rate that is not
 * positive and finite. */
kvx_status kvx_hit_curve_from_rate(const kvx_curve* non_transfer, int64_t bytes_per_token,
                                   double restore_GBps, double* out_seconds);

/* The bandwidth a cache path must sustain for a fully cached document of
 * doc_tokens to match recomputing it (Sec. 5.2): its KV bytes (doc_tokens *
 * bytes_per_token) over kvx_max_io, in GB/s (1e9 B/s); +infinity when the
 * budget is not positive. */
kvx_status kvx_required_GBps(const kvx_curve* cold, const kvx_curve* hit, const kvx_curve* copy,
                             int64_t doc_tokens, int64_t bytes_per_token, double* out_GBps);

/* The gate threshold of a source tier from its measured restore rate (Sec.
 * 6.6): kvx_break_even_tokens of the cold curve against the hit curve
 * kvx_hit_curve_from_rate builds from non_transfer, bytes_per_token and
 * restore_GBps. *out as for kvx_break_even_tokens (-1: loading never pays up
 * to max_tokens). */
kvx_status kvx_tier_threshold(const kvx_curve* cold, const kvx_curve* non_transfer,
                              int64_t bytes_per_token, double restore_GBps, int64_t max_tokens,
                              int32_t granularity, int64_t* out);

/* ---- measurement helper --------------------------------------------------------- */

/* HBM probe with the slab mover's shape (one workgroup per 4 KiB of
 * contiguous memory, 256 threads x one 16-byte vector, non-temporal loads and
 * the copy kernels' streaming stores, XCD-contiguous order), enqueued on `stream`. mode 0 reads `bytes` of src,
 * 1 writes `bytes` of dst, 2 copies src to dst. `bytes` a multiple of 4 KiB,
 * device pointers 16-byte aligned (src unused for mode 1, dst for mode 0);
 * else KVX_EINVAL. Mode 1 overwrites dst with a pattern. For roofline context
 * only: not part of the KV path. */
kvx_status kvx_probe_stream(const void* src, void* dst, int64_t bytes, int32_t mode,
                            hipStream_t stream);

/* Pinned host memory of exactly `bytes` (hipHostMalloc), for host images. */
kvx_status kvx_pinned_alloc(int64_t bytes, void** out);
kvx_status kvx_pinned_free(void* p);

#ifdef __cplusplus
}
#endif

#endif /* KVX_H_ */
