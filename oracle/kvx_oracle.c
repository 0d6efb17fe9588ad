/*
 * Plain CPU oracle for the paged-KV gather / scatter / staged-restore path.
 *
 * TEST INFRASTRUCTURE ONLY. Only the test suite, the smoke check and the
 * bench's CPU-baseline leg may load this library. It shares no code, header,
 * table or helper with the HIP path, and nothing on the product path calls it.
 *
 * What the path computes, restated from the paper:
 *   - Serving systems keep KV in fixed-size token blocks rather than one tensor
 *     per request; blocks of one prompt need not be adjacent in memory
 *     (Sec. 2.1, "KV Cache in LLM Serving"; PagedAttention).
 *   - Size model: bytes per token = layers x 2 x KV heads x head dim x dtype
 *     size (Sec. 2.1).
 *   - The external cache moves data in storage blocks that each group several
 *     of the engine's GPU blocks (Sec. 6.4); a batched block copy moves data
 *     between the GPU KV tensors and contiguous staging slots (Secs. 6.2, 6.4).
 *   - Staging is bounded; a request larger than the pool is moved piece by
 *     piece, and the result must not depend on how it was split (Sec. 6.4).
 *
 * The paper gives no byte layout for a storage block. Readings used here:
 *   - Cache: per layer, separate K and V tensors, each [num_blocks][block_size]
 *     [kv_heads][head_dim] of elem_bytes-byte words. A slab is one (layer, K|V,
 *     block): block_size*kv_heads*head_dim*elem_bytes contiguous bytes.
 *   - Chunk (storage block) of chunk_tokens tokens = chunk_tokens/block_size
 *     GPU blocks; chunk_tokens must be a positive multiple of block_size.
 *   - Inside a chunk: layer-major [layer in l0..l1-1][K then V][token][head]
 *     [dim]; chunk c starts at c * S with S = (l1-l0)*2*chunk_tokens*row bytes.
 *   - The last chunk may hold fewer blocks; it is compact (its internal strides
 *     use its own token count), so the packed image is exactly
 *     n_blocks*(l1-l0)*2*slab bytes with no padding.
 *   - Gather reads cache slabs named by block_table; scatter writes them, and
 *     leaves every byte it does not name unchanged.
 *   - A block id outside [0, num_blocks) is an error; nothing is written then.
 *
 * Cache layouts other than the default (the packed chunk layout is the same
 * for all of them; only where a cache element lives changes):
 *   KVO_LAYOUT_NHD        K and V [num_blocks][block_size][kv_heads][head_dim]
 *   KVO_LAYOUT_HND        K and V [num_blocks][kv_heads][block_size][head_dim]
 *   KVO_LAYOUT_PAGED_ATTN K [num_blocks][kv_heads][head_dim / x][block_size][x]
 *                         with x = 16 / elem_bytes elements (16-byte groups),
 *                         V [num_blocks][kv_heads][head_dim][block_size]
 * For these the oracle moves one element at a time.
 *
 * Words are copied as raw bytes (never converted), so NaN payloads, -0 and
 * denormals survive.
 */
#include <stdint.h>
#include <string.h>

typedef struct {
  int64_t num_layers, num_blocks, block_size, kv_heads, head_dim, elem_bytes;
  int64_t layout;
} kvo_shape;

enum { KVO_OK = 0, KVO_EINVAL = -1, KVO_EBADBLOCK = -4 };
enum { KVO_LAYOUT_NHD = 0, KVO_LAYOUT_HND = 1, KVO_LAYOUT_PAGED_ATTN = 2 };

/* Byte offset, inside one block's slab, of element (token t, head h, dim d)
 * of the K (kv = 0) or V (kv = 1) tensor. */
static int64_t elem_offset(const kvo_shape* s, int kv, int64_t t, int64_t h, int64_t d) {
  const int64_t BS = s->block_size, H = s->kv_heads, D = s->head_dim, e = s->elem_bytes;
  if (s->layout == KVO_LAYOUT_HND) return ((h * BS + t) * D + d) * e;
  if (s->layout == KVO_LAYOUT_PAGED_ATTN) {
    if (kv == 1) return ((h * D + d) * BS + t) * e;
    const int64_t x = 16 / e;
    return (((h * (D / x) + d / x) * BS + t) * x + d % x) * e;
  }
  return ((t * H + h) * D + d) * e;
}

/* Size model of Sec. 2.1. */
int64_t kvo_bytes_per_token(int64_t layers, int64_t kv_heads, int64_t head_dim,
                            int64_t elem_bytes) {
  return layers * 2 * kv_heads * head_dim * elem_bytes;
}

int64_t kvo_slab_bytes(const kvo_shape* s) {
  return s->block_size * s->kv_heads * s->head_dim * s->elem_bytes;
}

/* Bytes of the packed image of n blocks over layers [l0, l1). */
int64_t kvo_packed_bytes(const kvo_shape* s, int64_t l0, int64_t l1, int64_t n) {
  return n * (l1 - l0) * 2 * kvo_slab_bytes(s);
}

static int check_args(const kvo_shape* s, int64_t l0, int64_t l1, const int32_t* bt, int64_t n,
                      int64_t chunk_tokens) {
  if (!s || s->num_layers <= 0 || s->num_blocks <= 0 || s->block_size <= 0 ||
      s->kv_heads <= 0 || s->head_dim <= 0 || s->elem_bytes <= 0)
    return KVO_EINVAL;
  if (l0 < 0 || l1 < l0 || l1 > s->num_layers || n < 0) return KVO_EINVAL;
  if (chunk_tokens <= 0 || chunk_tokens % s->block_size != 0) return KVO_EINVAL;
  if (s->layout < KVO_LAYOUT_NHD || s->layout > KVO_LAYOUT_PAGED_ATTN) return KVO_EINVAL;
  if (s->layout == KVO_LAYOUT_PAGED_ATTN &&
      (16 % s->elem_bytes != 0 || s->head_dim % (16 / s->elem_bytes) != 0))
    return KVO_EINVAL;
  if (n > 0 && !bt) return KVO_EINVAL;
  for (int64_t i = 0; i < n; ++i)
    if (bt[i] < 0 || bt[i] >= s->num_blocks) return KVO_EBADBLOCK;
  return KVO_OK;
}

/* Move one block's slab between the cache (in the shape's layout) and the
 * packed chunk (always [token][head][dim]). */
static void move_slab(const kvo_shape* s, int kv, uint8_t* packed, uint8_t* cache, int to_packed) {
  const int64_t BS = s->block_size, H = s->kv_heads, D = s->head_dim, e = s->elem_bytes;
  if (s->layout == KVO_LAYOUT_NHD) {
    if (to_packed) memcpy(packed, cache, (size_t)(BS * H * D * e));
    else memcpy(cache, packed, (size_t)(BS * H * D * e));
    return;
  }
  for (int64_t t = 0; t < BS; ++t)
    for (int64_t h = 0; h < H; ++h)
      for (int64_t d = 0; d < D; ++d) {
        uint8_t* p = packed + ((t * H + h) * D + d) * e;
        uint8_t* c = cache + elem_offset(s, kv, t, h, d);
        if (to_packed) memcpy(p, c, (size_t)e);
        else memcpy(c, p, (size_t)e);
      }
}

/* Gather: dst[c*S + ((l-l0)*2 + kv)*T_c*row + j*slab, +slab) =
 *         cache[l][kv][bt[c*bpc + j]*slab, +slab)
 * for every chunk c, layer l in [l0, l1), kv in {K, V}, block j of the chunk
 * (element by element through the layout when it is not the default). */
int kvo_gather(const kvo_shape* s, const void* const* k, const void* const* v, int64_t l0,
               int64_t l1, const int32_t* bt, int64_t n, int64_t chunk_tokens, void* dst) {
  int rc = check_args(s, l0, l1, bt, n, chunk_tokens);
  if (rc != KVO_OK) return rc;
  if (n == 0 || l0 == l1) return KVO_OK;
  if (!k || !v || !dst) return KVO_EINVAL;
  const int64_t row = s->kv_heads * s->head_dim * s->elem_bytes;
  const int64_t slab = s->block_size * row;
  const int64_t bpc = chunk_tokens / s->block_size;
  const int64_t S = (l1 - l0) * 2 * chunk_tokens * row;
  const int64_t nchunks = (n + bpc - 1) / bpc;
  uint8_t* out = (uint8_t*)dst;
  for (int64_t c = 0; c < nchunks; ++c) {
    const int64_t nc = (n - c * bpc < bpc) ? n - c * bpc : bpc;
    const int64_t Tc = nc * s->block_size;
    for (int64_t l = l0; l < l1; ++l) {
      for (int kv = 0; kv < 2; ++kv) {
        const uint8_t* base = (const uint8_t*)(kv == 0 ? k[l] : v[l]);
        for (int64_t j = 0; j < nc; ++j) {
          const int64_t id = bt[c * bpc + j];
          move_slab(s, kv, out + c * S + ((l - l0) * 2 + kv) * Tc * row + j * slab,
                    (uint8_t*)base + id * slab, 1);
        }
      }
    }
  }
  return KVO_OK;
}

/* Scatter: the same equation with the assignment reversed. */
int kvo_scatter(const kvo_shape* s, void* const* k, void* const* v, int64_t l0, int64_t l1,
                const int32_t* bt, int64_t n, int64_t chunk_tokens, const void* src) {
  int rc = check_args(s, l0, l1, bt, n, chunk_tokens);
  if (rc != KVO_OK) return rc;
  if (n == 0 || l0 == l1) return KVO_OK;
  if (!k || !v || !src) return KVO_EINVAL;
  const int64_t row = s->kv_heads * s->head_dim * s->elem_bytes;
  const int64_t slab = s->block_size * row;
  const int64_t bpc = chunk_tokens / s->block_size;
  const int64_t S = (l1 - l0) * 2 * chunk_tokens * row;
  const int64_t nchunks = (n + bpc - 1) / bpc;
  const uint8_t* in = (const uint8_t*)src;
  for (int64_t c = 0; c < nchunks; ++c) {
    const int64_t nc = (n - c * bpc < bpc) ? n - c * bpc : bpc;
    const int64_t Tc = nc * s->block_size;
    for (int64_t l = l0; l < l1; ++l) {
      for (int kv = 0; kv < 2; ++kv) {
        uint8_t* base = (uint8_t*)(kv == 0 ? k[l] : v[l]);
        for (int64_t j = 0; j < nc; ++j) {
          const int64_t id = bt[c * bpc + j];
          move_slab(s, kv, (uint8_t*)in + c * S + ((l - l0) * 2 + kv) * Tc * row + j * slab,
                    base + id * slab, 0);
        }
      }
    }
  }
  return KVO_OK;
}
