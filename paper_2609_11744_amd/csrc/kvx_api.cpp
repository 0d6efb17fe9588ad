// C-ABI entry points of libkvx.so: argument validation and dispatch to the HIP
// kernels. Every check that the host can make happens here, before anything
// is enqueued; block ids live on the device and are checked by the kernels.
#include <hip/hip_runtime_api.h>

#include <cstdint>
#include <cstring>
#include <new>

#include "kvx.h"
#include "kvx_internal.h"

namespace kvx {

static bool mul_ok(int64_t a, int64_t b, int64_t* out) { return !__builtin_mul_overflow(a, b, out); }

kvx_status validate(const kvx_cache* c, int32_t l0, int32_t l1, int32_t n_blocks,
                    int32_t chunk_tokens, bool need_pointers, Geometry* g) {
  if (!c || !g) return KVX_EINVAL;
  if (c->num_layers <= 0 || c->num_blocks <= 0 || c->block_size <= 0 || c->num_kv_heads <= 0 ||
      c->head_dim <= 0)
    return KVX_EINVAL;
  if (c->elem_bytes != 1 && c->elem_bytes != 2 && c->elem_bytes != 4 && c->elem_bytes != 8)
    return KVX_EINVAL;
  if (l0 < 0 || l1 < l0 || l1 > c->num_layers || l1 - l0 > KVX_MAX_LAYERS) return KVX_EINVAL;
  if (n_blocks < 0) return KVX_EINVAL;
  if (chunk_tokens <= 0 || chunk_tokens % c->block_size != 0) return KVX_EINVAL;
  int64_t slab = 0, t = 0;
  if (!mul_ok(c->block_size, c->num_kv_heads, &t) || !mul_ok(t, c->head_dim, &t) ||
      !mul_ok(t, c->elem_bytes, &slab))
    return KVX_EINVAL;
  if (slab % 16 != 0) return KVX_EINVAL;
  if (c->layout != KVX_LAYOUT_NHD && c->layout != KVX_LAYOUT_HND &&
      c->layout != KVX_LAYOUT_PAGED_ATTN)
    return KVX_EINVAL;
  if (c->layout != KVX_LAYOUT_NHD) {
    // staged through LDS: whole 16-byte vectors per row, a bounded slab
    if (((int64_t)c->head_dim * c->elem_bytes) % 16 != 0 || slab > kMaxTransposedSlab)
      return KVX_EINVAL;
  }
  int64_t pool = 0;
  if (!mul_ok(slab, c->num_blocks, &pool)) return KVX_EINVAL;
  const int64_t lr = l1 - l0;
  const int64_t n_units = lr * 2 * (int64_t)n_blocks;
  if (n_units > INT32_MAX) return KVX_EINVAL;
  // one workgroup per part of a slab (4 KiB pieces with the default layout,
  // heads with the others): the launch counts them in 31 bits
  const int64_t parts = c->layout == KVX_LAYOUT_NHD ? (slab / 16 + kPartThreads - 1) / kPartThreads
                                                    : (int64_t)c->num_kv_heads;
  if (n_units * parts > INT32_MAX) return KVX_EINVAL;
  int64_t packed = 0;
  if (!mul_ok(n_units, slab, &packed)) return KVX_EINVAL;
  if (need_pointers && n_units > 0) {
    if (!c->k || !c->v) return KVX_EINVAL;
    for (int32_t l = l0; l < l1; ++l) {
      if (!c->k[l] || !c->v[l]) return KVX_EINVAL;
      if (((uintptr_t)c->k[l] | (uintptr_t)c->v[l]) & 15) return KVX_EINVAL;
    }
  }
  int64_t bpc = chunk_tokens / c->block_size;
  // A chunk longer than the prefix has the same layout as one holding exactly
  // the prefix; clamping keeps every unit count inside 32 bits.
  if (n_blocks > 0 && bpc > n_blocks) bpc = n_blocks;
  g->slab = slab;
  g->packed = packed;
  g->n_units = n_units;
  g->lr = (int32_t)lr;
  g->bpc = (int32_t)bpc;
  g->n_blocks = n_blocks;
  g->num_blocks = c->num_blocks;
  return KVX_OK;
}

bool overlaps_cache(const kvx_cache* c, int32_t l0, int32_t l1, const void* packed,
                    int64_t bytes) {
  if (bytes <= 0) return false;
  const uintptr_t a0 = (uintptr_t)packed, a1 = a0 + (uintptr_t)bytes;
  const uintptr_t tensor = (uintptr_t)c->num_blocks * (uintptr_t)c->block_size *
                           (uintptr_t)c->num_kv_heads * (uintptr_t)c->head_dim *
                           (uintptr_t)c->elem_bytes;
  for (int32_t l = l0; l < l1; ++l) {
    for (const void* p : {(const void*)c->k[l], (const void*)c->v[l]}) {
      const uintptr_t b0 = (uintptr_t)p, b1 = b0 + tensor;
      if (a0 < b1 && b0 < a1) return true;
    }
  }
  return false;
}

static kvx_status copy_entry(bool to_packed, const kvx_cache* cache, int32_t l0, int32_t l1,
                             const int32_t* block_table, int32_t n_blocks, int32_t chunk_tokens,
                             const void* packed, hipStream_t stream) {
  Geometry g;
  kvx_status st = validate(cache, l0, l1, n_blocks, chunk_tokens, true, &g);
  if (st != KVX_OK) return st;
  if (g.n_units == 0) return KVX_OK;
  if (!block_table || !packed || ((uintptr_t)packed & 15)) return KVX_EINVAL;
  if (overlaps_cache(cache, l0, l1, packed, g.packed)) return KVX_EINVAL;
  return launch_copy(to_packed, cache, l0, l1, block_table, g, const_cast<void*>(packed), stream,
                     stream_error_word(stream));
}

static kvx_status chunks_entry(bool to_packed, const kvx_cache* cache, int32_t l0, int32_t l1,
                               const int32_t* block_table, int32_t table_len,
                               const kvx_chunk_ref* chunks, int32_t n_chunks,
                               int32_t chunk_tokens, const void* packed, int64_t packed_bytes,
                               hipStream_t stream) {
  Geometry g;
  kvx_status st = validate(cache, l0, l1, 0, chunk_tokens, false, &g);
  if (st != KVX_OK) return st;
  if (n_chunks < 0 || table_len < 0) return KVX_EINVAL;
  if (n_chunks == 0 || l0 == l1) return KVX_OK;
  if (!chunks || !packed || ((uintptr_t)packed & 15) || packed_bytes <= 0) return KVX_EINVAL;
  if (table_len > 0 && !block_table) return KVX_EINVAL;
  if (!cache->k || !cache->v) return KVX_EINVAL;
  for (int32_t l = l0; l < l1; ++l) {
    if (!cache->k[l] || !cache->v[l]) return KVX_EINVAL;
    if (((uintptr_t)cache->k[l] | (uintptr_t)cache->v[l]) & 15) return KVX_EINVAL;
  }
  const int64_t units = (int64_t)n_chunks * (l1 - l0) * 2 * (chunk_tokens / cache->block_size);
  const int64_t parts = cache->layout == KVX_LAYOUT_NHD
                            ? (g.slab / 16 + kPartThreads - 1) / kPartThreads
                            : (int64_t)cache->num_kv_heads;
  if (units > INT32_MAX || units * parts > INT32_MAX) return KVX_EINVAL;
  if (overlaps_cache(cache, l0, l1, packed, packed_bytes)) return KVX_EINVAL;
  return launch_copy_chunks(to_packed, cache, l0, l1, block_table, table_len, chunks, n_chunks,
                            chunk_tokens, const_cast<void*>(packed), packed_bytes, stream,
                            stream_error_word(stream));
}

}  // namespace kvx

extern "C" {

int64_t kvx_bytes_per_token(int32_t layers, int32_t kv_heads, int32_t head_dim,
                            int32_t elem_bytes) {
  if (layers <= 0 || kv_heads <= 0 || head_dim <= 0 || elem_bytes <= 0) return -1;
  return (int64_t)layers * 2 * kv_heads * head_dim * elem_bytes;
}

int64_t kvx_packed_bytes(const kvx_cache* cache, int32_t l0, int32_t l1, int32_t n_blocks) {
  kvx::Geometry g;
  const int32_t ct = cache ? cache->block_size : 0;
  if (kvx::validate(cache, l0, l1, n_blocks, ct, false, &g) != KVX_OK) return -1;
  return g.packed;
}

int64_t kvx_chunk_stride(const kvx_cache* cache, int32_t l0, int32_t l1, int32_t chunk_tokens) {
  kvx::Geometry g;
  if (kvx::validate(cache, l0, l1, 0, chunk_tokens, false, &g) != KVX_OK) return -1;
  int64_t s = 0;
  if (__builtin_mul_overflow((int64_t)g.lr * 2 * g.bpc, g.slab, &s)) return -1;
  return s;
}

kvx_status kvx_gather_blocks(const kvx_cache* cache, int32_t l0, int32_t l1,
                             const int32_t* block_table, int32_t n_blocks, int32_t chunk_tokens,
                             void* dst, hipStream_t stream) {
  try {
    return kvx::copy_entry(true, cache, l0, l1, block_table, n_blocks, chunk_tokens, dst, stream);
  } catch (...) {
    return KVX_EINTERNAL;
  }
}

kvx_status kvx_scatter_blocks(const kvx_cache* cache, int32_t l0, int32_t l1,
                              const int32_t* block_table, int32_t n_blocks, int32_t chunk_tokens,
                              const void* src, hipStream_t stream) {
  try {
    return kvx::copy_entry(false, cache, l0, l1, block_table, n_blocks, chunk_tokens, src, stream);
  } catch (...) {
    return KVX_EINTERNAL;
  }
}

kvx_status kvx_gather_chunks(const kvx_cache* cache, int32_t l0, int32_t l1,
                             const int32_t* block_table, int32_t table_len,
                             const kvx_chunk_ref* chunks, int32_t n_chunks, int32_t chunk_tokens,
                             void* packed, int64_t packed_bytes, hipStream_t stream) {
  try {
    return kvx::chunks_entry(true, cache, l0, l1, block_table, table_len, chunks, n_chunks,
                             chunk_tokens, packed, packed_bytes, stream);
  } catch (...) {
    return KVX_EINTERNAL;
  }
}

kvx_status kvx_scatter_chunks(const kvx_cache* cache, int32_t l0, int32_t l1,
                              const int32_t* block_table, int32_t table_len,
                              const kvx_chunk_ref* chunks, int32_t n_chunks, int32_t chunk_tokens,
                              const void* packed, int64_t packed_bytes, hipStream_t stream) {
  try {
    return kvx::chunks_entry(false, cache, l0, l1, block_table, table_len, chunks, n_chunks,
                             chunk_tokens, packed, packed_bytes, stream);
  } catch (...) {
    return KVX_EINTERNAL;
  }
}

kvx_status kvx_check(hipStream_t stream) {
  if (hipStreamSynchronize(stream) != hipSuccess) return KVX_EHIP;
  int* w = kvx::stream_error_word(stream);
  if (!w) return KVX_EHIP;
  // read and clear the word through the stream itself, so that the check
  // waits for no other stream
  int v = 0;
  if (hipMemcpyAsync(&v, w, sizeof(int), hipMemcpyDeviceToHost, stream) != hipSuccess ||
      hipStreamSynchronize(stream) != hipSuccess)
    return KVX_EHIP;
  if (v != 0) {
    const int zero = 0;
    if (hipMemcpyAsync(w, &zero, sizeof(int), hipMemcpyHostToDevice, stream) != hipSuccess ||
        hipStreamSynchronize(stream) != hipSuccess)
      return KVX_EHIP;
    return (v & 2) ? KVX_EINVAL : KVX_EBADBLOCK;  // bit 1: bad chunk ref, bit 0: bad block id
  }
  return KVX_OK;
}

const char* kvx_strerror(kvx_status s) {
  switch (s) {
    case KVX_OK: return "ok";
    case KVX_EINVAL: return "invalid argument";
    case KVX_ENOMEM: return "out of memory";
    case KVX_EHIP: return "HIP runtime error";
    case KVX_EBADBLOCK: return "block id out of range";
    case KVX_ECLOSED: return "ring aborted";
    case KVX_EINTERNAL: return "internal error";
    case KVX_EIO: return "storage-tier file I/O failed";
    case KVX_EBUSY: return "ring busy with a transfer started by kvx_offload_begin or kvx_restore_begin";
  }
  return "unknown status";
}

kvx_status kvx_pinned_alloc(int64_t bytes, void** out) {
  if (!out || bytes <= 0) return KVX_EINVAL;
  *out = nullptr;
  if (hipHostMalloc(out, (size_t)bytes, hipHostMallocDefault) != hipSuccess) {
    *out = nullptr;
    return KVX_ENOMEM;
  }
  return KVX_OK;
}

kvx_status kvx_pinned_free(void* p) {
  if (!p) return KVX_OK;
  return hipHostFree(p) == hipSuccess ? KVX_OK : KVX_EHIP;
}

}  // extern "C"
