/*
 * A caller of libkvx.so written in C alone (no Python, no C++): the library's
 * boundary exercised the way a serving engine in any language would use it.
 * Test program: tests/test_gpu_c_caller.py prepares its inputs, runs it and
 * compares what it writes with the oracle.
 *
 * usage: kvx_c_caller DIR SEED MODE STREAM_BASE N CHUNK_TOKENS
 *   DIR/bt_src.bin, bt_dst.bin, bt_rst.bin  int32[N] block tables
 *   DIR/image.bin                           the packed image a staged restore loads
 * The cache (3 layers, 96 blocks of 16 tokens, 2 KV heads, head dim 64, 2-byte
 * words, default layout) is filled on the host with the seeded input
 * generator, tensor (layer l, K|V kv) from stream STREAM_BASE + 2 l + kv, and
 * copied to the device. Then, on a stream of its own:
 *   1. gather the N blocks of bt_src              -> DIR/gathered.bin
 *   2. scatter that image into the blocks of bt_dst
 *   3. restore image.bin into the blocks of bt_rst through a staging ring
 *      (2 slots of 64 KiB, 2 fill threads)
 *   4. copy the whole cache back                  -> DIR/cache_after.bin
 *      (K of layers 0..2, then V of layers 0..2)
 * and the error paths: a chunk size that is not a whole number of blocks and
 * a null cache are rejected on the host (KVX_EINVAL); a block id outside the
 * pool is reported by kvx_check (KVX_EBADBLOCK), once.
 * Prints the sizes the library reports and "c caller: ok"; exits 1 on any
 * failure, naming it.
 */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "kvx.h"

/* the seeded input generator's host fill (kvsynth/synth_host.c) */
int kvs_fill_host(void* out, uint64_t nbytes, uint64_t seed, uint64_t stream,
                  uint64_t byte_offset, int mode, int threads);

enum { L = 3, NB = 96, BS = 16, H = 2, D = 64, E = 2 };

static int failed(const char* what, long got) {
  fprintf(stderr, "c caller: %s (%ld)\n", what, got);
  return 1;
}

static void* read_file(const char* dir, const char* name, size_t want) {
  char path[4096];
  snprintf(path, sizeof path, "%s/%s", dir, name);
  FILE* f = fopen(path, "rb");
  if (!f) return NULL;
  void* p = malloc(want ? want : 1);
  size_t got = p ? fread(p, 1, want, f) : 0;
  fclose(f);
  if (got != want) {
    free(p);
    return NULL;
  }
  return p;
}

static int write_file(const char* dir, const char* name, const void* p, size_t n) {
  char path[4096];
  snprintf(path, sizeof path, "%s/%s", dir, name);
  FILE* f = fopen(path, "wb");
  if (!f) return -1;
  size_t put = fwrite(p, 1, n, f);
  return fclose(f) == 0 && put == n ? 0 : -1;
}

int main(int argc, char** argv) {
  if (argc != 7) {
    fprintf(stderr, "usage: %s DIR SEED MODE STREAM_BASE N CHUNK_TOKENS\n", argv[0]);
    return 2;
  }
  const char* dir = argv[1];
  const uint64_t seed = strtoull(argv[2], NULL, 0);
  const int mode = atoi(argv[3]);
  const uint64_t base = strtoull(argv[4], NULL, 0);
  const int32_t n = atoi(argv[5]), ct = atoi(argv[6]);
  const size_t tensor = (size_t)NB * BS * H * D * E;

  /* the cache: host fill, then one device tensor per (layer, K|V) */
  void* k[L];
  void* v[L];
  uint8_t* host = malloc(tensor);
  if (!host) return failed("host buffer", 0);
  for (int l = 0; l < L; ++l) {
    for (int kv = 0; kv < 2; ++kv) {
      void** t = kv ? &v[l] : &k[l];
      if (kvs_fill_host(host, tensor, seed, base + 2 * (uint64_t)l + kv, 0, mode, 2) != 0)
        return failed("generator fill", l);
      if (hipMalloc(t, tensor) != hipSuccess) return failed("hipMalloc cache", l);
      if (hipMemcpy(*t, host, tensor, hipMemcpyHostToDevice) != hipSuccess)
        return failed("hipMemcpy cache", l);
    }
  }
  kvx_cache cache = {k, v, L, NB, BS, H, D, E, KVX_LAYOUT_NHD};

  const int64_t bytes = kvx_packed_bytes(&cache, 0, L, n);
  const int64_t stride = kvx_chunk_stride(&cache, 0, L, ct);
  printf("packed_bytes=%lld chunk_stride=%lld\n", (long long)bytes, (long long)stride);
  if (bytes <= 0 || stride <= 0) return failed("size model", (long)bytes);

  int32_t* bt[3];
  const char* names[3] = {"bt_src.bin", "bt_dst.bin", "bt_rst.bin"};
  int32_t* d_bt[3];
  for (int i = 0; i < 3; ++i) {
    bt[i] = read_file(dir, names[i], (size_t)n * sizeof(int32_t));
    if (!bt[i]) return failed(names[i], i);
    if (hipMalloc((void**)&d_bt[i], (size_t)n * sizeof(int32_t)) != hipSuccess ||
        hipMemcpy(d_bt[i], bt[i], (size_t)n * sizeof(int32_t), hipMemcpyHostToDevice) !=
            hipSuccess)
      return failed("block table upload", i);
  }
  void* image = read_file(dir, "image.bin", (size_t)bytes);
  if (!image) return failed("image.bin", (long)bytes);

  hipStream_t stream;
  if (hipStreamCreateWithFlags(&stream, hipStreamNonBlocking) != hipSuccess)
    return failed("stream", 0);
  void* packed = NULL;
  if (hipMalloc(&packed, (size_t)bytes) != hipSuccess) return failed("hipMalloc packed", 0);

  /* 1. gather */
  kvx_status st = kvx_gather_blocks(&cache, 0, L, d_bt[0], n, ct, packed, stream);
  if (st != KVX_OK) return failed(kvx_strerror(st), st);
  if ((st = kvx_check(stream)) != KVX_OK) return failed("gather check", st);
  uint8_t* out = malloc((size_t)bytes);
  if (!out || hipMemcpy(out, packed, (size_t)bytes, hipMemcpyDeviceToHost) != hipSuccess)
    return failed("gathered copy-back", 0);
  if (write_file(dir, "gathered.bin", out, (size_t)bytes) != 0) return failed("gathered.bin", 0);

  /* 2. scatter */
  st = kvx_scatter_blocks(&cache, 0, L, d_bt[1], n, ct, packed, stream);
  if (st != KVX_OK) return failed(kvx_strerror(st), st);
  if ((st = kvx_check(stream)) != KVX_OK) return failed("scatter check", st);

  /* 3. staged restore from pinned host memory */
  void* pinned = NULL;
  if ((st = kvx_pinned_alloc(bytes, &pinned)) != KVX_OK) return failed("pinned alloc", st);
  memcpy(pinned, image, (size_t)bytes);
  kvx_ring* ring = NULL;
  if ((st = kvx_ring_create(0, 2, 64 << 10, NULL, &ring)) != KVX_OK) return failed("ring", st);
  if ((st = kvx_ring_bind(ring, &cache, 0, L, n, ct, pinned, 2)) != KVX_OK)
    return failed("ring bind", st);
  if ((st = kvx_restore_from_staging(ring, d_bt[2], stream)) != KVX_OK)
    return failed("restore", st);
  if ((st = kvx_check(stream)) != KVX_OK) return failed("restore check", st);
  if ((st = kvx_ring_destroy(ring)) != KVX_OK) return failed("ring destroy", st);
  if ((st = kvx_pinned_free(pinned)) != KVX_OK) return failed("pinned free", st);

  /* 4. the whole cache back to the host */
  uint8_t* all = malloc(2 * L * tensor);
  if (!all) return failed("host cache", 0);
  for (int l = 0; l < L; ++l) {
    if (hipMemcpy(all + (size_t)l * tensor, k[l], tensor, hipMemcpyDeviceToHost) != hipSuccess ||
        hipMemcpy(all + (size_t)(L + l) * tensor, v[l], tensor, hipMemcpyDeviceToHost) !=
            hipSuccess)
      return failed("cache copy-back", l);
  }
  if (write_file(dir, "cache_after.bin", all, 2 * L * tensor) != 0)
    return failed("cache_after.bin", 0);

  /* error paths */
  st = kvx_gather_blocks(&cache, 0, L, d_bt[0], n, BS + 1, packed, stream);
  if (st != KVX_EINVAL) return failed("chunk size not a multiple of the block size", st);
  st = kvx_gather_blocks(NULL, 0, L, d_bt[0], n, ct, packed, stream);
  if (st != KVX_EINVAL) return failed("null cache", st);
  const int32_t bad[1] = {NB + 5};
  int32_t* d_bad = NULL;
  if (hipMalloc((void**)&d_bad, sizeof bad) != hipSuccess ||
      hipMemcpy(d_bad, bad, sizeof bad, hipMemcpyHostToDevice) != hipSuccess)
    return failed("bad table upload", 0);
  if ((st = kvx_gather_blocks(&cache, 0, L, d_bad, 1, ct, packed, stream)) != KVX_OK)
    return failed("gather of a bad id was not enqueued", st);
  if ((st = kvx_check(stream)) != KVX_EBADBLOCK) return failed("bad block id not reported", st);
  if ((st = kvx_check(stream)) != KVX_OK) return failed("error word not cleared", st);
  if (!kvx_strerror(KVX_EBADBLOCK) || !*kvx_strerror(KVX_EBADBLOCK))
    return failed("kvx_strerror", 0);

  for (int i = 0; i < 3; ++i) {
    (void)hipFree(d_bt[i]);
    free(bt[i]);
  }
  for (int l = 0; l < L; ++l) {
    (void)hipFree(k[l]);
    (void)hipFree(v[l]);
  }
  (void)hipFree(d_bad);
  (void)hipFree(packed);
  (void)hipStreamDestroy(stream);
  free(all);
  free(out);
  free(image);
  free(host);
  printf("c caller: ok\n");
  return 0;
}
