/*
 * kvsynth host generator: seeded synthetic bytes for KV-cache tensors and
 * packed transfer images.
 *
 * This module is shared by the test suite, the oracle's inputs and the bench.
 * It knows nothing about paged blocks, chunks or layouts: it fills a flat byte
 * range of a named stream, so the bytes at (seed, stream, byte offset) are the
 * same whether a whole tensor or one slab of it is generated.
 *
 * Generator: splitmix64 (G. Steele, D. Lea, C. Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014), used counter-style:
 *   key(seed, stream) = mix(mix(seed + G) ^ (stream * M + 1))
 *   word(w)           = mix(key + (w + 1) * G)     for 8-byte word index w
 * where mix is splitmix64's output finaliser and G = 0x9E3779B97F4A7C15.
 *
 * Modes for turning a 64-bit word into 8 bytes:
 *   KVS_MODE_NORMAL_BF16: four bf16 values; 16-bit lane i of the word indexes a
 *     65,536-entry table of standard normal quantiles Phi^-1((k + 0.5) / 65536),
 *     each computed in double and rounded to nearest-even bf16. The elements are
 *     therefore N(0,1) to bf16 resolution and generation is integer-only.
 *   KVS_MODE_RAW: the word's bytes as they are (every 16-bit pattern, NaN
 *     payloads, infinities and denormals included).
 *
 * The device fill (synth_dev.hip) implements the same definition and takes the
 * same table, which it receives from kvs_normal_table().
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <string.h>

#define KVS_GOLDEN 0x9E3779B97F4A7C15ULL
#define KVS_STREAM_MUL 0xD1B54A32D192ED03ULL

enum { KVS_MODE_NORMAL_BF16 = 0, KVS_MODE_RAW = 1 };

static uint64_t kvs_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

uint64_t kvs_stream_key(uint64_t seed, uint64_t stream) {
  return kvs_mix(kvs_mix(seed + KVS_GOLDEN) ^ (stream * KVS_STREAM_MUL + 1ULL));
}

uint64_t kvs_word(uint64_t key, uint64_t w) { return kvs_mix(key + (w + 1ULL) * KVS_GOLDEN); }

/* ---- N(0,1) quantile table ------------------------------------------------ */

static uint16_t g_table[65536];
static pthread_once_t g_table_once = PTHREAD_ONCE_INIT;

/* Round a double to bf16 bits, nearest-even, in one step from the double's bits
 * (going through float first would round twice). bf16 keeps the sign, an 8-bit
 * exponent and 7 explicit mantissa bits; the 45 discarded mantissa bits decide
 * the rounding. Every quantile here satisfies 1e-6 < |x| < 6, far from bf16
 * overflow and underflow, so only the normal case is needed. */
static uint16_t bf16_from_double(double x) {
  uint64_t b;
  memcpy(&b, &x, 8);
  uint64_t sign = b >> 63;
  int64_t e = (int64_t)((b >> 52) & 0x7FF) - 1023;
  uint64_t man = b & ((1ULL << 52) - 1);
  uint64_t keep = man >> 45;              /* 7 bits */
  uint64_t rest = man & ((1ULL << 45) - 1);
  uint64_t half = 1ULL << 44;
  if (rest > half || (rest == half && (keep & 1))) {
    keep += 1;
    if (keep == 128) { keep = 0; e += 1; }
  }
  uint64_t fe = (uint64_t)(e + 127);
  return (uint16_t)((sign << 15) | (fe << 7) | keep);
}

/* Standard normal CDF. */
static double phi(double x) { return 0.5 * erfc(-x / sqrt(2.0)); }

/* Phi^-1(p) by bisection on the CDF: slow but plainly correct, run once. */
static double phi_inv(double p) {
  double lo = -40.0, hi = 40.0;
  for (int it = 0; it < 200; ++it) {
    double mid = 0.5 * (lo + hi);
    if (phi(mid) < p) lo = mid; else hi = mid;
    if (hi - lo < 1e-15) break;
  }
  return 0.5 * (lo + hi);
}

static void build_table(void) {
  /* Symmetry Phi^-1(1-p) = -Phi^-1(p): compute the upper half, mirror it, so
   * the table is exactly antisymmetric in its bits. */
  for (int k = 32768; k < 65536; ++k) {
    double p = ((double)k + 0.5) / 65536.0;
    uint16_t v = bf16_from_double(phi_inv(p));
    g_table[k] = v;
    g_table[65535 - k] = (uint16_t)(v ^ 0x8000u);
  }
}

const uint16_t* kvs_normal_table(void) {
  pthread_once(&g_table_once, build_table);
  return g_table;
}

/* ---- fill ------------------------------------------------------------------ */

static void fill_words(uint8_t* out, uint64_t key, uint64_t w0, uint64_t nwords, int mode,
                       const uint16_t* tab) {
  for (uint64_t i = 0; i < nwords; ++i) {
    uint64_t h = kvs_word(key, w0 + i);
    if (mode == KVS_MODE_NORMAL_BF16) {
      uint16_t e4[4];
      for (int q = 0; q < 4; ++q) e4[q] = tab[(h >> (16 * q)) & 0xFFFFu];
      memcpy(out + 8 * i, e4, 8);
    } else {
      memcpy(out + 8 * i, &h, 8); /* little-endian host */
    }
  }
}

typedef struct {
  uint8_t* out;
  uint64_t key, w0, nwords;
  int mode;
  const uint16_t* tab;
} fill_job;

static void* fill_thread(void* arg) {
  fill_job* j = (fill_job*)arg;
  fill_words(j->out, j->key, j->w0, j->nwords, j->mode, j->tab);
  return 0;
}

/* Fill `nbytes` at `out` with stream (seed, stream) bytes [byte_offset,
 * byte_offset + nbytes). byte_offset and nbytes must be multiples of 8.
 * Returns 0, or -1 on a bad argument. Uses up to `threads` threads. */
int kvs_fill_host(void* out, uint64_t nbytes, uint64_t seed, uint64_t stream,
                  uint64_t byte_offset, int mode, int threads) {
  if ((nbytes & 7) || (byte_offset & 7) || (mode != KVS_MODE_NORMAL_BF16 && mode != KVS_MODE_RAW))
    return -1;
  if (nbytes == 0) return 0;
  if (!out) return -1;
  const uint16_t* tab = kvs_normal_table();
  uint64_t key = kvs_stream_key(seed, stream);
  uint64_t nwords = nbytes / 8, w0 = byte_offset / 8;
  if (threads < 1) threads = 1;
  if (threads > 64) threads = 64;
  if (nwords < (1ULL << 20) || threads == 1) {
    fill_words((uint8_t*)out, key, w0, nwords, mode, tab);
    return 0;
  }
  pthread_t th[64];
  int created[64];
  fill_job jobs[64];
  uint64_t per = (nwords + threads - 1) / threads;
  int started = 0;
  for (int t = 0; t < threads; ++t) {
    uint64_t a = per * t, b = a + per < nwords ? a + per : nwords;
    if (a >= b) break;
    jobs[t] = (fill_job){(uint8_t*)out + 8 * a, key, w0 + a, b - a, mode, tab};
    created[t] = pthread_create(&th[t], 0, fill_thread, &jobs[t]) == 0;
    if (!created[t]) fill_thread(&jobs[t]);
    started = t + 1;
  }
  for (int t = 0; t < started; ++t)
    if (created[t]) pthread_join(th[t], 0);
  return 0;
}

/* Fill many equal-length ranges of one stream: for i < n,
 * out_base[offsets[i], offsets[i] + len) = stream bytes [offsets[i], +len).
 * Offsets and len must be multiples of 8. Ranges are split over threads. */
typedef struct {
  uint8_t* base;
  const uint64_t* offsets;
  uint64_t n, len, key;
  int mode, stride, start;
  const uint16_t* tab;
} ranges_job;

static void* ranges_thread(void* arg) {
  ranges_job* j = (ranges_job*)arg;
  for (uint64_t i = (uint64_t)j->start; i < j->n; i += (uint64_t)j->stride)
    fill_words(j->base + j->offsets[i], j->key, j->offsets[i] / 8, j->len / 8, j->mode, j->tab);
  return 0;
}

int kvs_fill_ranges(void* out_base, const uint64_t* offsets, uint64_t n, uint64_t len,
                    uint64_t seed, uint64_t stream, int mode, int threads) {
  if ((len & 7) || (mode != KVS_MODE_NORMAL_BF16 && mode != KVS_MODE_RAW)) return -1;
  if (n == 0 || len == 0) return 0;
  if (!out_base || !offsets) return -1;
  for (uint64_t i = 0; i < n; ++i)
    if (offsets[i] & 7) return -1;
  const uint16_t* tab = kvs_normal_table();
  uint64_t key = kvs_stream_key(seed, stream);
  if (threads < 1) threads = 1;
  if (threads > 64) threads = 64;
  if ((uint64_t)threads > n) threads = (int)n;
  pthread_t th[64];
  int created[64];
  ranges_job jobs[64];
  for (int t = 0; t < threads; ++t) {
    jobs[t] = (ranges_job){(uint8_t*)out_base, offsets, n, len, key, mode, threads, t, tab};
    created[t] = threads > 1 && pthread_create(&th[t], 0, ranges_thread, &jobs[t]) == 0;
    if (!created[t]) ranges_thread(&jobs[t]);
  }
  for (int t = 0; t < threads; ++t)
    if (created[t]) pthread_join(th[t], 0);
  return 0;
}
