// Host-only builds of libkvx for the sanitizer tests (no GPU code is built into
// them): the entry points that live in the HIP translation units, as stubs
// that report a HIP failure. Every host-side check before them still runs.
#include "kvx.h"
#include "kvx_internal.h"

namespace kvx {

kvx_status launch_copy(bool, const kvx_cache*, int32_t, int32_t, const int32_t*, const Geometry&,
                       void*, hipStream_t, int*, void*) {
  return KVX_EHIP;
}

kvx_status launch_copy_chunks(bool, const kvx_cache*, int32_t, int32_t, const int32_t*, int32_t,
                              const kvx_chunk_ref*, int32_t, int32_t, void*, int64_t, hipStream_t,
                              int*) {
  return KVX_EHIP;
}

int* stream_error_word(hipStream_t) { return nullptr; }

}  // namespace kvx

extern "C" kvx_status kvx_probe_stream(const void*, void*, int64_t, int32_t, hipStream_t) {
  return KVX_EHIP;
}

extern "C" kvx_status kvx_scatter_blocks_noalloc(const kvx_cache*, int32_t, int32_t, const int32_t*,
                                                 int32_t, int32_t, const void*, hipStream_t) {
  return KVX_EHIP;
}
