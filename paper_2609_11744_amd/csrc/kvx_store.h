// The 16-byte store that the copy kernels and the bandwidth probe issue.
// Device code only; included by the HIP translation units.
#pragma once

#include <hip/hip_runtime.h>

#include <stdint.h>

namespace kvx_dev {

typedef unsigned int v4u __attribute__((ext_vector_type(4)));

// Cache-policy bits of a gfx950 vector-memory store: nt (non-temporal) and
// sc1, which together stream the line to memory at device scope. On the 80k
// gather and scatter patterns this measured 78.8 % and 74.0 % of the 8 TB/s
// peak against 77.0 % and 72.6 % with the plain non-temporal store (same
// kernel shape, same machine); the load's policy bits made no difference.
constexpr int kStorePolicy = 2 | 16;

// Buffer-resource word 3 of a raw (untyped, unswizzled) buffer on gfx9-family
// GPUs: 32-bit data format, no index stride.
constexpr int kRawBufferWord3 = 0x00020000;

// Destination of streaming stores: a buffer resource over the `bytes` bytes at
// base (a store outside them is dropped by the hardware rather than landing
// elsewhere). base and bytes must be wave-uniform, and the resource is made
// once, outside any divergent branch, so that it stays in scalar registers.
struct StreamDst {
  __amdgpu_buffer_rsrc_t rsrc;
};

__device__ __forceinline__ StreamDst stream_dst(v4u* base, uint32_t bytes) {
  // The values are the same in every lane; reading them from the first active
  // lane says so to the compiler, which otherwise may keep a value derived
  // from vector registers there and wrap every store in a loop over lanes.
  const uint64_t a = (uint64_t)base;
  const uint64_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  const uint64_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32));
  const int n = __builtin_amdgcn_readfirstlane((int)bytes);
  return StreamDst{
      __builtin_amdgcn_make_buffer_rsrc((void*)((hi << 32) | lo), 0, n, kRawBufferWord3)};
}

// Store v at vector i of the destination with kStorePolicy.
__device__ __forceinline__ void store_stream(const StreamDst& d, uint32_t i, v4u v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, d.rsrc, i * 16u, 0, kStorePolicy);
}

}  // namespace kvx_dev
