// kvsynth device fill: the same seeded byte streams as synth_host.c, written
// straight into device memory so that multi-GB KV-cache tensors can be filled
// in milliseconds. The definition (splitmix64 counter stream, bf16 normal
// quantile table or raw words) is stated in synth_host.c; the table comes from
// the host (kvs_normal_table) so both sides agree bit for bit.
//
// Not part of the KV transfer library: this only makes test and bench inputs.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ULL;

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

// Each thread writes 16 bytes (two consecutive 8-byte words) per step.
__global__ void __launch_bounds__(256) fill_kernel(uint64_t* __restrict__ out, uint64_t nwords,
                                                   uint64_t key, uint64_t w0, int mode,
                                                   const uint16_t* __restrict__ table) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x * 2;
  for (uint64_t i = ((uint64_t)blockIdx.x * blockDim.x + threadIdx.x) * 2; i < nwords;
       i += stride) {
    const int cnt = (i + 1 < nwords) ? 2 : 1;
    for (int q = 0; q < cnt; ++q) {
      uint64_t h = mix64(key + (w0 + i + q + 1ULL) * kGolden);
      if (mode == 0) {
        uint64_t v = 0;
        for (int e = 0; e < 4; ++e) v |= (uint64_t)table[(h >> (16 * e)) & 0xFFFFu] << (16 * e);
        h = v;
      }
      out[i + q] = h;
    }
  }
}

}  // namespace

extern "C" {

// Fill `nbytes` of device memory at `out` with bytes [byte_offset, byte_offset
// + nbytes) of stream `key` (from kvs_stream_key). `table` is a device copy of
// the 65,536-entry bf16 quantile table (needed only for mode 0). nbytes and
// byte_offset must be multiples of 8 and `out` 8-byte aligned. Enqueues on
// `stream`; returns a hipError_t value (0 on success).
int kvs_fill_device(void* out, uint64_t nbytes, uint64_t key, uint64_t byte_offset, int mode,
                    const void* table, hipStream_t stream) {
  if ((nbytes & 7) || (byte_offset & 7) || ((uintptr_t)out & 7) || (mode != 0 && mode != 1))
    return (int)hipErrorInvalidValue;
  if (mode == 0 && !table) return (int)hipErrorInvalidValue;
  if (nbytes == 0) return 0;
  if (!out) return (int)hipErrorInvalidValue;
  const uint64_t nwords = nbytes / 8;
  const uint64_t pairs = (nwords + 1) / 2;
  uint64_t blocks = (pairs + 255) / 256;
  if (blocks > 65536ULL * 8) blocks = 65536ULL * 8;
  hipLaunchKernelGGL(fill_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, (uint64_t*)out,
                     nwords, key, byte_offset / 8, mode, (const uint16_t*)table);
  return (int)hipGetLastError();
}

}  // extern "C"
