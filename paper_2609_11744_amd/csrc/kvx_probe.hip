// Measurement helper: the HBM rate that a kernel shaped like the slab mover
// (one workgroup per 4 KiB, 256 threads x one 16-byte vector, non-temporal
// loads and the kernels' streaming store,
// XCD-contiguous workgroup order) reaches on contiguous memory when it only
// reads, only writes, or copies. The bench reports these beside the spec peak,
// so the gap between a gather and 8 TB/s can be split into what any copy of
// this shape pays on the chip and what the gather's block-table indirection
// adds. Not part of the KV path.
#include <hip/hip_runtime.h>

#include "kvx.h"
#include "kvx_store.h"

namespace {

using kvx_dev::store_stream;
using kvx_dev::stream_dst;
using kvx_dev::v4u;

constexpr int kThreads = 256;
constexpr int kVec = 1;
constexpr int64_t kUnit = (int64_t)kThreads * kVec * 16;  // 4 KiB per workgroup
constexpr uint32_t kXcds = 8;
constexpr uint32_t kMaxUnitsPerLaunch = 1u << 22;

__device__ __forceinline__ uint32_t xcd_contiguous(uint32_t b, uint32_t n) {
  const uint32_t q = n / kXcds, r = n % kXcds, x = b % kXcds, k = b / kXcds;
  return x * q + (x < r ? x : r) + k;
}

// mode 0: read only (an empty asm statement that takes the loaded values
// keeps the loads; nothing is written); 1: write only; 2: copy src -> dst.
template <int kMode>
__global__ void __launch_bounds__(kThreads)
    probe_kernel(const v4u* __restrict__ src, v4u* __restrict__ dst, uint32_t unit_base,
                 uint32_t unit_count) {
  const uint64_t u = unit_base + xcd_contiguous(blockIdx.x, unit_count);
  const uint64_t base = u * (uint64_t)(kThreads * kVec) + threadIdx.x;
  const auto out = stream_dst(dst + u * (uint64_t)(kThreads * kVec), (uint32_t)kUnit);
  if (kMode == 1) {
    const v4u val = {(uint32_t)u, threadIdx.x, 0x9E3779B9u, 0x7F4A7C15u};
#pragma unroll
    for (int q = 0; q < kVec; ++q)
      store_stream(out, threadIdx.x + q * kThreads, val);
    return;
  }
  v4u r[kVec];
#pragma unroll
  for (int q = 0; q < kVec; ++q) r[q] = __builtin_nontemporal_load(src + base + q * kThreads);
  if (kMode == 2) {
#pragma unroll
    for (int q = 0; q < kVec; ++q)
      store_stream(out, threadIdx.x + q * kThreads, r[q]);
  } else {
    v4u acc = r[0];
#pragma unroll
    for (int q = 1; q < kVec; ++q) acc ^= r[q];
    __asm__ volatile("" : : "v"(acc.x), "v"(acc.y), "v"(acc.z), "v"(acc.w));
  }
}

}  // namespace

extern "C" kvx_status kvx_probe_stream(const void* src, void* dst, int64_t bytes, int32_t mode,
                                       hipStream_t stream) {
  if (bytes < 0 || bytes % kUnit != 0 || mode < 0 || mode > 2) return KVX_EINVAL;
  if ((mode != 1 && !src) || (mode != 0 && !dst)) return KVX_EINVAL;
  if (((uintptr_t)src & 15) || ((uintptr_t)dst & 15)) return KVX_EINVAL;
  const int64_t units = bytes / kUnit;
  if (units > 0x7FFFFFFF) return KVX_EINVAL;  // unit indexes are 32-bit
  for (int64_t base = 0; base < units; base += kMaxUnitsPerLaunch) {
    const uint32_t cnt = (uint32_t)(units - base < kMaxUnitsPerLaunch ? units - base
                                                                      : kMaxUnitsPerLaunch);
    const v4u* s = static_cast<const v4u*>(src);
    v4u* d = static_cast<v4u*>(dst);
    if (mode == 0)
      hipLaunchKernelGGL(probe_kernel<0>, dim3(cnt), dim3(kThreads), 0, stream, s, d,
                         (uint32_t)base, cnt);
    else if (mode == 1)
      hipLaunchKernelGGL(probe_kernel<1>, dim3(cnt), dim3(kThreads), 0, stream, s, d,
                         (uint32_t)base, cnt);
    else
      hipLaunchKernelGGL(probe_kernel<2>, dim3(cnt), dim3(kThreads), 0, stream, s, d,
                         (uint32_t)base, cnt);
    if (hipGetLastError() != hipSuccess) return KVX_EHIP;
  }
  return KVX_OK;
}
