// Streaming copy used to calibrate traffic counters (not part of the layer).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/pss_bench.h"

namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void copy_kernel(const f4* __restrict__ src, f4* __restrict__ dst,
                                                   const int64_t n) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * 256;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < n; i += stride)
    __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

}  // namespace

extern "C" int pss_bench_copy(void* dst, const void* src, size_t bytes, hipStream_t stream) {
  if (dst == nullptr || src == nullptr || bytes % 16 != 0) return 1;
  if ((reinterpret_cast<uintptr_t>(dst) | reinterpret_cast<uintptr_t>(src)) % 16 != 0) return 1;
  const int64_t n = static_cast<int64_t>(bytes / 16);
  if (n == 0) return 0;
  const int64_t want = (n + 255) / 256;
  const uint32_t grid = static_cast<uint32_t>(want < 4096 ? want : 4096);
  hipLaunchKernelGGL(copy_kernel, dim3(grid), dim3(256), 0, stream, static_cast<const f4*>(src),
                     static_cast<f4*>(dst), n);
  return hipGetLastError() == hipSuccess ? 0 : 3;
}
