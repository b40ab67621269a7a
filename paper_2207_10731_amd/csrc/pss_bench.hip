// Measurement kernels that sit beside the PSS layer (libpss_bench.so, not
// part of the layer): a streaming copy of known size for calibrating traffic
// counters, and the bandwidth denominators of the roofline at each memory
// level (streaming reads and random 64-byte gathers, from a buffer that one
// XCD's L2 holds, from one the memory-side cache holds, and from HBM).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/pss_bench.h"

namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr uint32_t kXcds = 8;          // XCDs of an MI355X (workgroup b runs on XCD b mod 8)
constexpr uint32_t kBlocksPerCu = 8;   // resident workgroups per compute unit asked for

__global__ __launch_bounds__(kThreads) void copy_kernel(const f4* __restrict__ src, f4* __restrict__ dst,
                                                        const int64_t n) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kThreads;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; i < n; i += stride)
    __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

// Workgroups of slice s (workgroup b takes slice b mod slices) read the
// slice's n16 16-byte words `passes` times with ordinary (cached) loads.
__global__ __launch_bounds__(kThreads) void read_kernel(const f4* __restrict__ buf, const int64_t n16,
                                                        const int passes, const uint32_t slices,
                                                        float* __restrict__ sink) {
  const uint32_t s = blockIdx.x % slices;
  const int64_t per = gridDim.x / slices;
  const int64_t bi = blockIdx.x / slices;
  const f4* base = buf + static_cast<int64_t>(s) * n16;
  const int64_t stride = per * kThreads;
  float acc = 0.f;
  for (int pass = 0; pass < passes; ++pass) {
#pragma unroll 8
    for (int64_t i = bi * kThreads + threadIdx.x; i < n16; i += stride) {
      const f4 x = base[i];
      acc += x.x + x.y + x.z + x.w;
    }
  }
  if (acc == -1.2345e-37f) sink[threadIdx.x] = acc;  // keeps the loads; never true for the fill used
}

// Each group of 16 lanes reads 16 consecutive floats (64 bytes, at any
// 4-byte offset, as a chunk of Z = 16 weights) at `iters` pseudo-random
// positions of its slice.
__global__ __launch_bounds__(kThreads) void gather_kernel(const float* __restrict__ buf,
                                                          const int64_t slice_floats,
                                                          const int iters, const uint32_t slices,
                                                          const uint32_t seed, float* __restrict__ sink) {
  const uint32_t s = blockIdx.x % slices;
  const float* base = buf + static_cast<int64_t>(s) * slice_floats;
  const int sub = threadIdx.x & 15;
  const uint32_t group = (blockIdx.x * kThreads + threadIdx.x) >> 4;
  uint32_t x = group * 2654435761u ^ seed;  // per-group LCG state
  const uint64_t span = static_cast<uint64_t>(slice_floats - 16);
  float acc = 0.f;
#pragma unroll 8
  for (int it = 0; it < iters; ++it) {
    x = x * 1664525u + 1013904223u;
    const uint64_t off = (static_cast<uint64_t>(x) * span) >> 32;  // < span
    acc += base[off + sub];
  }
  if (acc == -1.2345e-37f) sink[threadIdx.x] = acc;
}

int cus_of_device() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
    return 256;
  return n;
}

}  // namespace

extern "C" {

int pss_bench_copy(void* dst, const void* src, size_t bytes, hipStream_t stream) {
  if (dst == nullptr || src == nullptr || bytes % 16 != 0) return 1;
  if ((reinterpret_cast<uintptr_t>(dst) | reinterpret_cast<uintptr_t>(src)) % 16 != 0) return 1;
  const int64_t n = static_cast<int64_t>(bytes / 16);
  if (n == 0) return 0;
  const int64_t want = (n + kThreads - 1) / kThreads;
  const uint32_t grid = static_cast<uint32_t>(want < 4096 ? want : 4096);
  hipLaunchKernelGGL(copy_kernel, dim3(grid), dim3(kThreads), 0, stream, static_cast<const f4*>(src),
                     static_cast<f4*>(dst), n);
  return hipGetLastError() == hipSuccess ? 0 : 3;
}

int pss_bench_read(const void* buf, size_t bytes, int passes, int xcd_slices, float* sink,
                   hipStream_t stream) {
  const uint32_t slices = xcd_slices ? kXcds : 1u;
  if (buf == nullptr || sink == nullptr || passes < 1) return 1;
  if (reinterpret_cast<uintptr_t>(buf) % 16 != 0 || bytes == 0 || bytes % (16 * slices) != 0) return 1;
  const int64_t n16 = static_cast<int64_t>(bytes / 16 / slices);
  const uint32_t grid = static_cast<uint32_t>(cus_of_device()) * kBlocksPerCu;  // a multiple of 8
  hipLaunchKernelGGL(read_kernel, dim3(grid), dim3(kThreads), 0, stream, static_cast<const f4*>(buf),
                     n16, passes, slices, sink);
  return hipGetLastError() == hipSuccess ? 0 : 3;
}

int pss_bench_gather(const void* buf, size_t bytes, int iters, int xcd_slices, uint32_t seed,
                     float* sink, int64_t* gathers, hipStream_t stream) {
  const uint32_t slices = xcd_slices ? kXcds : 1u;
  if (buf == nullptr || sink == nullptr || gathers == nullptr || iters < 1) return 1;
  if (reinterpret_cast<uintptr_t>(buf) % 4 != 0 || bytes % (4 * slices) != 0) return 1;
  const int64_t slice_floats = static_cast<int64_t>(bytes / 4 / slices);
  if (slice_floats < 32 || slice_floats > (1ll << 32)) return 1;
  const uint32_t grid = static_cast<uint32_t>(cus_of_device()) * kBlocksPerCu;
  hipLaunchKernelGGL(gather_kernel, dim3(grid), dim3(kThreads), 0, stream,
                     static_cast<const float*>(buf), slice_floats, iters, slices, seed, sink);
  *gathers = static_cast<int64_t>(grid) * (kThreads / 16) * iters;
  return hipGetLastError() == hipSuccess ? 0 : 3;
}

}  // extern "C"
