// Host-side launchers of the PSS kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pss_kernels.hpp"

namespace pss {

// Forward: pooled rows of every bag into out[B][T*d].
hipError_t launch_forward(const void* w, bool bf16, const KParams& p, const int64_t* indices,
                          const int64_t* offsets, float* out, hipStream_t stream);

// Atomic deposit: dst[addr] += scale * grad for every (item, dim).
hipError_t launch_deposit_atomic(float* dst, float scale, const KParams& p, const int64_t* indices,
                                 const int64_t* offsets, const float* grad, hipStream_t stream);

// Sorted deposit: lookups grouped by token (radix sort on the item hash),
// gradient rows summed per token, one deposit of scale * sum per token and
// wavefront.  `workspace` must hold sorted_workspace_bytes(p.N) bytes.
size_t sorted_workspace_bytes(int64_t N);
hipError_t launch_deposit_sorted(float* dst, float scale, const KParams& p, const int64_t* indices,
                                 const int64_t* offsets, const float* grad, void* workspace,
                                 hipStream_t stream);

// Dense optimizer pass over the M elements of a gradient buffer G (G[m] == 0
// leaves element m untouched).  state == nullptr selects SGD.
hipError_t launch_optimizer(void* w, bool bf16, float* state, const float* G, int64_t M, float lr,
                            float eps, hipStream_t stream);

// dst[0..n) = 0 with a fill kernel (no memset node, so the call can be
// captured into a graph).
hipError_t launch_zero(float* dst, int64_t n, hipStream_t stream);

// Chunk bases of every item into base_out[N][C].
hipError_t launch_debug_addresses(const KParams& p, const int64_t* indices, const int64_t* offsets,
                                  uint32_t* base_out, hipStream_t stream);

}  // namespace pss
