// Host-side launchers of the PSS kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pss_kernels.hpp"

namespace pss {

// First stage of the grouping (keys, rows, the first radix pass's digit
// counts, inv_len with mean pooling) as laid out in its workspace; the
// streamed forward can write it (keys == nullptr: not requested).
struct KeygenOut {
  uint32_t* keys = nullptr;
  uint32_t* rows = nullptr;
  float* inv_len = nullptr;
  uint32_t* counts = nullptr;
  uint32_t nblocks = 0;
};
// Forward: pooled rows of every bag into out[B][T*d].
// indices / offsets are int64 (int32 when p.idx32); out / grad rows are
// float32 (bfloat16 when p.rows_bf16).  With kg (streamed kernel only, see
// forward_streams) the kernel also writes the grouping's first stage there.
hipError_t launch_forward(const void* w, bool bf16, const KParams& p, const void* indices,
                          const void* offsets, void* out, hipStream_t stream,
                          const KeygenOut* kg = nullptr);
// Whether the forward of this batch runs the streamed kernel.
bool forward_streams(const KParams& p, bool bf16);

// Atomic deposit: dst[addr] += scale * grad for every (item, dim).
hipError_t launch_deposit_atomic(float* dst, float scale, const KParams& p, const void* indices,
                                 const void* offsets, const void* grad, hipStream_t stream);

// Sorted deposit: lookups grouped by token (radix sort on the item hash),
// gradient rows summed per token, one deposit of scale * sum per token and
// 256-pair piece of the grouped order.  `workspace` must hold
// sorted_workspace_bytes(p) bytes.
size_t sorted_workspace_bytes(const KParams& p);
hipError_t launch_deposit_sorted(float* dst, float scale, const KParams& p, const void* indices,
                                 const void* offsets, const void* grad, void* workspace,
                                 hipStream_t stream);
// Its two halves.  The grouping depends on the indices, offsets and hash
// parameters only (not on grad or the shared array), so it may run ahead on
// another stream; it leaves the grouped pairs inside `workspace`.
struct GroupedPairs {
  const uint32_t* keys = nullptr;  // item hash h0 of each lookup, grouped
  const uint32_t* rows = nullptr;  // its pooled row b*T + t
  const float* inv_len = nullptr;  // 1 / |bag| per pooled row (mean pooling)
};
KeygenOut keygen_layout(const KParams& p, void* workspace);
// The rest of the grouping once its first stage is in the workspace
// (first_counted: the first pass's digit counts are there too).
hipError_t finish_group_sorted(const KParams& p, void* workspace, bool first_counted,
                               hipStream_t stream, GroupedPairs* out);
hipError_t launch_group_sorted(const KParams& p, const void* indices, const void* offsets,
                               void* workspace, hipStream_t stream, GroupedPairs* out);
// Events recorded around every later reduce-and-deposit launch (both null:
// none).
void set_reduce_events(hipEvent_t before, hipEvent_t after);

hipError_t launch_reduce_sorted(float* dst, float scale, const KParams& p, const GroupedPairs& g,
                                const void* grad, hipStream_t stream);

// Building blocks of the sorted path, shared with the sparse-gradient path.
// keygen: keys[e] = item part of the hash of lookup e, rows[e] = b*T + t;
// with mean pooling also inv_len[b*T + t] = 1 / |bag| (nonempty bags).
hipError_t launch_keygen(const KParams& p, const void* indices, const void* offsets,
                         uint32_t* keys, uint32_t* rows, float* inv_len, hipStream_t stream);
// Stable LSD radix sort of (keys, vals) by the `bits` bits from bit shift0
// up (8-bit digits); on return keys/vals point at whichever buffer pair holds
// the result.  scratch: radix_scratch_bytes(n) bytes.  With n_dev the number of
// pairs is min(n, *n_dev) (read on the device; n sizes the launch).  With
// first_counted the first pass's per-tile digit counts are already at the
// start of scratch (written while the keys were made).
size_t radix_scratch_bytes(int64_t n);
hipError_t radix_sort_pairs(uint32_t*& keys, uint32_t*& vals, uint32_t* ktmp, uint32_t* vtmp,
                            int64_t n, int bits, uint32_t* scratch, hipStream_t stream,
                            const uint32_t* n_dev = nullptr, bool first_counted = false,
                            int shift0 = 0);
// Bits of the item hash the grouping sort orders for N lookups.
int grouping_bits(int64_t N);

// Sparse gradient (Alg. 1 sparse branch): ascending unique locations and
// summed values into locations/values (at most `capacity` entries written),
// their count into *num_unique32 (device).  workspace:
// sparse_workspace_bytes(p) bytes.  Requires p.N * p.C < 2^31.
size_t sparse_workspace_bytes(const KParams& p);
hipError_t launch_gradient_sparse(const KParams& p, const void* indices, const void* offsets,
                                  const void* grad, void* workspace, uint32_t* locations,
                                  float* values, int64_t capacity, uint32_t* num_unique32,
                                  hipStream_t stream);
hipError_t launch_store_count(const uint32_t* total, int64_t* out, hipStream_t stream);
// Same pipeline, but SGD / Adagrad is applied at each unique location in
// place of writing the list (*num_unique32 still receives the count).
hipError_t launch_sparse_update(const KParams& p, const void* indices, const void* offsets,
                                const void* grad, void* workspace, uint32_t* num_unique32, void* w,
                                bool bf16, float* state, float lr, float eps, hipStream_t stream);

// Address-sorted deposit: every (lookup, dim) contribution becomes a record
// (address, scale * value), the records are radix-sorted by address tile
// (2^kAddrTileShift elements), each tile's records are summed in LDS and the
// tile is applied once: added to dst (fused SGD) or stored as the tile of a
// float32 gradient buffer dst of M elements (assign; no zero-fill needed).
// Requires p.N * p.d < 2^31.  workspace: addr_workspace_bytes(p) bytes.
constexpr int kAddrTileShift = 14;
size_t addr_workspace_bytes(const KParams& p);
hipError_t launch_deposit_addr(float* dst, bool assign, float scale, const KParams& p,
                               const void* indices, const void* offsets, const void* grad,
                               void* workspace, hipStream_t stream);

// Run sums by address: with the lookups grouped by token (g), every run
// sum becomes one record per chunk, the records are radix-sorted by address
// tile and each tile applies SGD or Adagrad (state != nullptr) to its
// elements directly; w is float32 or bfloat16 storage.  Requires Z >= 1,
// Z <= 4096 and p.N * p.C < 2^31.  workspace: runs_workspace_bytes(p).
size_t runs_workspace_bytes(const KParams& p);
hipError_t launch_deposit_runs(void* w, bool bf16, float* state, float lr, float eps,
                               const KParams& p, const GroupedPairs& g, const void* grad,
                               void* workspace, hipStream_t stream);
// The reduce stage writing records instead of depositing: payload rows
// (N x d floats), record keys and slots (N * C each).
hipError_t launch_reduce_records(float* payload, float scale, const KParams& p,
                                 const GroupedPairs& g, const void* grad, uint32_t* rkey,
                                 uint32_t* rval, hipStream_t stream);

// Dense optimizer pass over the M elements of a gradient buffer G (G[m] == 0
// leaves element m untouched).  state == nullptr selects SGD.
hipError_t launch_optimizer(void* w, bool bf16, float* state, const float* G, int64_t M, float lr,
                            float eps, hipStream_t stream);

// dst[0..n) = 0 with a fill kernel (no memset node, so the call can be
// captured into a graph).
hipError_t launch_zero(float* dst, int64_t n, hipStream_t stream);

// Chunk bases of every item into base_out[N][C] and/or sign factors
// (+1, -1, 0) into sign_out[N][C] (either may be null).
hipError_t launch_debug_addresses(const KParams& p, const void* indices, const void* offsets,
                                  uint32_t* base_out, int8_t* sign_out, hipStream_t stream);

}  // namespace pss
