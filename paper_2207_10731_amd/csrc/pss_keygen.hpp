// Keygen of the sorted backward's grouping (paper Sec. 3, Alg. 1: lookups
// with equal tokens are grouped before their gradient rows are summed),
// shared by the grouping's own keygen kernel and by the streamed forward,
// which can run it while it reads the batch's index and offset entries.
//
// For every item e of a sort tile (kSortTile consecutive items) it writes
// the pair (h0, r): h0 = the item hash of (index, table), equal for equal
// tokens, and r = b*T + t, the pooled row of its bag; and the tile's counts
// of h0's low kSortBits bits, the first radix pass's histogram
// (counts[d * nblocks + tile]).
#pragma once

#include "pss_kernels.hpp"

namespace pss {

constexpr int kSortBits = 8;
constexpr int kBins = 1 << kSortBits;
constexpr int kSortItemsPerLane = 8;
constexpr int kSortTile = kBlockThreads * kSortItemsPerLane;  // keys per block
constexpr int kWaveSortKeys = kWave * kSortItemsPerLane;       // keys per wave

// indices[e] / offsets[g] with the integer width fixed at compile time;
// NT: non-temporal (a stream read once), else cached.
template <bool I32, bool NT = true>
__device__ __forceinline__ int64_t load_int(const void* a, uint64_t i) {
  if constexpr (I32) {
    const int32_t* q = static_cast<const int32_t*>(a) + i;
    return NT ? __builtin_nontemporal_load(q) : *q;
  } else {
    const int64_t* q = static_cast<const int64_t*>(a) + i;
    return NT ? __builtin_nontemporal_load(q) : *q;
  }
}

// LDS of keygen_process.
struct KeygenLds {
  uint32_t hist[kWavesPerBlock][kBins];
  int irregular;
};

// Inputs of one sort tile, requested ahead of their use (keygen_load), so
// that a workgroup can ask for its next tile's entries before it works on
// the current one.
struct KeygenIn {
  uint32_t ix[kSortItemsPerLane];
  int64_t ofs[kSortItemsPerLane];
  int64_t oend;
};

// Requests the thread's indices and offsets of sort tile `tile` (items
// [tile * kSortTile, ...)): every load is issued before any is used.  An
// item's index does not depend on its bag.
template <bool I32, bool NT>
__device__ __forceinline__ void keygen_load(const KParams& p, const void* __restrict__ indices,
                                            const void* __restrict__ offsets, const uint32_t tile,
                                            KeygenIn& in) {
  const int64_t tile0 = static_cast<int64_t>(tile) * kSortTile;
  const int in_tile = p.N - tile0 < kSortTile ? static_cast<int>(p.N - tile0) : kSortTile;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & (kWave - 1);
  const int lbase = w * kWaveSortKeys;
#pragma unroll
  for (int s = 0; s < kSortItemsPerLane; ++s) {
    const int li = lbase + s * kWave + lane;
    const int64_t e = tile0 + li;
    in.ix[s] = 0;
    in.ofs[s] = e;
    if (li < in_tile) {
      in.ix[s] = static_cast<uint32_t>(load_int<I32, NT>(indices, static_cast<uint64_t>(e)));
      in.ofs[s] = load_int<I32, NT>(offsets, static_cast<uint64_t>(e));
    }
  }
  const int64_t end = tile0 + in_tile;
  in.oend = threadIdx.x == 0 ? load_int<I32, NT>(offsets, static_cast<uint64_t>(end)) : end;
}

// Keygen of sort tile `tile` in item space, for batches with as many items
// as bags, from its requested inputs, by the whole workgroup (kBlockThreads
// threads; contains workgroup barriers, so every thread calls it with the
// same tile).  When every item of the tile is its own bag (offsets[e] == e),
// item e belongs to bag e; otherwise each item finds its bag by binary
// search over the offsets (the largest g with offsets[g] <= e).  With mean
// pooling it also writes inv_len[r] = 1 / |bag| for the row of every
// nonempty bag whose first item lies in the tile.
template <bool I32, bool NT>
__device__ __forceinline__ void keygen_process(const KParams& p, const void* __restrict__ offsets,
                                               uint32_t* __restrict__ keys,
                                               uint32_t* __restrict__ rows,
                                               float* __restrict__ inv_len,
                                               uint32_t* __restrict__ counts,
                                               const uint32_t nblocks, const uint32_t tile,
                                               const KeygenIn& in, KeygenLds& lds) {
  const int64_t tile0 = static_cast<int64_t>(tile) * kSortTile;
  const int in_tile = p.N - tile0 < kSortTile ? static_cast<int>(p.N - tile0) : kSortTile;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & (kWave - 1);
  const int lbase = w * kWaveSortKeys;
  const int64_t end = tile0 + in_tile;
  __syncthreads();  // a previous tile of this workgroup is done with the LDS
  for (int i = threadIdx.x; i < kWavesPerBlock * kBins; i += kBlockThreads)
    (&lds.hist[0][0])[i] = 0;
  if (threadIdx.x == 0) lds.irregular = 0;
  __syncthreads();
  bool mine_ok = in.oend == end;
#pragma unroll
  for (int s = 0; s < kSortItemsPerLane; ++s)
    if (in.ofs[s] != tile0 + lbase + s * kWave + lane) mine_ok = false;
  if (!mine_ok) lds.irregular = 1;
  __syncthreads();
  const bool onehot = lds.irregular == 0;
#pragma unroll
  for (int s = 0; s < kSortItemsPerLane; ++s) {
    const int li = lbase + s * kWave + lane;
    const bool valid = li < in_tile;
    uint32_t digit = 0;
    if (valid) {
      const int64_t e = tile0 + li;
      // bag numbers are below 2^32
      uint32_t g = static_cast<uint32_t>(e);
      float il = 1.f;
      bool first = true;
      if (!onehot) {
        uint64_t lo = 0, hi = p.num_bags - 1;  // largest g with offsets[g] <= e
        while (lo < hi) {
          const uint64_t mid = (lo + hi + 1) >> 1;
          if (load_int<I32, NT>(offsets, mid) <= e) lo = mid; else hi = mid - 1;
        }
        g = static_cast<uint32_t>(lo);
        const int64_t s0 = load_int<I32, NT>(offsets, lo);
        const int64_t s1 = load_int<I32, NT>(offsets, lo + 1);
        first = s0 == e;
        il = s1 > s0 ? 1.f / static_cast<float>(s1 - s0) : 1.f;
      }
      const uint32_t t = g / p.B;
      const uint32_t b = g - t * p.B;
      const uint32_t r = b * p.T + t;
      const uint32_t key = item_hash(in.ix[s], t * p.C, p.TC, p.a, p.b);
      keys[e] = key;
      rows[e] = r;
      if (p.mean && first) inv_len[r] = il;
      digit = key & (kBins - 1);
    }
    if (valid) atomicAdd(&lds.hist[w][digit], 1u);
  }
  __syncthreads();
  for (int d = threadIdx.x; d < kBins; d += kBlockThreads) {
    uint32_t c = 0;
#pragma unroll
    for (int ww = 0; ww < kWavesPerBlock; ++ww) c += lds.hist[ww][d];
    counts[static_cast<uint64_t>(d) * nblocks + tile] = c;
  }
}

}  // namespace pss
