// Sorted backward: group lookups by token, reduce, deposit once per token.
//
// Alg. 1's sparse branch (unique locations + scatter_add of the values onto
// them) made hardware-friendly.  Identical tokens of a table read identical
// chunk addresses, so their output-gradient rows can be summed first and the
// sum deposited once: with the skewed token frequencies of recommendation
// data this removes most of the deposits (and all of the hot spots).
//
//   keygen    item e -> (h0, r): h0 = item part of the hash (a * key0 + b
//             mod p, identical for identical tokens, 31 bits), r = b*T + t
//             the pooled row its gradient is read from.
//   sort      LSD radix sort of the (h0, r) pairs on the low 8, 16 or 24
//             bits of h0 (groups of at most ~8192 pairs), 8-bit digits, stable;
//             per pass a histogram kernel (two tiles per workgroup), a scan
//             of the per-tile digit counts (one workgroup per digit, or per
//             digit and chunk of 4096 tiles for long inputs) and a scatter
//             kernel whose per-wave ranks come from ballot matching (digit
//             counts by LDS integer adds; no atomics on the data path).
//   reduce    one workgroup per 256 consecutive sorted pairs: sort them by
//             the full h0 (bitonic network per wavefront, then a merge of
//             the four lists through LDS), accumulate the gradient rows of
//             each run of equal h0 in registers (lanes over the dims), then
//             add the run's sum at the run's hashed addresses with float
//             atomics.  A token spanning several pieces deposits one partial
//             sum per piece.
#include <hip/hip_ext.h>

#include <atomic>

#include "pss_keygen.hpp"
#include "pss_launch.hpp"

namespace pss {

constexpr int kDigitsPerThread = kBins / kBlockThreads;
static_assert(kBins % kBlockThreads == 0, "whole digits per thread in the scatter prologue");

// Sort tile of this workgroup.  Workgroups are dispatched to the XCDs in
// turn (workgroup i to XCD i mod kXcds), and each XCD has an L2 of its own.
// Numbered this way, XCD x takes the contiguous tiles [x * per_xcd,
// (x + 1) * per_xcd): the count words and digit runs of neighbouring tiles,
// which lie side by side in memory, are then written through one L2 and
// leave it as whole lines.  The grid holds kXcds * per_xcd workgroups;
// those whose tile is at or past the last do nothing.  Any other dispatch
// order only changes which L2 a tile's writes pass through.  per_xcd = 0
// keeps tile = workgroup: a sort whose live keys are counted on the device
// has its live tiles at the front, and contiguous ranges would put them all
// on the first XCDs.
__device__ __forceinline__ uint32_t sort_tile_index(const uint32_t per_xcd) {
  return per_xcd ? (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds : blockIdx.x;
}

// ---------------------------------------------------------------------------
// keygen
// ---------------------------------------------------------------------------
// With mean pooling it also writes inv_len[r] = 1 / |bag| for every pooled
// row r = b*T + t of a nonempty bag (each bag belongs to exactly one tile).
__global__ __launch_bounds__(kBlockThreads) void keygen_kernel(
    const KParams p, const void* __restrict__ indices, const void* __restrict__ offsets,
    uint32_t* __restrict__ keys, uint32_t* __restrict__ rows, float* __restrict__ inv_len) {
  const int lane = threadIdx.x & (kWave - 1);
  const uint64_t wave = static_cast<uint64_t>(blockIdx.x) * kWavesPerBlock + (threadIdx.x >> 6);
  const uint64_t g0 = wave * kTileBags;
  if (g0 >= p.num_bags) return;
  const Tile tl = load_tile(p, offsets, g0, lane);
  // pooled row index r = b*T + t of bag g0 + lane
  const uint64_t g = g0 + static_cast<uint64_t>(lane < tl.nb ? lane : 0);
  const uint32_t t = static_cast<uint32_t>(g / p.B);
  const uint32_t b = static_cast<uint32_t>(g - static_cast<uint64_t>(t) * p.B);
  const uint32_t rr = b * p.T + t;
  if (p.mean && lane < tl.nb && tl.len) inv_len[rr] = 1.f / static_cast<float>(tl.len);
  if (__ballot(lane >= tl.nb || tl.len == 1) == ~0ull) {
    // one-hot tile: item E0 + l belongs to bag l
    if (lane < tl.nb) {
      const int64_t e = tl.E0 + lane;
      keys[e] = item_hash(load_index(indices, e, p.idx32), tl.tC, p.TC, p.a, p.b);
      rows[e] = rr;
    }
    return;
  }
  for (int64_t blk = tl.E0; blk < tl.E1; blk += kWave) {
    const int64_t rem = tl.E1 - blk;
    const int n = rem < kWave ? static_cast<int>(rem) : kWave;
    const int64_t e = blk + lane;
    const int bag = bag_of_item(tl, e);
    const uint32_t tC = __shfl(tl.tC, bag);
    const uint32_t r = __shfl(rr, bag);
    if (lane < n) {
      const uint32_t i = load_index(indices, e, p.idx32);
      keys[e] = item_hash(i, tC, p.TC, p.a, p.b);
      rows[e] = r;
    }
  }
}

// ---------------------------------------------------------------------------
// radix sort pieces
// ---------------------------------------------------------------------------

// Lanes holding the same digit as this lane (among lanes with `valid`).
__device__ __forceinline__ uint64_t match_digit(uint32_t digit, bool valid) {
  uint64_t eq = __ballot(valid);
#pragma unroll
  for (int bit = 0; bit < kSortBits; ++bit) {
    const uint64_t m = __ballot((digit >> bit) & 1u);
    eq &= ((digit >> bit) & 1u) ? m : ~m;
  }
  return eq;
}

__device__ __forceinline__ uint64_t lanes_below(int lane) {
  return lane == 0 ? 0ull : (~0ull >> (kWave - lane));
}

// Number of keys to sort: the host's count, or fewer when the caller keeps
// the real count in device memory (the host count is then an upper bound).
__device__ __forceinline__ int64_t live_count(int64_t n, const uint32_t* n_dev) {
  if (n_dev == nullptr) return n;
  const int64_t d = *n_dev;
  return d < n ? d : n;
}

// counts[d * nblocks + tile] = number of keys of the tile with digit d.
// A workgroup counts kHistTiles consecutive tiles (kHistKeysPerLane keys
// per lane, all requested before any is counted), so that more of the keys
// are in flight at once.  `pair` numbering follows
// sort_tile_index over the groups of tiles.
constexpr int kHistTiles = 2;
constexpr int kHistWavesPerTile = kWavesPerBlock / kHistTiles;
constexpr int kHistKeysPerLane = kSortTile * kHistTiles / kBlockThreads;
constexpr int kHistWaveKeys = kHistKeysPerLane * kWave;
static_assert(kHistWavesPerTile * kHistTiles == kWavesPerBlock, "whole wavefronts per tile");
__global__ __launch_bounds__(kBlockThreads) void sort_hist_kernel(
    const uint32_t* __restrict__ keys, int64_t n, const int shift,
    uint32_t* __restrict__ counts, const uint32_t nblocks, const uint32_t per_xcd,
    const uint32_t* __restrict__ n_dev) {
  const uint32_t group = sort_tile_index(per_xcd);
  const uint32_t tile0 = group * kHistTiles;
  if (tile0 >= nblocks) return;
  n = live_count(n, n_dev);
  // no live key in these tiles: the scan reads the live tiles' counts only
  if (static_cast<int64_t>(tile0) * kSortTile >= n) return;
  __shared__ uint32_t hist[kWavesPerBlock][kBins];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & (kWave - 1);
  for (int i = threadIdx.x; i < kWavesPerBlock * kBins; i += kBlockThreads) (&hist[0][0])[i] = 0;
  const int64_t base = static_cast<int64_t>(tile0) * kSortTile + w * kHistWaveKeys;
  uint32_t kx[kHistKeysPerLane];
#pragma unroll
  for (int s = 0; s < kHistKeysPerLane; ++s) {
    const int64_t idx = base + s * kWave + lane;
    kx[s] = idx < n ? keys[idx] : 0u;
  }
  __syncthreads();
#pragma unroll
  for (int s = 0; s < kHistKeysPerLane; ++s) {
    const bool valid = base + s * kWave + lane < n;
    const uint32_t digit = (kx[s] >> shift) & (kBins - 1);
    // counts are order-free: LDS integer adds (fewer instructions than
    // ballot matching; measured 404 -> 260 us on 218 M keys)
    if (valid) atomicAdd(&hist[w][digit], 1u);
  }
  __syncthreads();
  const int d = threadIdx.x;  // one digit per thread
#pragma unroll
  for (int t = 0; t < kHistTiles; ++t) {
    const uint32_t tile = tile0 + t;
    if (tile < nblocks && static_cast<int64_t>(tile) * kSortTile < n) {
      uint32_t c = 0;
#pragma unroll
      for (int i = 0; i < kHistWavesPerTile; ++i) c += hist[kHistWavesPerTile * t + i][d];
      counts[static_cast<uint64_t>(d) * nblocks + tile] = c;
    }
  }
}

// Keygen in item space for batches with as many items as bags, fused with
// the first radix pass's histogram: one sort tile per workgroup.
template <bool I32>
__global__ __launch_bounds__(kBlockThreads) void keygen_hist_kernel(
    const KParams p, const void* __restrict__ indices, const void* __restrict__ offsets,
    uint32_t* __restrict__ keys, uint32_t* __restrict__ rows, float* __restrict__ inv_len,
    uint32_t* __restrict__ counts, const uint32_t nblocks, const uint32_t per_xcd) {
  const uint32_t tile = sort_tile_index(per_xcd);
  if (tile >= nblocks) return;
  __shared__ KeygenLds lds;
  KeygenIn in;
  keygen_load<I32, true>(p, indices, offsets, tile, in);
  keygen_process<I32, true>(p, offsets, keys, rows, inv_len, counts, nblocks, tile, in, lds);
}

// Scans of the count rows.  A chunk of kScanChunk consecutive entries is
// scanned by the workgroup's wavefronts, each a contiguous quarter read and
// written 64 entries (one line) per instruction.
constexpr int kScanPerThread = 16;
constexpr uint32_t kScanChunk = kBlockThreads * kScanPerThread;
constexpr uint32_t kScanWaveEntries = kScanChunk / kWavesPerBlock;

// Exclusive scan in place of row[c0, min(c0 + kScanChunk, end)), every
// entry raised by `carry`; returns the chunk's sum.
__device__ __forceinline__ uint32_t scan_chunk(uint32_t* __restrict__ row, const uint32_t c0,
                                               const uint32_t end, const uint32_t carry,
                                               uint32_t* wsum) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & (kWave - 1);
  const uint32_t q0 = c0 + w * kScanWaveEntries;
  uint32_t v[kScanPerThread];
#pragma unroll
  for (int j = 0; j < kScanPerThread; ++j) {
    const uint32_t i = q0 + j * kWave + lane;
    v[j] = i < end ? row[i] : 0u;
  }
  uint32_t run = 0;  // sum of the wavefront's earlier groups of 64
#pragma unroll
  for (int j = 0; j < kScanPerThread; ++j) {
    uint32_t x = v[j];
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      const uint32_t y = __shfl_up(x, off);
      if (lane >= off) x += y;
    }
    const uint32_t excl = run + x - v[j];
    run += __shfl(x, kWave - 1);
    v[j] = excl;
  }
  if (lane == 0) wsum[w] = run;
  __syncthreads();
  uint32_t before = carry, all = 0;
#pragma unroll
  for (int ww = 0; ww < kWavesPerBlock; ++ww) {
    before += ww < w ? wsum[ww] : 0u;
    all += wsum[ww];
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kScanPerThread; ++j) {
    const uint32_t i = q0 + j * kWave + lane;
    if (i < end) row[i] = before + v[j];
  }
  return all;
}

__device__ __forceinline__ uint32_t live_tiles(int64_t n, const uint32_t* n_dev, uint32_t nblocks) {
  n = live_count(n, n_dev);
  const uint64_t live = (static_cast<uint64_t>(n) + kSortTile - 1) / kSortTile;
  return live < nblocks ? static_cast<uint32_t>(live) : nblocks;
}

// Row d of counts (one digit, one entry per tile): exclusive scan in place
// over the tiles that hold live keys (the others are never read: their
// scatter workgroups exit at once); totals[d] = the row's sum.  One
// workgroup per digit, for rows of a few chunks.
__global__ __launch_bounds__(kBlockThreads) void sort_scan_kernel(uint32_t* __restrict__ counts,
                                                                  const uint32_t nblocks,
                                                                  uint32_t* __restrict__ totals,
                                                                  int64_t n,
                                                                  const uint32_t* __restrict__ n_dev) {
  __shared__ uint32_t wsum[kWavesPerBlock];
  const uint32_t ntiles = live_tiles(n, n_dev, nblocks);
  uint32_t* row = counts + static_cast<uint64_t>(blockIdx.x) * nblocks;
  uint32_t carry = 0;
  for (uint32_t c0 = 0; c0 < ntiles; c0 += kScanChunk) carry += scan_chunk(row, c0, ntiles, carry, wsum);
  if (threadIdx.x == 0) totals[blockIdx.x] = carry;
}

// Longer rows: grid (chunk, digit).  sort_scan_sums_kernel writes each
// chunk's sum into partial[digit * nchunks + chunk]; sort_scan_apply_kernel
// scans the chunk after the sums of the row's earlier chunks, and the last
// live chunk writes totals[digit].
__global__ __launch_bounds__(kBlockThreads) void sort_scan_sums_kernel(
    const uint32_t* __restrict__ counts, const uint32_t nblocks, uint32_t* __restrict__ partial,
    int64_t n, const uint32_t* __restrict__ n_dev) {
  __shared__ uint32_t wsum[kWavesPerBlock];
  const uint32_t ntiles = live_tiles(n, n_dev, nblocks);
  const uint32_t c0 = blockIdx.x * kScanChunk;
  if (c0 >= ntiles) return;
  const uint32_t* row = counts + static_cast<uint64_t>(blockIdx.y) * nblocks;
  uint32_t sum = 0;
#pragma unroll
  for (int j = 0; j < kScanPerThread; ++j) {
    const uint32_t i = c0 + j * kBlockThreads + threadIdx.x;
    sum += i < ntiles ? row[i] : 0u;
  }
  uint32_t tot;
  block_exclusive_scan(sum, wsum, &tot);
  if (threadIdx.x == 0) partial[static_cast<uint64_t>(blockIdx.y) * gridDim.x + blockIdx.x] = tot;
}
__global__ __launch_bounds__(kBlockThreads) void sort_scan_apply_kernel(
    uint32_t* __restrict__ counts, const uint32_t nblocks, const uint32_t* __restrict__ partial,
    uint32_t* __restrict__ totals, int64_t n, const uint32_t* __restrict__ n_dev) {
  __shared__ uint32_t wsum[kWavesPerBlock];
  const uint32_t ntiles = live_tiles(n, n_dev, nblocks);
  const uint32_t c0 = blockIdx.x * kScanChunk;
  if (c0 >= ntiles) return;
  const uint32_t* prow = partial + static_cast<uint64_t>(blockIdx.y) * gridDim.x;
  uint32_t pre = 0;  // sum of the row's earlier chunks (each thread a strided share)
  for (uint32_t c = threadIdx.x; c < blockIdx.x; c += kBlockThreads) pre += prow[c];
  uint32_t carry;
  block_exclusive_scan(pre, wsum, &carry);
  uint32_t* row = counts + static_cast<uint64_t>(blockIdx.y) * nblocks;
  const uint32_t tot = scan_chunk(row, c0, ntiles, carry, wsum);
  if (threadIdx.x == 0 && c0 + kScanChunk >= ntiles) totals[blockIdx.y] = carry + tot;
}

// Stable scatter of one tile by digit into its global slots.  The tile is
// first reordered by digit in LDS, then written out with consecutive threads
// on consecutive slots of a digit's run, so that stores coalesce.
static_assert(kDigitsPerThread == 1, "one digit per thread in the scatter prologue");
//
// At most 4 wavefronts per SIMD: with more resident tiles (7, which its
// registers and LDS would allow) the large sorts slowed down (218 M keys:
// 1282 -> 1469 us per pass), at 2 or 3 every size did.
__global__ __launch_bounds__(kBlockThreads) __attribute__((amdgpu_waves_per_eu(1, 4))) void sort_scatter_kernel(
    const uint32_t* __restrict__ keys_in, const uint32_t* __restrict__ vals_in,
    uint32_t* __restrict__ keys_out, uint32_t* __restrict__ vals_out, int64_t n,
    const int shift, const uint32_t* __restrict__ offsets, const uint32_t nblocks,
    const uint32_t* __restrict__ totals, const uint32_t per_xcd,
    const uint32_t* __restrict__ n_dev) {
  const uint32_t tile = sort_tile_index(per_xcd);
  if (tile >= nblocks) return;
  n = live_count(n, n_dev);
  // tiles wholly past the live keys hold nothing (their counts are zero)
  const int64_t tile0 = static_cast<int64_t>(tile) * kSortTile;
  if (tile0 >= n) return;
  const int in_tile = n - tile0 < kSortTile ? static_cast<int>(n - tile0) : kSortTile;
  __shared__ uint32_t cur[kWavesPerBlock][kBins];
  __shared__ uint32_t gdst[kBins];  // global slot of the digit's run minus its LDS start
  __shared__ uint32_t wsum[kWavesPerBlock];
  __shared__ uint32_t sk[kSortTile], sv[kSortTile];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & (kWave - 1);
  for (int i = threadIdx.x; i < kWavesPerBlock * kBins; i += kBlockThreads) (&cur[0][0])[i] = 0;
  __syncthreads();
  const int lbase = w * kWaveSortKeys;
  // thread d owns digit d: its totals and this tile's offset are requested
  // with the tile's pairs (one wait for memory)
  const int d = threadIdx.x;
  const uint32_t total_d = totals[d];
  const uint32_t offset_d = offsets[static_cast<uint64_t>(d) * nblocks + tile];
  uint32_t k[kSortItemsPerLane], v[kSortItemsPerLane];
#pragma unroll
  for (int s = 0; s < kSortItemsPerLane; ++s) {
    const int li = lbase + s * kWave + lane;
    k[s] = li < in_tile ? keys_in[tile0 + li] : 0u;
    v[s] = li < in_tile ? vals_in[tile0 + li] : 0u;
  }
  // per-wave digit counts (LDS integer adds; the stable ranks below come
  // from ballot matching)
#pragma unroll
  for (int s = 0; s < kSortItemsPerLane; ++s) {
    const bool valid = lbase + s * kWave + lane < in_tile;
    const uint32_t digit = (k[s] >> shift) & (kBins - 1);
    if (valid) atomicAdd(&cur[w][digit], 1u);
  }
  __syncthreads();
  // digit d's LDS run starts after the tile's smaller digits; its global
  // run after all smaller digits and earlier tiles
  uint32_t here = 0;
#pragma unroll
  for (int ww = 0; ww < kWavesPerBlock; ++ww) here += cur[ww][d];
  uint32_t unused;
  const uint32_t local0 = block_exclusive_scan(here, wsum, &unused);
  const uint32_t global0 = block_exclusive_scan(total_d, wsum, &unused) + offset_d;
  gdst[d] = global0 - local0;  // modulo 2^32; slot = gdst + LDS index
  uint32_t run = local0;
#pragma unroll
  for (int ww = 0; ww < kWavesPerBlock; ++ww) {
    const uint32_t c = cur[ww][d];
    cur[ww][d] = run;
    run += c;
  }
  __syncthreads();
#pragma unroll
  for (int s = 0; s < kSortItemsPerLane; ++s) {
    const bool valid = lbase + s * kWave + lane < in_tile;
    const uint32_t digit = (k[s] >> shift) & (kBins - 1);
    const uint64_t eq = match_digit(digit, valid);
    if (valid) {
      const uint32_t li = cur[w][digit] + static_cast<uint32_t>(__popcll(eq & lanes_below(lane)));
      sk[li] = k[s];
      sv[li] = v[s];
    }
    // all lanes have read cur[w][digit] above; group leaders advance it
    if (valid && (eq & lanes_below(lane)) == 0) cur[w][digit] += __popcll(eq);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < in_tile; i += kBlockThreads) {
    const uint32_t key = sk[i];
    const uint32_t pos = gdst[(key >> shift) & (kBins - 1)] + static_cast<uint32_t>(i);
    if (pos < n) {  // always true when the counts agree; guards memory anyway
      keys_out[pos] = key;
      vals_out[pos] = sv[i];
    }
  }
}

// ---------------------------------------------------------------------------
// segmented reduction + deposit
// ---------------------------------------------------------------------------
// One workgroup per piece of kPiece = 256 consecutive pairs of the grouped
// order, with two kinds of wavefronts:
//
//  * 4 readers.  Each sorts 64 pairs by the full key in registers (bitonic);
//    the four sorted lists are merged through LDS (a pair's rank is its own
//    index plus, per other list, how many of that list's pairs precede it: a
//    7-step binary search), so every token of the piece forms one run.  A
//    reader then walks its quarter of the merged order U rows at a time,
//    sums the gradient rows of each run in registers (lanes over the dims)
//    and hands every finished run sum to its depositor through LDS.
//  * 4 depositors.  Each adds the run sums of its reader at the runs' hashed
//    addresses with float atomics.
//
// Why two kinds: on gfx9 loads and atomics count in one in-order wait
// counter, so a wavefront that did both would wait for its last batch's
// atomics (which resolve far away, at the memory side) before it could use
// its next batch's rows.  Split, the readers' waits cover loads only and the
// depositors never wait for memory at all.  Readers and depositors step in
// phases separated by workgroup barriers (LDS-only fences: no wait for the
// atomics); in phase k a reader fills buffer k mod 2 while its depositor
// drains buffer (k-1) mod 2.  Rows of batch k+1 are requested before batch
// k is summed.  A run crossing a quarter boundary leaves one partial sum per
// quarter in LDS and is deposited once, after the last phase.
constexpr int kPiece = 256;                 // pairs per workgroup
constexpr int kReaders = kPiece / kWave;    // 4
constexpr int kReduceThreads = 2 * kPiece;  // readers + depositors
constexpr int kSlotFloats = 1024;           // per buffer: U run sums of 64 * EPL dims

// How many of the 64 sorted keys in `list` precede `key`: all smaller keys,
// and equal keys too when `ties` (the list comes earlier in merge order).
__device__ __forceinline__ int count_before(const uint32_t* list, uint32_t key, bool ties) {
  int c = 0;
#pragma unroll
  for (int step = kWave; step >= 1; step >>= 1) {
    if (c + step <= kWave) {
      const uint32_t k = list[c + step - 1];
      if (k < key || (ties && k == key)) c += step;
    }
  }
  return c;
}

// Workgroup barrier whose fences cover LDS only: global atomics in flight
// are not waited for.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Rows of U merged positions (q .. q+U-1 of the quarter, clamped to its last
// position) into g; lanes over the dims, mean pooling applied.
template <int EPL, int U, typename GT>
__device__ __forceinline__ void load_rows(float (&g)[U][EPL], const GT* __restrict__ grad,
                                          const float* __restrict__ inv_len, const KParams& p,
                                          uint32_t wr, int q, int nq, uint32_t c0, int lane,
                                          const bool* act) {
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int uu = q + u < nq ? q + u : nq - 1;
    const uint32_t ru = readlane_u32(wr, uu);
    const GT* grow = grad + static_cast<uint64_t>(ru) * p.d;
    const float il = p.mean ? inv_len[ru] : 1.f;
#pragma unroll
    for (int r = 0; r < EPL; ++r) {
      const float x = load_row(grow, act[r] ? c0 + lane + kWave * r : 0u);
      g[u][r] = p.mean ? x * il : x;
    }
  }
}

// Sums the rows of positions q .. q+U-1 into acc; every run that ends there
// goes to the buffer (values, key), except the quarter's first run while
// `head` is set (it continues a run of the previous quarter): that one goes
// to headv and clears `head`.  Returns the number of runs put in the buffer.
//
// With REC the merged position of each buffered run's first pair goes to
// rst[] (run_start: first position of the run in progress, updated as runs
// end; q0 is the quarter's first position in the piece).
template <int EPL, int U, bool REC = false>
__device__ __forceinline__ int sum_runs(const float (&g)[U][EPL], float* acc, uint32_t wk, int q,
                                        int nq, uint32_t after, float* vals, uint32_t* rkeys,
                                        bool& head, float* headv, int lane, uint32_t* rst = nullptr,
                                        uint32_t* run_start = nullptr, int q0 = 0) {
  int nrun = 0;
#pragma unroll
  for (int u = 0; u < U; ++u) {
    if (q + u < nq) {
#pragma unroll
      for (int r = 0; r < EPL; ++r) acc[r] += g[u][r];
      const uint32_t h = readlane_u32(wk, q + u);
      const uint32_t hn = q + u + 1 < nq ? readlane_u32(wk, q + u + 1) : after;
      if (hn != h) {
        float* dstv = head ? headv : vals + nrun * (kWave * EPL);
#pragma unroll
        for (int r = 0; r < EPL; ++r) {
          dstv[kWave * r + lane] = acc[r];
          acc[r] = 0.f;
        }
        if (head) {
          head = false;
        } else {
          if (lane == 0) {
            rkeys[nrun] = h;
            if (REC) rst[nrun] = *run_start;
          }
          ++nrun;
        }
        if (REC) *run_start = static_cast<uint32_t>(q0 + q + u + 1);
      }
    }
  }
  return nrun;
}

// Adds scale * v (lane's EPL values of the run with item hash h) at the
// run's hashed addresses.
template <int EPL, bool SIGN>
__device__ __forceinline__ void deposit_run(float* __restrict__ dst, float scale, const KParams& p,
                                            uint32_t h, const float* v, const bool* act,
                                            const uint32_t* step, const uint32_t* step2,
                                            const uint32_t* kk) {
  const uint32_t h20 = SIGN ? sign_hash0(h, p.s_alpha, p.s_beta) : 0u;
#pragma unroll
  for (int r = 0; r < EPL; ++r) {
    if (!act[r]) continue;
    const uint32_t ent = chunk_entry<SIGN>(fast_mod(add_mod_p(h, step[r]), p.fm_c, p.M),
                                           add_mod_p(h20, step2[r]), p);
    const Elem el = elem_of<SIGN>(ent, kk[r], p.M);
    const float x = scale * v[r];
    if (!SIGN || el.read) unsafeAtomicAdd(dst + el.m, SIGN ? apply_sign(x, el) : x);
  }
}

// Record form of deposit_run: the lane's EPL values of the run, scaled and
// signed per chunk (0 for a chunk that is not read), become row `slot_row`
// of the payload array (d floats per row).
template <int EPL, bool SIGN>
__device__ __forceinline__ void record_run(float* __restrict__ payload, float scale,
                                           const KParams& p, uint32_t h, uint64_t slot_row,
                                           const float* v, const bool* act, const uint32_t* step,
                                           const uint32_t* step2, const uint32_t* kk,
                                           uint32_t c0, int lane) {
  const uint32_t h20 = SIGN ? sign_hash0(h, p.s_alpha, p.s_beta) : 0u;
#pragma unroll
  for (int r = 0; r < EPL; ++r) {
    if (!act[r]) continue;
    float x = scale * v[r];
    if (SIGN) {
      const uint32_t ent = chunk_entry<SIGN>(fast_mod(add_mod_p(h, step[r]), p.fm_c, p.M),
                                             add_mod_p(h20, step2[r]), p);
      x = apply_sign(x, elem_of<SIGN>(ent, kk[r], p.M));
    }
    payload[slot_row * p.d + c0 + lane + kWave * r] = x;
  }
}

// Without REC: the reduce-and-deposit kernel described above (dst, scale).
// With REC (run sums deposited by address): no atomics; every run of the
// piece becomes one record per chunk, slot (p0 + i) * C + j for the run's
// first merged position i and chunk j: payload row p0 + i holds the run's
// scaled, signed sum (dst is the payload array, N x d floats), rkey[slot] the
// chunk's base (kNoRecord for a chunk that is not read and for every
// position that starts no run), rval[slot] = slot.
constexpr uint32_t kNoRecord = 0xffffffffu;
template <int EPL, int U, bool SIGN, typename GT, bool REC>
__global__ __launch_bounds__(kReduceThreads) void reduce_deposit_kernel(
    float* __restrict__ dst, const float scale, const KParams p,
    const uint32_t* __restrict__ keys, const uint32_t* __restrict__ rows,
    const GT* __restrict__ grad, const float* __restrict__ inv_len, const int64_t n,
    uint32_t* __restrict__ rkey, uint32_t* __restrict__ rval) {
  static_assert(U * kWave * EPL == kSlotFloats, "a buffer holds U run sums");
  const int lane = threadIdx.x & (kWave - 1);
  const int w = static_cast<int>(__builtin_amdgcn_readfirstlane(threadIdx.x >> 6));
  const bool reader = w < kReaders;
  const int pair = reader ? w : w - kReaders;
  const int64_t p0 = static_cast<int64_t>(blockIdx.x) * kPiece;
  if (p0 >= n) return;  // whole workgroup
  const int cnt = n - p0 < kPiece ? static_cast<int>(n - p0) : kPiece;
  const uint32_t c0 = blockIdx.y * (kWave * EPL);
  // The readers' sorted lists and the merged order; once every reader holds
  // its quarter in registers the same LDS takes the partial sums of runs
  // that cross a quarter boundary (headv: the part in the quarter where the
  // run ends, tailv: the part in the quarter it leaves).
  constexpr int kRowF = kWave * EPL;
  constexpr int kSortWords = 4 * kPiece;
  constexpr int kPartWords = 2 * kReaders * kRowF;
  __shared__ uint32_t sortbuf[kSortWords > kPartWords ? kSortWords : kPartWords];
  uint32_t* lk = sortbuf;
  uint32_t* lr = sortbuf + kPiece;
  uint32_t* mk = sortbuf + 2 * kPiece;
  uint32_t* mr = sortbuf + 3 * kPiece;
  float* headv = reinterpret_cast<float*>(sortbuf);
  float* tailv = headv + kReaders * kRowF;
  __shared__ float vals[kReaders][2][kSlotFloats];
  __shared__ uint32_t rkeys[kReaders][2][U];
  __shared__ int nruns[kReaders][2];
  __shared__ uint32_t qkey[kReaders];  // key at the start of each quarter
  __shared__ int qflags[kReaders];     // bit 0: tail open, bit 1: through (no run ends inside)
  __shared__ uint32_t rst[kReaders][2][REC ? U : 1];  // REC: first position of each buffered run
  __shared__ uint32_t lastst[kReaders];               // REC: first position of the open run

  bool act[EPL];
#pragma unroll
  for (int r = 0; r < EPL; ++r) act[r] = c0 + lane + kWave * r < p.d;

  // 1. readers sort their pairs; empty slots hold key 0xffffffff (above any
  //    hash) and stay behind every real pair
  const int my = pair * kWave + lane;
  uint32_t key = 0xffffffffu, row = 0;
  if (reader) {
    if (my < cnt) {
      key = keys[p0 + my];
      row = rows[p0 + my];
      if (row >= p.num_bags) row = 0;  // rows come from keygen; clamp keeps reads in bounds
    }
    wave_sort_pairs(key, row, lane);
    lk[my] = key;
    lr[my] = row;
  }
  lds_barrier();
  // 2. merge: stable across lists (equal keys of an earlier list first)
  if (reader) {
    int rank = lane;
#pragma unroll
    for (int v = 0; v < kReaders; ++v)
      if (v != w) rank += count_before(lk + v * kWave, key, v < w);
    mk[rank] = key;
    mr[rank] = row;
  }
  lds_barrier();

  // 3. phases: reader sums batch k into buffer k&1, depositor drains the
  //    other buffer.  Every wavefront runs the same number of phases.  A run
  //    that crosses from one quarter into the next is not cut: its part in
  //    each quarter goes to tailv / headv and is deposited once at the end.
  const int q0 = pair * kWave;
  const int nq = cnt - q0 < kWave ? (cnt - q0 > 0 ? cnt - q0 : 0) : kWave;
  constexpr int kBatches = kWave / U;
  uint32_t wk = 0xffffffffu, wr = 0;
  bool head_open = false, tail_open = false;
  uint32_t after = 0xffffffffu;
  if (reader && nq > 0) {
    wk = mk[my];
    wr = mr[my];
    head_open = q0 > 0 && mk[q0] == mk[q0 - 1];
    if (q0 + nq < cnt && mk[q0 + nq] == mk[q0 + nq - 1]) {
      tail_open = true;
      after = mk[q0 + nq];  // the run goes on past the quarter
    }
    if (lane == 0) qkey[pair] = mk[q0];
    if (REC && blockIdx.y == 0 && lane < nq) {
      // a run starts here when the key differs from the previous position's
      const bool starts = my == 0 || mk[my] != mk[my - 1];
      const uint32_t h20 = SIGN ? sign_hash0(wk, p.s_alpha, p.s_beta) : 0u;
      uint32_t step = 0, step2 = 0;
      for (uint32_t j = 0; j < p.C; ++j) {
        const uint64_t slot = static_cast<uint64_t>(p0 + my) * p.C + j;
        uint32_t key = kNoRecord;
        if (starts) {
          const uint32_t ent = chunk_entry<SIGN>(fast_mod(add_mod_p(wk, step), p.fm_c, p.M),
                                                 add_mod_p(h20, step2), p);
          if (ent != kSkip) key = ent & 0x7fffffffu;
        }
        rkey[slot] = key;
        rval[slot] = static_cast<uint32_t>(slot);
        step = add_mod_p(step, p.a);
        if (SIGN) step2 = add_mod_p(step2, p.a2);
      }
    }
  }
  lds_barrier();  // every reader holds its quarter: the sort buffers are free
  if (reader && nq > 0) {
    bool head = head_open;
    uint32_t run_start = static_cast<uint32_t>(q0);
    float acc[EPL];
#pragma unroll
    for (int r = 0; r < EPL; ++r) acc[r] = 0.f;
    float ga[U][EPL], gb[U][EPL];
    load_rows<EPL, U>(ga, grad, inv_len, p, wr, 0, nq, c0, lane, act);
#pragma unroll
    for (int k = 0; k <= kBatches; ++k) {
      if (k < kBatches) {
        const int q = k * U;
        // Rows of the next batch are requested before this one is summed
        // (unconditionally, so that the wait for this batch's rows is exact;
        // past the quarter's end they repeat its last row).
        if (k + 1 < kBatches) {
          if (k & 1) load_rows<EPL, U>(ga, grad, inv_len, p, wr, q + U, nq, c0, lane, act);
          else load_rows<EPL, U>(gb, grad, inv_len, p, wr, q + U, nq, c0, lane, act);
        }
        int nr = 0;
        float* hv = headv + pair * kRowF;
        if (q < nq)
          nr = (k & 1) ? sum_runs<EPL, U, REC>(gb, acc, wk, q, nq, after, vals[pair][k & 1],
                                               rkeys[pair][k & 1], head, hv, lane,
                                               rst[pair][k & 1], &run_start, q0)
                       : sum_runs<EPL, U, REC>(ga, acc, wk, q, nq, after, vals[pair][k & 1],
                                               rkeys[pair][k & 1], head, hv, lane,
                                               rst[pair][k & 1], &run_start, q0);
        if (lane == 0) nruns[pair][k & 1] = nr;
      } else {
        // the open run's part in this quarter (with no run ending inside,
        // the quarter lies wholly within one run: "through")
        if (tail_open) {
#pragma unroll
          for (int r = 0; r < EPL; ++r) tailv[pair * kRowF + kWave * r + lane] = acc[r];
        }
        if (lane == 0) {
          qflags[pair] = (tail_open ? 1 : 0) | (head ? 2 : 0);
          if (REC) lastst[pair] = run_start;
        }
      }
      lds_barrier();
    }
  } else if (reader) {  // an empty quarter (last piece): no runs
#pragma unroll
    for (int k = 0; k <= kBatches; ++k) {
      if (k < kBatches && lane == 0) nruns[pair][k & 1] = 0;
      if (k == kBatches && lane == 0) qflags[pair] = 0;
      lds_barrier();
    }
  } else {
    uint32_t step[EPL], step2[EPL], kk[EPL];
#pragma unroll
    for (int r = 0; r < EPL; ++r) {
      const uint32_t cc = act[r] ? c0 + lane + kWave * r : 0u;
      const uint32_t jj = cc / p.Z;
      kk[r] = cc - jj * p.Z;
      step[r] = chunk_step(p.a, jj);
      step2[r] = SIGN ? chunk_step(p.a2, jj) : 0u;
    }
#pragma unroll
    for (int k = 0; k <= kBatches; ++k) {
      if (k > 0) {
        const int b = (k - 1) & 1;
        const int nr = nruns[pair][b];
        for (int s = 0; s < nr; ++s) {
          float v[EPL];
#pragma unroll
          for (int r = 0; r < EPL; ++r) v[r] = vals[pair][b][s * kRowF + kWave * r + lane];
          if (REC)
            record_run<EPL, SIGN>(dst, scale, p, rkeys[pair][b][s],
                                  static_cast<uint64_t>(p0) + rst[pair][b][s], v, act, step,
                                  step2, kk, c0, lane);
          else
            deposit_run<EPL, SIGN>(dst, scale, p, rkeys[pair][b][s], v, act, step, step2, kk);
        }
      }
      lds_barrier();
    }
    // Runs crossing quarter boundaries: depositor `pair` takes the run that
    // leaves quarter `pair` (unless quarter `pair` lies inside a run that
    // began earlier) and adds the parts of every quarter it passes through
    // and of the quarter where it ends.
    const int fl = qflags[pair];
    if ((fl & 1) && !(fl & 2)) {
      float v[EPL];
#pragma unroll
      for (int r = 0; r < EPL; ++r) v[r] = tailv[pair * kRowF + kWave * r + lane];
      int q = pair + 1;
      while (q < kReaders - 1 && (qflags[q] & 3) == 3) {  // through quarters
#pragma unroll
        for (int r = 0; r < EPL; ++r) v[r] += tailv[q * kRowF + kWave * r + lane];
        ++q;
      }
#pragma unroll
      for (int r = 0; r < EPL; ++r) v[r] += headv[q * kRowF + kWave * r + lane];
      if (REC)
        record_run<EPL, SIGN>(dst, scale, p, qkey[q], static_cast<uint64_t>(p0) + lastst[pair], v,
                              act, step, step2, kk, c0, lane);
      else
        deposit_run<EPL, SIGN>(dst, scale, p, qkey[q], v, act, step, step2, kk);
    }
  }
}

// Sort tiles per XCD in the numbering of sort_tile_index.
static uint32_t sort_tiles_per_xcd(uint32_t nblocks) {
  return static_cast<uint32_t>((nblocks + kXcds - 1) / kXcds);
}

static uint32_t scan_chunks(uint32_t nblocks) { return (nblocks + kScanChunk - 1) / kScanChunk; }

size_t radix_scratch_bytes(int64_t n) {
  const uint64_t nblocks = (static_cast<uint64_t>(n) + kSortTile - 1) / kSortTile;
  return (nblocks * kBins + kBins + static_cast<uint64_t>(kBins) * scan_chunks(static_cast<uint32_t>(nblocks))) * 4 + 256;
}

size_t sorted_workspace_bytes(const KParams& p) {
  size_t s = static_cast<size_t>(p.N) * 16 + radix_scratch_bytes(p.N);
  if (p.mean) s += (p.num_bags * 4 + 255) & ~uint64_t(255);
  return s;
}

hipError_t radix_sort_pairs(uint32_t*& keys, uint32_t*& vals, uint32_t* ktmp, uint32_t* vtmp,
                            int64_t n, int bits, uint32_t* scratch, hipStream_t stream,
                            const uint32_t* n_dev, bool first_counted, int shift0) {
  if (n == 0) return hipSuccess;
  const uint32_t nblocks = static_cast<uint32_t>((n + kSortTile - 1) / kSortTile);
  // live keys counted on the device fill a prefix of the tiles: numbered
  // in dispatch order so that they spread over every XCD
  const uint32_t per_xcd = n_dev == nullptr ? sort_tiles_per_xcd(nblocks) : 0u;
  const dim3 grid(per_xcd ? per_xcd * static_cast<uint32_t>(kXcds) : nblocks);
  const uint32_t ngroups = (nblocks + kHistTiles - 1) / kHistTiles;
  const uint32_t hper_xcd = n_dev == nullptr ? sort_tiles_per_xcd(ngroups) : 0u;
  const dim3 hgrid(hper_xcd ? hper_xcd * static_cast<uint32_t>(kXcds) : ngroups);
  uint32_t* counts = scratch;
  uint32_t* totals = counts + static_cast<uint64_t>(nblocks) * kBins;
  for (int shift = shift0; shift < shift0 + bits; shift += kSortBits) {
    if (shift > shift0 || !first_counted)
      hipLaunchKernelGGL(sort_hist_kernel, hgrid, dim3(kBlockThreads), 0, stream, keys, n, shift,
                         counts, nblocks, hper_xcd, n_dev);
    const uint32_t nch = scan_chunks(nblocks);
    if (nch <= 2) {
      hipLaunchKernelGGL(sort_scan_kernel, dim3(kBins), dim3(kBlockThreads), 0, stream, counts,
                         nblocks, totals, n, n_dev);
    } else {
      uint32_t* partial = totals + kBins;
      hipLaunchKernelGGL(sort_scan_sums_kernel, dim3(nch, kBins), dim3(kBlockThreads), 0, stream,
                         counts, nblocks, partial, n, n_dev);
      hipLaunchKernelGGL(sort_scan_apply_kernel, dim3(nch, kBins), dim3(kBlockThreads), 0, stream,
                         counts, nblocks, partial, totals, n, n_dev);
    }
    hipLaunchKernelGGL(sort_scatter_kernel, grid, dim3(kBlockThreads), 0, stream, keys, vals,
                       ktmp, vtmp, n, shift, counts, nblocks, totals, per_xcd, n_dev);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    uint32_t* t = keys; keys = ktmp; ktmp = t;
    t = vals; vals = vtmp; vtmp = t;
  }
  return hipSuccess;
}

// Grouping only needs equal keys close together: the pairs are sorted by the
// low bits of h0 and the in-register sort of each 64-pair piece separates
// tokens that share them.  Frequent tokens already fill whole pieces after
// one 8-bit pass; more bits only pay off once a group of equal low bits
// holds many pairs, so a pass is added while the groups would average more
// than 8192 pairs (measured on the one-hot and row-hash workloads: 1.7M
// pairs -> one 8-bit pass, 6.8M -> two).  Wider digits group better per
// pass but cost more in the histogram and scatter than they save.
int grouping_bits(int64_t N) {
  int bits = kSortBits;
  while (bits < 3 * kSortBits && (N >> bits) > 8192) bits += kSortBits;
  return bits;
}

hipError_t launch_keygen(const KParams& p, const void* indices, const void* offsets,
                         uint32_t* keys, uint32_t* rows, float* inv_len, hipStream_t stream) {
  const uint64_t tiles = (p.num_bags + kTileBags - 1) / kTileBags;
  const uint64_t blocks = (tiles + kWavesPerBlock - 1) / kWavesPerBlock;
  hipLaunchKernelGGL(keygen_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(kBlockThreads), 0,
                     stream, p, indices, offsets, keys, rows, inv_len);
  return hipGetLastError();
}

// Timing hook (pss_debug_reduce_events): events recorded at the start and
// end of each reduce-and-deposit kernel, both or neither set.
static std::atomic<hipEvent_t> g_reduce_before{nullptr}, g_reduce_after{nullptr};

void set_reduce_events(hipEvent_t before, hipEvent_t after) {
  g_reduce_before.store(before);
  g_reduce_after.store(after);
}

template <int EPL, int U, bool SIGN, typename GT, bool REC>
static hipError_t launch_reduce_t(float* dst, float scale, const KParams& p, const uint32_t* keys,
                                  const uint32_t* rows, const GT* grad, const float* inv_len,
                                  uint32_t* rkey, uint32_t* rval, hipStream_t stream) {
  const uint64_t blocks = (static_cast<uint64_t>(p.N) + kPiece - 1) / kPiece;
  const uint32_t slabs = (p.d + kWave * EPL - 1) / (kWave * EPL);
  const dim3 grid(static_cast<uint32_t>(blocks), slabs);
  const hipEvent_t before = g_reduce_before.load(), after = g_reduce_after.load();
  if (before != nullptr && after != nullptr) {
    // the kernel's dispatch records both events: they bracket its execution
    // alone, not the wait for the previous kernel or the dispatch itself
    hipExtLaunchKernelGGL((reduce_deposit_kernel<EPL, U, SIGN, GT, REC>), grid,
                          dim3(kReduceThreads), 0, stream, before, after, 0u, dst, scale, p, keys,
                          rows, grad, inv_len, p.N, rkey, rval);
  } else {
    hipLaunchKernelGGL((reduce_deposit_kernel<EPL, U, SIGN, GT, REC>), grid, dim3(kReduceThreads),
                       0, stream, dst, scale, p, keys, rows, grad, inv_len, p.N, rkey, rval);
  }
  return hipGetLastError();
}

template <bool SIGN, typename GT, bool REC>
static hipError_t launch_reduce_s(float* dst, float scale, const KParams& p, const uint32_t* keys,
                                  const uint32_t* rows, const GT* grad, const float* il,
                                  uint32_t* rk, uint32_t* rv, hipStream_t stream) {
  if (p.d <= 64)
    return launch_reduce_t<1, 16, SIGN, GT, REC>(dst, scale, p, keys, rows, grad, il, rk, rv, stream);
  if (p.d <= 128)
    return launch_reduce_t<2, 8, SIGN, GT, REC>(dst, scale, p, keys, rows, grad, il, rk, rv, stream);
  if (p.d <= 256)
    return launch_reduce_t<4, 4, SIGN, GT, REC>(dst, scale, p, keys, rows, grad, il, rk, rv, stream);
  return launch_reduce_t<8, 2, SIGN, GT, REC>(dst, scale, p, keys, rows, grad, il, rk, rv, stream);
}

template <typename GT, bool REC>
static hipError_t launch_reduce_g(float* dst, float scale, const KParams& p, const uint32_t* keys,
                                  const uint32_t* rows, const GT* grad, const float* il,
                                  uint32_t* rk, uint32_t* rv, hipStream_t stream) {
  if (p.sign_mode)
    return launch_reduce_s<true, GT, REC>(dst, scale, p, keys, rows, grad, il, rk, rv, stream);
  return launch_reduce_s<false, GT, REC>(dst, scale, p, keys, rows, grad, il, rk, rv, stream);
}

// Workspace of the grouping: k0, v0, k1, v1 (N words each), the radix
// scratch (digit counts first), then inv_len (mean pooling).
KeygenOut keygen_layout(const KParams& p, void* workspace) {
  const int64_t N = p.N;
  uint32_t* k0 = static_cast<uint32_t*>(workspace);
  uint32_t* scratch = k0 + 4 * N;
  KeygenOut kg;
  kg.keys = k0;
  kg.rows = k0 + N;
  kg.inv_len = p.mean ? reinterpret_cast<float*>(reinterpret_cast<char*>(scratch) +
                                                 radix_scratch_bytes(N))
                      : nullptr;
  kg.counts = scratch;
  kg.nblocks = static_cast<uint32_t>((N + kSortTile - 1) / kSortTile);
  return kg;
}

hipError_t finish_group_sorted(const KParams& p, void* workspace, bool first_counted,
                               hipStream_t stream, GroupedPairs* out) {
  const int64_t N = p.N;
  const KeygenOut kg = keygen_layout(p, workspace);
  uint32_t* k0 = kg.keys;
  uint32_t* v0 = kg.rows;
  uint32_t* k1 = v0 + N;
  uint32_t* v1 = k1 + N;
  hipError_t e = hipSuccess;
  if (N > 0)
    e = radix_sort_pairs(k0, v0, k1, v1, N, grouping_bits(N), kg.counts, stream, nullptr,
                         first_counted);
  out->keys = k0;
  out->rows = v0;
  out->inv_len = kg.inv_len;
  return e;
}

hipError_t launch_group_sorted(const KParams& p, const void* indices, const void* offsets,
                               void* workspace, hipStream_t stream, GroupedPairs* out) {
  const int64_t N = p.N;
  const KeygenOut kg = keygen_layout(p, workspace);
  if (N == 0) return finish_group_sorted(p, workspace, false, stream, out);
  // As many items as bags (one-hot batches): keygen in item space, fused
  // with the first pass's histogram.
  const bool item_space = static_cast<uint64_t>(N) == p.num_bags;
  hipError_t e = hipSuccess;
  if (item_space) {
    const uint32_t per_xcd = sort_tiles_per_xcd(kg.nblocks);
    const dim3 grid(per_xcd * static_cast<uint32_t>(kXcds));
    if (p.idx32)
      hipLaunchKernelGGL(keygen_hist_kernel<true>, grid, dim3(kBlockThreads), 0, stream, p,
                         indices, offsets, kg.keys, kg.rows, kg.inv_len, kg.counts, kg.nblocks,
                         per_xcd);
    else
      hipLaunchKernelGGL(keygen_hist_kernel<false>, grid, dim3(kBlockThreads), 0, stream, p,
                         indices, offsets, kg.keys, kg.rows, kg.inv_len, kg.counts, kg.nblocks,
                         per_xcd);
    e = hipGetLastError();
  } else {
    e = launch_keygen(p, indices, offsets, kg.keys, kg.rows, kg.inv_len, stream);
  }
  if (e != hipSuccess) return e;
  return finish_group_sorted(p, workspace, item_space, stream, out);
}

hipError_t launch_reduce_sorted(float* dst, float scale, const KParams& p, const GroupedPairs& g,
                                const void* grad, hipStream_t stream) {
  if (p.N == 0) return hipSuccess;
  if (p.rows_bf16)
    return launch_reduce_g<uint16_t, false>(dst, scale, p, g.keys, g.rows,
                                            static_cast<const uint16_t*>(grad), g.inv_len, nullptr,
                                            nullptr, stream);
  return launch_reduce_g<float, false>(dst, scale, p, g.keys, g.rows,
                                       static_cast<const float*>(grad), g.inv_len, nullptr,
                                       nullptr, stream);
}

hipError_t launch_reduce_records(float* payload, float scale, const KParams& p,
                                 const GroupedPairs& g, const void* grad, uint32_t* rkey,
                                 uint32_t* rval, hipStream_t stream) {
  if (p.N == 0) return hipSuccess;
  if (p.rows_bf16)
    return launch_reduce_g<uint16_t, true>(payload, scale, p, g.keys, g.rows,
                                           static_cast<const uint16_t*>(grad), g.inv_len, rkey,
                                           rval, stream);
  return launch_reduce_g<float, true>(payload, scale, p, g.keys, g.rows,
                                      static_cast<const float*>(grad), g.inv_len, rkey, rval,
                                      stream);
}

hipError_t launch_deposit_sorted(float* dst, float scale, const KParams& p, const void* indices,
                                 const void* offsets, const void* grad, void* workspace,
                                 hipStream_t stream) {
  GroupedPairs g;
  const hipError_t e = launch_group_sorted(p, indices, offsets, workspace, stream, &g);
  if (e != hipSuccess) return e;
  return launch_reduce_sorted(dst, scale, p, g, grad, stream);
}

}  // namespace pss
