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
//             per pass a histogram kernel, a per-digit scan (one workgroup
//             per digit) and a scatter kernel whose per-wave ranks come from
//             ballot matching (no atomics on the data path).
//   reduce    one wavefront per 64 consecutive sorted pairs: sort them by
//             the full h0 (bitonic network over the lanes), accumulate the
//             gradient rows of each run of equal h0 in registers (lanes over
//             the dims), then add the run's sum at the run's hashed
//             addresses with float atomics.  A token spanning several
//             wavefronts deposits one partial sum per wavefront.
#include "pss_launch.hpp"

namespace pss {

constexpr int kSortBits = 8;
constexpr int kBins = 1 << kSortBits;
constexpr int kSortItemsPerLane = 8;
constexpr int kSortTile = kBlockThreads * kSortItemsPerLane;  // keys per block
constexpr int kWaveSortKeys = kWave * kSortItemsPerLane;       // keys per wave
constexpr int kDigitsPerThread = kBins / kBlockThreads;
static_assert(kBins % kBlockThreads == 0, "whole digits per thread in the scatter prologue");

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

// counts[d * nblocks + blk] = number of keys of tile blk with digit d.
__global__ __launch_bounds__(kBlockThreads) void sort_hist_kernel(
    const uint32_t* __restrict__ keys, int64_t n, const int shift,
    uint32_t* __restrict__ counts, const uint32_t nblocks, const uint32_t* __restrict__ n_dev) {
  n = live_count(n, n_dev);
  if (static_cast<int64_t>(blockIdx.x) * kSortTile >= n) {  // no live key in this tile
    for (int d = threadIdx.x; d < kBins; d += kBlockThreads)
      counts[static_cast<uint64_t>(d) * nblocks + blockIdx.x] = 0;
    return;
  }
  __shared__ uint32_t hist[kWavesPerBlock][kBins];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & (kWave - 1);
  for (int i = threadIdx.x; i < kWavesPerBlock * kBins; i += kBlockThreads) (&hist[0][0])[i] = 0;
  __syncthreads();
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kSortTile + w * kWaveSortKeys;
#pragma unroll 4
  for (int s = 0; s < kSortItemsPerLane; ++s) {
    const int64_t idx = base + s * kWave + lane;
    const bool valid = idx < n;
    const uint32_t digit = valid ? (keys[idx] >> shift) & (kBins - 1) : 0u;
    const uint64_t eq = match_digit(digit, valid);
    // the lowest lane of each group adds the group's size (wave-private row)
    if (valid && (eq & lanes_below(lane)) == 0) hist[w][digit] += __popcll(eq);
  }
  __syncthreads();
  for (int d = threadIdx.x; d < kBins; d += kBlockThreads) {
    uint32_t s = 0;
#pragma unroll
    for (int ww = 0; ww < kWavesPerBlock; ++ww) s += hist[ww][d];
    counts[static_cast<uint64_t>(d) * nblocks + blockIdx.x] = s;
  }
}

// Row d of counts (one digit, nblocks entries): exclusive scan in place;
// totals[d] = the row's sum.  One workgroup per digit.
__global__ __launch_bounds__(kBlockThreads) void sort_scan_kernel(uint32_t* __restrict__ counts,
                                                                  const uint32_t nblocks,
                                                                  uint32_t* __restrict__ totals) {
  __shared__ uint32_t wsum[kWavesPerBlock];
  uint32_t* row = counts + static_cast<uint64_t>(blockIdx.x) * nblocks;
  uint32_t carry = 0;
  for (uint32_t base = 0; base < nblocks; base += kBlockThreads) {
    const uint32_t i = base + threadIdx.x;
    const uint32_t v = i < nblocks ? row[i] : 0u;
    uint32_t tot;
    const uint32_t ex = block_exclusive_scan(v, wsum, &tot);
    if (i < nblocks) row[i] = carry + ex;
    carry += tot;
  }
  if (threadIdx.x == 0) totals[blockIdx.x] = carry;
}

// Stable scatter of one tile by digit into its global slots.
__global__ __launch_bounds__(kBlockThreads) void sort_scatter_kernel(
    const uint32_t* __restrict__ keys_in, const uint32_t* __restrict__ vals_in,
    uint32_t* __restrict__ keys_out, uint32_t* __restrict__ vals_out, int64_t n,
    const int shift, const uint32_t* __restrict__ offsets, const uint32_t nblocks,
    const uint32_t* __restrict__ totals, const uint32_t* __restrict__ n_dev) {
  n = live_count(n, n_dev);
  // tiles wholly past the live keys hold nothing (their counts are zero)
  if (static_cast<int64_t>(blockIdx.x) * kSortTile >= n) return;
  __shared__ uint32_t cur[kWavesPerBlock][kBins];
  __shared__ uint32_t wsum[kWavesPerBlock];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & (kWave - 1);
  for (int i = threadIdx.x; i < kWavesPerBlock * kBins; i += kBlockThreads) (&cur[0][0])[i] = 0;
  __syncthreads();
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kSortTile + w * kWaveSortKeys;
  uint32_t k[kSortItemsPerLane], v[kSortItemsPerLane];
#pragma unroll
  for (int s = 0; s < kSortItemsPerLane; ++s) {
    const int64_t idx = base + s * kWave + lane;
    k[s] = idx < n ? keys_in[idx] : 0u;
    v[s] = idx < n ? vals_in[idx] : 0u;
  }
  // per-wave digit counts
#pragma unroll
  for (int s = 0; s < kSortItemsPerLane; ++s) {
    const bool valid = base + s * kWave + lane < n;
    const uint32_t digit = (k[s] >> shift) & (kBins - 1);
    const uint64_t eq = match_digit(digit, valid);
    if (valid && (eq & lanes_below(lane)) == 0) cur[w][digit] += __popcll(eq);
  }
  // First slot of each digit: exclusive scan of the digit totals; thread t
  // owns digits [t*kDigitsPerThread, (t+1)*kDigitsPerThread).
  const int d0 = threadIdx.x * kDigitsPerThread;
  uint32_t tot[kDigitsPerThread];
  uint32_t mine = 0;
#pragma unroll
  for (int i = 0; i < kDigitsPerThread; ++i) {
    tot[i] = totals[d0 + i];
    mine += tot[i];
  }
  uint32_t unused;
  uint32_t digit_base = block_exclusive_scan(mine, wsum, &unused);
  __syncthreads();
  // wave start offsets: global slot of the tile + counts of earlier waves
#pragma unroll
  for (int i = 0; i < kDigitsPerThread; ++i) {
    const int d = d0 + i;
    uint32_t run = digit_base + offsets[static_cast<uint64_t>(d) * nblocks + blockIdx.x];
    digit_base += tot[i];
#pragma unroll
    for (int ww = 0; ww < kWavesPerBlock; ++ww) {
      const uint32_t c = cur[ww][d];
      cur[ww][d] = run;
      run += c;
    }
  }
  __syncthreads();
#pragma unroll
  for (int s = 0; s < kSortItemsPerLane; ++s) {
    const bool valid = base + s * kWave + lane < n;
    const uint32_t digit = (k[s] >> shift) & (kBins - 1);
    const uint64_t eq = match_digit(digit, valid);
    const uint32_t pos = cur[w][digit] + static_cast<uint32_t>(__popcll(eq & lanes_below(lane)));
    if (valid && pos < n) {  // always true when the counts agree; guards memory anyway
      keys_out[pos] = k[s];
      vals_out[pos] = v[s];
    }
    // all lanes have read cur[w][digit] above; group leaders advance it
    if (valid && (eq & lanes_below(lane)) == 0) cur[w][digit] += __popcll(eq);
  }
}

// ---------------------------------------------------------------------------
// segmented reduction + deposit
// ---------------------------------------------------------------------------
template <int EPL, int U, bool TAB, bool SIGN, typename GT>
__global__ __launch_bounds__(kBlockThreads) void reduce_deposit_kernel(
    float* __restrict__ dst, const float scale, const KParams p,
    const uint32_t* __restrict__ keys, const uint32_t* __restrict__ rows,
    const GT* __restrict__ grad, const float* __restrict__ inv_len, const int64_t n) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t p0 = (static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + (threadIdx.x >> 6)) * kWave;
  if (p0 >= n) return;
  const int cnt = n - p0 < kWave ? static_cast<int>(n - p0) : kWave;
  const uint32_t c0 = blockIdx.y * (kWave * EPL);
  __shared__ uint32_t tab_all[TAB ? kWavesPerBlock * kWave * kTabStride : 1];
  uint32_t* tab = tab_all + (TAB ? (threadIdx.x >> 6) * kWave * kTabStride : 0);

  uint32_t step[EPL], step2[EPL], kk[EPL], jj[EPL];
  bool act[EPL];
#pragma unroll
  for (int r = 0; r < EPL; ++r) {
    const uint32_t c = c0 + lane + kWave * r;
    act[r] = c < p.d;
    const uint32_t cc = act[r] ? c : 0;
    jj[r] = cc / p.Z;
    kk[r] = cc - jj[r] * p.Z;
    step[r] = TAB ? 0u : chunk_step(p.a, jj[r]);
    step2[r] = (TAB || !SIGN) ? 0u : chunk_step(p.a2, jj[r]);
  }
  uint32_t key = 0xffffffffu, row = 0;
  if (lane < cnt) {
    key = keys[p0 + lane];
    row = rows[p0 + lane];
    if (row >= p.num_bags) row = 0;  // rows come from keygen; clamp keeps reads in bounds
  }
  // Bitonic sort of the wave's 64 (key, row) pairs by the full key: the
  // global sort only orders the low bits, so tokens that share them can
  // arrive interleaved; sorted, each token of the piece forms one run.
  // Empty lanes hold key 0xffffffff (> any hash) and stay at the end.
  wave_sort_pairs(key, row, lane);
  // lane l: chunk bases of the key it holds after the sort
  if (TAB) fill_base_table<SIGN>(tab, key, p, lane);
  float acc[EPL];
#pragma unroll
  for (int r = 0; r < EPL; ++r) acc[r] = 0.f;

  for (int q = 0; q < cnt; q += U) {
    // Load phase: straight-line, U rows in flight (past-the-end positions
    // re-read the last row of the piece; inactive dims read the row start).
    float gv[U][EPL];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int uu = q + u < cnt ? q + u : cnt - 1;
      const uint32_t ru = readlane_u32(row, uu);
      const GT* grow = grad + static_cast<uint64_t>(ru) * p.d;
      const float il = p.mean ? inv_len[ru] : 1.f;
#pragma unroll
      for (int r = 0; r < EPL; ++r) {
        const float x = load_row(grow, act[r] ? c0 + lane + kWave * r : 0u);
        gv[u][r] = p.mean ? x * il : x;
      }
    }
    // Reduce phase: deposits (atomics) only after every load of the batch
    // was issued; loads and atomics share one wait counter on gfx9.
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (q + u < cnt) {
#pragma unroll
        for (int r = 0; r < EPL; ++r) acc[r] += gv[u][r];
        const uint32_t h = readlane_u32(key, q + u);
        const uint32_t hn = q + u + 1 < cnt ? readlane_u32(key, q + u + 1) : ~h;
        if (hn != h) {
          const uint32_t h20 = (!TAB && SIGN) ? sign_hash0(h, p.s_alpha, p.s_beta) : 0u;
#pragma unroll
          for (int r = 0; r < EPL; ++r) {
            if (act[r]) {
              const uint32_t ent =
                  TAB ? tab[(q + u) * kTabStride + jj[r]]
                      : chunk_entry<SIGN>(fast_mod(add_mod_p(h, step[r]), p.fm_c, p.M),
                                          add_mod_p(h20, step2[r]), p);
              const Elem el = elem_of<SIGN>(ent, kk[r], p.M);
              if (!SIGN || el.read)
                unsafeAtomicAdd(dst + el.m, SIGN ? apply_sign(scale * acc[r], el) : scale * acc[r]);
            }
            acc[r] = 0.f;
          }
        }
      }
    }
  }
}

size_t radix_scratch_bytes(int64_t n) {
  const uint64_t nblocks = (static_cast<uint64_t>(n) + kSortTile - 1) / kSortTile;
  return (nblocks * kBins + kBins) * 4 + 256;
}

size_t sorted_workspace_bytes(const KParams& p) {
  size_t s = static_cast<size_t>(p.N) * 16 + radix_scratch_bytes(p.N);
  if (p.mean) s += (p.num_bags * 4 + 255) & ~uint64_t(255);
  return s;
}

hipError_t radix_sort_pairs(uint32_t*& keys, uint32_t*& vals, uint32_t* ktmp, uint32_t* vtmp,
                            int64_t n, int bits, uint32_t* scratch, hipStream_t stream,
                            const uint32_t* n_dev) {
  if (n == 0) return hipSuccess;
  const uint32_t nblocks = static_cast<uint32_t>((n + kSortTile - 1) / kSortTile);
  uint32_t* counts = scratch;
  uint32_t* totals = counts + static_cast<uint64_t>(nblocks) * kBins;
  for (int shift = 0; shift < bits; shift += kSortBits) {
    hipLaunchKernelGGL(sort_hist_kernel, dim3(nblocks), dim3(kBlockThreads), 0, stream, keys, n,
                       shift, counts, nblocks, n_dev);
    hipLaunchKernelGGL(sort_scan_kernel, dim3(kBins), dim3(kBlockThreads), 0, stream, counts,
                       nblocks, totals);
    hipLaunchKernelGGL(sort_scatter_kernel, dim3(nblocks), dim3(kBlockThreads), 0, stream, keys,
                       vals, ktmp, vtmp, n, shift, counts, nblocks, totals, n_dev);
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

template <int EPL, int U, bool TAB, bool SIGN, typename GT>
static hipError_t launch_reduce_t(float* dst, float scale, const KParams& p, const uint32_t* keys,
                                  const uint32_t* rows, const GT* grad, const float* inv_len,
                                  hipStream_t stream) {
  const uint64_t waves = (static_cast<uint64_t>(p.N) + kWave - 1) / kWave;
  const uint64_t blocks = (waves + kWavesPerBlock - 1) / kWavesPerBlock;
  const uint32_t slabs = (p.d + kWave * EPL - 1) / (kWave * EPL);
  hipLaunchKernelGGL((reduce_deposit_kernel<EPL, U, TAB, SIGN, GT>),
                     dim3(static_cast<uint32_t>(blocks), slabs), dim3(kBlockThreads), 0, stream, dst,
                     scale, p, keys, rows, grad, inv_len, p.N);
  return hipGetLastError();
}

template <bool TAB, bool SIGN, typename GT>
static hipError_t launch_reduce_c(float* dst, float scale, const KParams& p, const uint32_t* keys,
                                  const uint32_t* rows, const GT* grad, const float* il,
                                  hipStream_t stream) {
  if (p.d <= 64) return launch_reduce_t<1, 16, TAB, SIGN>(dst, scale, p, keys, rows, grad, il, stream);
  if (p.d <= 128) return launch_reduce_t<2, 8, TAB, SIGN>(dst, scale, p, keys, rows, grad, il, stream);
  if (p.d <= 256) return launch_reduce_t<4, 4, TAB, SIGN>(dst, scale, p, keys, rows, grad, il, stream);
  return launch_reduce_t<8, 2, TAB, SIGN>(dst, scale, p, keys, rows, grad, il, stream);
}

template <bool SIGN, typename GT>
static hipError_t launch_reduce_s(float* dst, float scale, const KParams& p, const uint32_t* keys,
                                  const uint32_t* rows, const GT* grad, const float* il,
                                  hipStream_t stream) {
  if (p.C <= static_cast<uint32_t>(kTabChunks))
    return launch_reduce_c<true, SIGN>(dst, scale, p, keys, rows, grad, il, stream);
  return launch_reduce_c<false, SIGN>(dst, scale, p, keys, rows, grad, il, stream);
}

template <typename GT>
static hipError_t launch_reduce_g(float* dst, float scale, const KParams& p, const uint32_t* keys,
                                  const uint32_t* rows, const GT* grad, const float* il,
                                  hipStream_t stream) {
  if (p.sign_mode) return launch_reduce_s<true>(dst, scale, p, keys, rows, grad, il, stream);
  return launch_reduce_s<false>(dst, scale, p, keys, rows, grad, il, stream);
}

hipError_t launch_deposit_sorted(float* dst, float scale, const KParams& p, const void* indices,
                                 const void* offsets, const void* grad, void* workspace,
                                 hipStream_t stream) {
  const int64_t N = p.N;
  if (N == 0) return hipSuccess;
  uint32_t* k0 = static_cast<uint32_t*>(workspace);
  uint32_t* v0 = k0 + N;
  uint32_t* k1 = v0 + N;
  uint32_t* v1 = k1 + N;
  uint32_t* scratch = v1 + N;
  float* inv_len = p.mean ? reinterpret_cast<float*>(
                                reinterpret_cast<char*>(scratch) + radix_scratch_bytes(N))
                          : nullptr;
  hipError_t e = launch_keygen(p, indices, offsets, k0, v0, inv_len, stream);
  if (e == hipSuccess) e = radix_sort_pairs(k0, v0, k1, v1, N, grouping_bits(N), scratch, stream);
  if (e != hipSuccess) return e;
  if (p.rows_bf16)
    return launch_reduce_g(dst, scale, p, k0, v0, static_cast<const uint16_t*>(grad), inv_len,
                           stream);
  return launch_reduce_g(dst, scale, p, k0, v0, static_cast<const float*>(grad), inv_len, stream);
}

}  // namespace pss
