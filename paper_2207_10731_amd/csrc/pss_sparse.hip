// Sparse gradient of the shared array (Alg. 1, sparse branch): the sorted
// unique locations that any lookup reads and the summed output gradient at
// each of them.  Cost follows the number of distinct tokens in the batch,
// not M.  Every sum is taken in a fixed order, so the result is bit-identical
// from run to run.
//
//   group      keygen + radix sort on the item hash (as the sorted deposit);
//              piece_runs sorts each 64-pair piece by the full hash in
//              registers and counts its runs (one run = one token of the
//              piece); a scan turns the counts into run slots.
//   run sums   run_sums writes the summed gradient row of every run (d
//              floats) and its hash.
//   chunks     one record (chunk base, run*C + j) per run and chunk, sorted
//              by base (bases < M; unused records hold a sentinel base that
//              sorts last).  With a chunk sign, bit 31 of the record id marks
//              a -1 chunk and chunks of factor 0 get the sentinel base (they
//              read nothing, so they own and add nothing).
//   merge      element m is owned by the last chunk, in base order, whose
//              span [base, base + Z) covers it.  A chunk that runs past M
//              wraps to 0: it is also entered, shifted by -M, in front of
//              the list ("extended order").  own[x] = elements chunk x owns;
//              a scan gives every owned element its output slot, so the
//              locations come out ascending.  The value at m is the sum, over
//              the chunks covering m, walked from the owner backwards, of the
//              run-sum entry for m.
#include "pss_launch.hpp"

namespace pss {

constexpr int kScanTile = kBlockThreads * 16;

// ---------------------------------------------------------------------------
// device-wide exclusive scan of uint32 (three phases)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlockThreads) void scan_reduce_kernel(const uint32_t* __restrict__ in,
                                                                    const int64_t n,
                                                                    uint32_t* __restrict__ sums) {
  __shared__ uint32_t wsum[kWavesPerBlock];
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kScanTile + threadIdx.x * 16;
  uint32_t s = 0;
#pragma unroll
  for (int i = 0; i < 16; ++i) s += base + i < n ? in[base + i] : 0u;
  uint32_t tot;
  block_exclusive_scan(s, wsum, &tot);
  if (threadIdx.x == 0) sums[blockIdx.x] = tot;
}

__global__ __launch_bounds__(kBlockThreads) void scan_sums_kernel(uint32_t* __restrict__ sums,
                                                                  const uint32_t nsums,
                                                                  uint32_t* __restrict__ total) {
  __shared__ uint32_t wsum[kWavesPerBlock];
  uint32_t carry = 0;
  for (uint32_t base = 0; base < nsums; base += kBlockThreads) {
    const uint32_t i = base + threadIdx.x;
    const uint32_t v = i < nsums ? sums[i] : 0u;
    uint32_t tot;
    const uint32_t ex = block_exclusive_scan(v, wsum, &tot);
    if (i < nsums) sums[i] = carry + ex;
    carry += tot;
  }
  if (threadIdx.x == 0) *total = carry;
}

__global__ __launch_bounds__(kBlockThreads) void scan_apply_kernel(uint32_t* __restrict__ data,
                                                                   const int64_t n,
                                                                   const uint32_t* __restrict__ sums) {
  __shared__ uint32_t wsum[kWavesPerBlock];
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kScanTile + threadIdx.x * 16;
  uint32_t v[16];
  uint32_t s = 0;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    v[i] = base + i < n ? data[base + i] : 0u;
    s += v[i];
  }
  uint32_t tot;
  uint32_t run = sums[blockIdx.x] + block_exclusive_scan(s, wsum, &tot);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    if (base + i < n) data[base + i] = run;
    run += v[i];
  }
}

static size_t scan_scratch_bytes(int64_t n) {
  return ((static_cast<uint64_t>(n) + kScanTile - 1) / kScanTile + 1) * 4;
}

// data[0..n) <- exclusive prefix sums; *total <- sum.  n >= 1.
static hipError_t exclusive_scan(uint32_t* data, int64_t n, uint32_t* sums, uint32_t* total,
                                 hipStream_t stream) {
  const uint32_t nsums = static_cast<uint32_t>((n + kScanTile - 1) / kScanTile);
  hipLaunchKernelGGL(scan_reduce_kernel, dim3(nsums), dim3(kBlockThreads), 0, stream, data, n, sums);
  hipLaunchKernelGGL(scan_sums_kernel, dim3(1), dim3(kBlockThreads), 0, stream, sums, nsums, total);
  hipLaunchKernelGGL(scan_apply_kernel, dim3(nsums), dim3(kBlockThreads), 0, stream, data, n, sums);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// runs of each 64-pair piece
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint64_t lanes_upto(int lane) {  // lanes 0 .. lane
  return lane == kWave - 1 ? ~0ull : ((1ull << (lane + 1)) - 1);
}

__global__ __launch_bounds__(kBlockThreads) void piece_runs_kernel(uint32_t* __restrict__ keys,
                                                                   uint32_t* __restrict__ rows,
                                                                   const int64_t n,
                                                                   uint32_t* __restrict__ counts) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t piece = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + (threadIdx.x >> 6);
  const int64_t p0 = piece * kWave;
  if (p0 >= n) return;
  const int cnt = n - p0 < kWave ? static_cast<int>(n - p0) : kWave;
  uint32_t key = 0xffffffffu, row = 0;
  if (lane < cnt) {
    key = keys[p0 + lane];
    row = rows[p0 + lane];
  }
  wave_sort_pairs(key, row, lane);
  if (lane < cnt) {
    keys[p0 + lane] = key;
    rows[p0 + lane] = row;
  }
  const uint32_t prev = __shfl_up(key, 1);
  const uint64_t starts = __ballot(lane < cnt && (lane == 0 || prev != key));
  if (lane == 0) counts[piece] = static_cast<uint32_t>(__popcll(starts));
}

// Summed gradient row of every run; run slots from the scanned counts.
template <int EPL, int U, typename GT>
__global__ __launch_bounds__(kBlockThreads) void run_sums_kernel(
    const KParams p, const uint32_t* __restrict__ keys, const uint32_t* __restrict__ rows,
    const int64_t n, const uint32_t* __restrict__ run_off, const GT* __restrict__ grad,
    const float* __restrict__ inv_len, float* __restrict__ rs, uint32_t* __restrict__ rk) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t piece = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + (threadIdx.x >> 6);
  const int64_t p0 = piece * kWave;
  if (p0 >= n) return;
  const int cnt = n - p0 < kWave ? static_cast<int>(n - p0) : kWave;
  const uint32_t c0 = blockIdx.y * (kWave * EPL);
  bool act[EPL];
#pragma unroll
  for (int r = 0; r < EPL; ++r) act[r] = c0 + lane + kWave * r < p.d;
  uint32_t key = 0xffffffffu, row = 0;
  if (lane < cnt) {
    key = keys[p0 + lane];
    row = rows[p0 + lane];
    if (row >= p.num_bags) row = 0;
  }
  uint64_t slot = run_off[piece];
  float acc[EPL];
#pragma unroll
  for (int r = 0; r < EPL; ++r) acc[r] = 0.f;
  for (int q = 0; q < cnt; q += U) {
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
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (q + u < cnt) {
#pragma unroll
        for (int r = 0; r < EPL; ++r) acc[r] += gv[u][r];
        const uint32_t h = readlane_u32(key, q + u);
        const uint32_t hn = q + u + 1 < cnt ? readlane_u32(key, q + u + 1) : ~h;
        if (hn != h) {
          float* dstrow = rs + slot * p.d + c0 + lane;
#pragma unroll
          for (int r = 0; r < EPL; ++r) {
            if (act[r]) dstrow[kWave * r] = acc[r];
            acc[r] = 0.f;
          }
          if (blockIdx.y == 0 && lane == 0) rk[slot] = h;
          ++slot;
        }
      }
    }
  }
}

// One (chunk base, run*C + j) record per run and chunk; records past the
// last run hold the sentinel base 0xffffffff.
__global__ __launch_bounds__(kBlockThreads) void chunk_records_kernel(
    const KParams p, const uint32_t* __restrict__ rk, const uint32_t* __restrict__ num_runs,
    const int64_t cap, uint32_t* __restrict__ cb, uint32_t* __restrict__ cv) {
  const int64_t x = static_cast<int64_t>(blockIdx.x) * kBlockThreads + threadIdx.x;
  if (x >= cap) return;
  const int64_t rc = static_cast<int64_t>(*num_runs) * p.C;
  uint32_t b = 0xffffffffu, id = static_cast<uint32_t>(x);
  if (x < rc) {
    const uint32_t r = static_cast<uint32_t>(x / p.C);
    const uint32_t j = static_cast<uint32_t>(x - static_cast<int64_t>(r) * p.C);
    b = fast_mod(add_mod_p(rk[r], chunk_step(p.a, j)), p.fm_c, p.M);
    if (p.sign_mode) {
      const uint32_t h2 = add_mod_p(sign_hash0(rk[r], p.s_alpha, p.s_beta), chunk_step(p.a2, j));
      const uint32_t code = sign_code(h2, p.sign_mode);
      if (code == 2u) b = 0xffffffffu;
      id |= code << 31;  // code 1: negative (code 2 records are never read)
    }
  }
  cb[x] = b;
  cv[x] = id;
}

// info[0] = number of chunk records RC that read something (the sorted
// records before the first sentinel), info[1] = records whose span wraps
// (base > M - Z; a suffix of those RC).
__global__ void tail_count_kernel(const KParams p, const uint32_t* __restrict__ cb,
                                  const uint32_t* __restrict__ num_runs, uint32_t* __restrict__ info) {
  uint64_t rc = static_cast<uint64_t>(*num_runs) * p.C;
  {  // first sorted position holding the sentinel
    uint64_t lo = 0, hi = rc;
    while (lo < hi) {
      const uint64_t mid = (lo + hi) / 2;
      if (cb[mid] == 0xffffffffu) hi = mid; else lo = mid + 1;
    }
    rc = lo;
  }
  // first sorted position with base > M - Z
  uint64_t lo = 0, hi = rc;
  const uint32_t lim = p.M - p.Z;
  while (lo < hi) {
    const uint64_t mid = (lo + hi) / 2;
    if (cb[mid] > lim) hi = mid; else lo = mid + 1;
  }
  info[0] = static_cast<uint32_t>(rc);
  info[1] = static_cast<uint32_t>(rc - lo);
}

struct ExtList {  // the extended order: wrapped copies first, then all records
  const uint32_t* cb;
  uint32_t rc, tail, M;
  __device__ __forceinline__ uint32_t len() const { return rc + tail; }
  __device__ __forceinline__ uint32_t sorted_index(uint32_t x) const {
    return x < tail ? rc - tail + x : x - tail;
  }
  __device__ __forceinline__ int64_t base(uint32_t x) const {
    const int64_t b = cb[sorted_index(x)];
    return x < tail ? b - static_cast<int64_t>(M) : b;
  }
};

__global__ __launch_bounds__(kBlockThreads) void own_kernel(const KParams p,
                                                            const uint32_t* __restrict__ cb,
                                                            const uint32_t* __restrict__ info,
                                                            const int64_t cap2,
                                                            uint32_t* __restrict__ own) {
  const int64_t x = static_cast<int64_t>(blockIdx.x) * kBlockThreads + threadIdx.x;
  if (x >= cap2) return;
  ExtList e{cb, info[0], info[1], p.M};
  uint32_t o = 0;
  if (x < e.len()) {
    const int64_t b = e.base(static_cast<uint32_t>(x));
    const int64_t bn = x + 1 < e.len() ? e.base(static_cast<uint32_t>(x + 1)) : INT64_MAX;
    if (bn != b) {  // last record of its base owns the elements
      const int64_t lo = b < 0 ? 0 : b;
      int64_t hi = b + p.Z;
      if (bn < hi) hi = bn;
      if (hi > static_cast<int64_t>(p.M)) hi = p.M;
      o = hi > lo ? static_cast<uint32_t>(hi - lo) : 0u;
    }
  }
  own[x] = o;
}

__global__ __launch_bounds__(kBlockThreads) void emit_kernel(
    const KParams p, const uint32_t* __restrict__ cb, const uint32_t* __restrict__ cv,
    const uint32_t* __restrict__ info, const uint32_t* __restrict__ slot,
    const float* __restrict__ rs, const int64_t cap2, const int64_t capacity,
    uint32_t* __restrict__ locations, float* __restrict__ values) {
  const int64_t x = static_cast<int64_t>(blockIdx.x) * kBlockThreads + threadIdx.x;
  if (x >= cap2) return;
  ExtList e{cb, info[0], info[1], p.M};
  if (x >= e.len()) return;
  const int64_t b = e.base(static_cast<uint32_t>(x));
  const int64_t bn = x + 1 < e.len() ? e.base(static_cast<uint32_t>(x + 1)) : INT64_MAX;
  if (bn == b) return;
  const int64_t lo = b < 0 ? 0 : b;
  int64_t hi = b + p.Z;
  if (bn < hi) hi = bn;
  if (hi > static_cast<int64_t>(p.M)) hi = p.M;
  uint64_t out = slot[x];
  for (int64_t m = lo; m < hi; ++m, ++out) {
    float v = 0.f;
    // every record covering m sits at or before x in the extended order
    for (int64_t y = x; y >= 0; --y) {
      const int64_t by = e.base(static_cast<uint32_t>(y));
      if (by + p.Z <= m) break;
      const uint32_t rec = cv[e.sorted_index(static_cast<uint32_t>(y))];
      const uint32_t id = rec & 0x7fffffffu;
      const uint32_t run = id / p.C, j = id - run * p.C;
      const float x = rs[static_cast<uint64_t>(run) * p.d + j * p.Z + static_cast<uint32_t>(m - by)];
      v += (rec >> 31) ? -x : x;
    }
    if (static_cast<int64_t>(out) < capacity) {
      locations[out] = static_cast<uint32_t>(m);
      values[out] = v;
    }
  }
}

__global__ void store_count_kernel(const uint32_t* __restrict__ total, int64_t* __restrict__ out) {
  *out = *total;
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------

// Records have 31-bit ids (bit 31 carries the sign): N*C must stay below 2^31.
static int64_t record_cap(const KParams& p) { return p.N * static_cast<int64_t>(p.C); }

static int base_bits(uint32_t M) {  // smallest multiple of 8 with 2^bits > M
  int bits = 8;
  while (bits < 32 && (1ull << bits) <= M) bits += 8;
  return bits;
}

size_t sparse_workspace_bytes(const KParams& p) {
  const int64_t N = p.N, cap = record_cap(p), cap2 = 2 * cap;
  const int64_t npieces = (N + kWave - 1) / kWave;
  size_t s = 0;
  s += static_cast<size_t>(N) * 16 + radix_scratch_bytes(N);  // grouping
  s += static_cast<size_t>(npieces) * 4 + scan_scratch_bytes(npieces) + 16;  // run slots
  s += static_cast<size_t>(N) * p.d * 4 + static_cast<size_t>(N) * 4;  // run sums + keys
  s += static_cast<size_t>(cap) * 16 + radix_scratch_bytes(cap);  // chunk records
  s += static_cast<size_t>(cap2) * 4 + scan_scratch_bytes(cap2) + 16;  // ownership
  if (p.mean) s += static_cast<size_t>(p.num_bags) * 4;  // 1 / |bag| per pooled row
  return s + 64 * 16;  // alignment slack
}

template <typename T>
static T* carve(char*& cur, size_t count) {
  T* p = reinterpret_cast<T*>(cur);
  cur += (count * sizeof(T) + 255) & ~size_t(255);
  return p;
}

template <int EPL, int U, typename GT>
static void launch_run_sums_t(const KParams& p, const uint32_t* keys, const uint32_t* rows,
                              const uint32_t* run_off, const GT* grad, const float* inv_len,
                              float* rs, uint32_t* rk, hipStream_t stream) {
  const uint64_t waves = (static_cast<uint64_t>(p.N) + kWave - 1) / kWave;
  const uint64_t blocks = (waves + kWavesPerBlock - 1) / kWavesPerBlock;
  const uint32_t slabs = (p.d + kWave * EPL - 1) / (kWave * EPL);
  hipLaunchKernelGGL((run_sums_kernel<EPL, U, GT>), dim3(static_cast<uint32_t>(blocks), slabs),
                     dim3(kBlockThreads), 0, stream, p, keys, rows, p.N, run_off, grad, inv_len,
                     rs, rk);
}

template <typename GT>
static void launch_run_sums(const KParams& p, const uint32_t* keys, const uint32_t* rows,
                            const uint32_t* run_off, const GT* grad, const float* inv_len,
                            float* rs, uint32_t* rk, hipStream_t stream) {
  if (p.d <= 64) launch_run_sums_t<1, 16>(p, keys, rows, run_off, grad, inv_len, rs, rk, stream);
  else if (p.d <= 128) launch_run_sums_t<2, 8>(p, keys, rows, run_off, grad, inv_len, rs, rk, stream);
  else if (p.d <= 256) launch_run_sums_t<4, 4>(p, keys, rows, run_off, grad, inv_len, rs, rk, stream);
  else launch_run_sums_t<8, 2>(p, keys, rows, run_off, grad, inv_len, rs, rk, stream);
}

static uint32_t blocks_for(int64_t n) {
  return static_cast<uint32_t>((n + kBlockThreads - 1) / kBlockThreads);
}

hipError_t launch_gradient_sparse(const KParams& p, const void* indices, const void* offsets,
                                  const void* grad, void* workspace, uint32_t* locations,
                                  float* values, int64_t capacity, uint32_t* num_unique32,
                                  hipStream_t stream) {
  const int64_t N = p.N, cap = record_cap(p), cap2 = 2 * cap;
  const int64_t npieces = (N + kWave - 1) / kWave;
  char* cur = static_cast<char*>(workspace);
  uint32_t* k0 = carve<uint32_t>(cur, N);
  uint32_t* v0 = carve<uint32_t>(cur, N);
  uint32_t* k1 = carve<uint32_t>(cur, N);
  uint32_t* v1 = carve<uint32_t>(cur, N);
  uint32_t* rscr = carve<uint32_t>(cur, radix_scratch_bytes(N) / 4 + 1);
  uint32_t* runs = carve<uint32_t>(cur, npieces);
  uint32_t* sscr = carve<uint32_t>(cur, scan_scratch_bytes(npieces) / 4 + 1);
  uint32_t* num_runs = carve<uint32_t>(cur, 4);
  float* rs = carve<float>(cur, static_cast<size_t>(N) * p.d);
  uint32_t* rk = carve<uint32_t>(cur, N);
  uint32_t* cb = carve<uint32_t>(cur, cap);
  uint32_t* cv = carve<uint32_t>(cur, cap);
  uint32_t* cb1 = carve<uint32_t>(cur, cap);
  uint32_t* cv1 = carve<uint32_t>(cur, cap);
  uint32_t* cscr = carve<uint32_t>(cur, radix_scratch_bytes(cap) / 4 + 1);
  uint32_t* own = carve<uint32_t>(cur, cap2);
  uint32_t* oscr = carve<uint32_t>(cur, scan_scratch_bytes(cap2) / 4 + 1);
  uint32_t* info = carve<uint32_t>(cur, 4);
  float* inv_len = p.mean ? carve<float>(cur, p.num_bags) : nullptr;

  hipError_t e = launch_keygen(p, indices, offsets, k0, v0, inv_len, stream);
  if (e == hipSuccess) e = radix_sort_pairs(k0, v0, k1, v1, N, grouping_bits(N), rscr, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(piece_runs_kernel, dim3(static_cast<uint32_t>((npieces + kWavesPerBlock - 1) / kWavesPerBlock)),
                     dim3(kBlockThreads), 0, stream, k0, v0, N, runs);
  e = exclusive_scan(runs, npieces, sscr, num_runs, stream);
  if (e != hipSuccess) return e;
  if (p.rows_bf16)
    launch_run_sums(p, k0, v0, runs, static_cast<const uint16_t*>(grad), inv_len, rs, rk, stream);
  else
    launch_run_sums(p, k0, v0, runs, static_cast<const float*>(grad), inv_len, rs, rk, stream);
  hipLaunchKernelGGL(chunk_records_kernel, dim3(blocks_for(cap)), dim3(kBlockThreads), 0, stream, p,
                     rk, num_runs, cap, cb, cv);
  e = hipGetLastError();
  if (e == hipSuccess) e = radix_sort_pairs(cb, cv, cb1, cv1, cap, base_bits(p.M), cscr, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(tail_count_kernel, dim3(1), dim3(1), 0, stream, p, cb, num_runs, info);
  hipLaunchKernelGGL(own_kernel, dim3(blocks_for(cap2)), dim3(kBlockThreads), 0, stream, p, cb, info,
                     cap2, own);
  e = exclusive_scan(own, cap2, oscr, num_unique32, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(emit_kernel, dim3(blocks_for(cap2)), dim3(kBlockThreads), 0, stream, p, cb, cv,
                     info, own, rs, cap2, capacity, locations, values);
  return hipGetLastError();
}

hipError_t launch_store_count(const uint32_t* total, int64_t* out, hipStream_t stream) {
  hipLaunchKernelGGL(store_count_kernel, dim3(1), dim3(1), 0, stream, total, out);
  return hipGetLastError();
}

// Optimizer on the unique locations only (no two entries share a location).
template <typename WT, bool ADAGRAD>
__global__ __launch_bounds__(kBlockThreads) void sparse_optimizer_kernel(
    WT* __restrict__ w, float* __restrict__ s, const uint32_t* __restrict__ loc,
    const float* __restrict__ val, const uint32_t* __restrict__ count, const int64_t capacity,
    const float lr, const float eps) {
  const int64_t n = *count < capacity ? static_cast<int64_t>(*count) : capacity;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlockThreads;
  for (int64_t k = static_cast<int64_t>(blockIdx.x) * kBlockThreads + threadIdx.x; k < n; k += stride) {
    const uint32_t m = loc[k];
    const float g = val[k];
    if (g == 0.f) continue;
    float upd;
    if (ADAGRAD) {
      const float sn = s[m] + g * g;
      s[m] = sn;
      upd = lr * g / (sqrtf(sn) + eps);
    } else {
      upd = lr * g;
    }
    if constexpr (sizeof(WT) == 4) {
      w[m] = w[m] - upd;
    } else {
      w[m] = f32_to_bf16_rne(bf16_to_f32(w[m]) - upd);
    }
  }
}

hipError_t launch_sparse_optimizer(void* w, bool bf16, float* state, const uint32_t* loc,
                                   const float* val, const uint32_t* count, int64_t capacity,
                                   float lr, float eps, hipStream_t stream) {
  const int64_t want = (capacity + kBlockThreads * 4 - 1) / (kBlockThreads * 4);
  const dim3 grid(static_cast<uint32_t>(want < 1 ? 1 : (want > 8192 ? 8192 : want)));
  if (bf16) {
    uint16_t* wb = static_cast<uint16_t*>(w);
    if (state)
      hipLaunchKernelGGL((sparse_optimizer_kernel<uint16_t, true>), grid, dim3(kBlockThreads), 0, stream,
                         wb, state, loc, val, count, capacity, lr, eps);
    else
      hipLaunchKernelGGL((sparse_optimizer_kernel<uint16_t, false>), grid, dim3(kBlockThreads), 0, stream,
                         wb, state, loc, val, count, capacity, lr, eps);
  } else {
    float* wf = static_cast<float*>(w);
    if (state)
      hipLaunchKernelGGL((sparse_optimizer_kernel<float, true>), grid, dim3(kBlockThreads), 0, stream, wf,
                         state, loc, val, count, capacity, lr, eps);
    else
      hipLaunchKernelGGL((sparse_optimizer_kernel<float, false>), grid, dim3(kBlockThreads), 0, stream, wf,
                         state, loc, val, count, capacity, lr, eps);
  }
  return hipGetLastError();
}

}  // namespace pss
