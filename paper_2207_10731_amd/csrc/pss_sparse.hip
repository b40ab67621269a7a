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
//   pre-merge  when the records average 16 or more per base of the array
//              (N * C >= 16 * M), the records that share a base are summed
//              once (their signed run-sum pieces, in record order) into one
//              record per distinct base, so that an element's walk below
//              meets at most Z records
//   merge      element m is owned by the last chunk, in base order, whose
//              span [base, base + Z) covers it.  A chunk that runs past M
//              wraps to 0: it is also entered, shifted by -M, in front of
//              the list ("extended order").  own[x] = elements chunk x owns;
//              a scan gives every owned element its output slot, so the
//              locations come out ascending.  The value at m is the sum, over
//              the chunks covering m, walked from the owner backwards, of the
//              run-sum entry for m (element-parallel, see emit_kernel).  The
//              backward's SPARSE variant applies the optimizer there instead
//              of writing the list.
#include "pss_launch.hpp"

namespace pss {

constexpr int kScanTile = kBlockThreads * 16;

// ---------------------------------------------------------------------------
// device-wide exclusive scan of uint32 (three phases)
// ---------------------------------------------------------------------------
// Live length: n, or min(n, *n_dev) when the real length is on the device.
__device__ __forceinline__ int64_t live_len(int64_t n, const uint32_t* n_dev) {
  if (n_dev == nullptr) return n;
  const int64_t d = *n_dev;
  return d < n ? d : n;
}

__global__ __launch_bounds__(kBlockThreads) void scan_reduce_kernel(const uint32_t* __restrict__ in,
                                                                    int64_t n,
                                                                    uint32_t* __restrict__ sums,
                                                                    const uint32_t* __restrict__ n_dev) {
  n = live_len(n, n_dev);
  if (static_cast<int64_t>(blockIdx.x) * kScanTile >= n) {
    if (threadIdx.x == 0) sums[blockIdx.x] = 0;
    return;
  }
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
                                                                   int64_t n,
                                                                   const uint32_t* __restrict__ sums,
                                                                   const uint32_t* __restrict__ n_dev) {
  n = live_len(n, n_dev);
  if (static_cast<int64_t>(blockIdx.x) * kScanTile >= n) return;
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

// data[0..n') <- exclusive prefix sums; *total <- sum, with n' = n, or
// min(n, *n_dev) when given (entries past n' are left as they are).  n >= 1.
static hipError_t exclusive_scan(uint32_t* data, int64_t n, uint32_t* sums, uint32_t* total,
                                 hipStream_t stream, const uint32_t* n_dev = nullptr) {
  const uint32_t nsums = static_cast<uint32_t>((n + kScanTile - 1) / kScanTile);
  hipLaunchKernelGGL(scan_reduce_kernel, dim3(nsums), dim3(kBlockThreads), 0, stream, data, n, sums,
                     n_dev);
  hipLaunchKernelGGL(scan_sums_kernel, dim3(1), dim3(kBlockThreads), 0, stream, sums, nsums, total);
  hipLaunchKernelGGL(scan_apply_kernel, dim3(nsums), dim3(kBlockThreads), 0, stream, data, n, sums,
                     n_dev);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// runs of each 64-pair piece
// ---------------------------------------------------------------------------
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
// info[2] <- number of records (runs * C).  Grid-stride over the records
// that exist (the launch is sized for the bound N * C).
__global__ __launch_bounds__(kBlockThreads) void chunk_records_kernel(
    const KParams p, const uint32_t* __restrict__ rk, const uint32_t* __restrict__ num_runs,
    const int64_t cap, uint32_t* __restrict__ cb, uint32_t* __restrict__ cv,
    uint32_t* __restrict__ info) {
  const int64_t rc = static_cast<int64_t>(*num_runs) * p.C;
  if (blockIdx.x == 0 && threadIdx.x == 0) info[2] = static_cast<uint32_t>(rc);
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlockThreads;
  for (int64_t x = static_cast<int64_t>(blockIdx.x) * kBlockThreads + threadIdx.x; x < rc;
       x += stride) {
    uint32_t id = static_cast<uint32_t>(x);
    const uint32_t r = static_cast<uint32_t>(x / p.C);
    const uint32_t j = static_cast<uint32_t>(x - static_cast<int64_t>(r) * p.C);
    uint32_t b = fast_mod(add_mod_p(rk[r], chunk_step(p.a, j)), p.fm_c, p.M);
    if (p.sign_mode) {
      const uint32_t h2 = add_mod_p(sign_hash0(rk[r], p.s_alpha, p.s_beta), chunk_step(p.a2, j));
      const uint32_t code = sign_code(h2, p.sign_mode);
      if (code == 2u) b = 0xffffffffu;
      id |= code << 31;  // code 1: negative (code 2 records are never read)
    }
    cb[x] = b;
    cv[x] = id;
  }
}

// info[0] = number of chunk records RC that read something (the sorted
// records before the first sentinel), info[1] = records whose span wraps
// (base > M - Z; a suffix of those RC), info[3] = RC + info[1].
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
  info[3] = static_cast<uint32_t>(rc + (rc - lo));  // length of the extended order
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
                                                            uint32_t* __restrict__ own) {
  ExtList e{cb, info[0], info[1], p.M};
  const int64_t len = e.len();
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlockThreads;
  for (int64_t x = static_cast<int64_t>(blockIdx.x) * kBlockThreads + threadIdx.x; x < len;
       x += stride) {
    uint32_t o = 0;
    const int64_t b = e.base(static_cast<uint32_t>(x));
    const int64_t bn = x + 1 < len ? e.base(static_cast<uint32_t>(x + 1)) : INT64_MAX;
    if (bn != b) {  // last record of its base owns the elements
      const int64_t lo = b < 0 ? 0 : b;
      int64_t hi = b + p.Z;
      if (bn < hi) hi = bn;
      if (hi > static_cast<int64_t>(p.M)) hi = p.M;
      o = hi > lo ? static_cast<uint32_t>(hi - lo) : 0u;
    }
    own[x] = o;
  }
}

// Emit, element-parallel with balanced work.  A wavefront takes 64
// consecutive records of the extended order; lane l holds record x = x0 + l,
// the number of elements it owns o(x) (from the scanned ownership) and their
// first output slot.  The wave expands its owned elements 64 at a time: the
// lane for element e finds its record by a search over the lanes' prefix
// sums, then sums, from the owner backwards, the run-sum entries of every
// record covering its element (records are in base order, so the covering
// ones are contiguous and end at the owner).  Sums run in a fixed order.
// MODE 0 writes (location, value) at the element's output slot; MODE 1
// applies SGD / Adagrad to the element in place (each element is owned once).
struct EmitList {
  uint32_t* locations;
  float* values;
  int64_t capacity;
};
template <typename WT>
struct EmitUpdate {
  WT* w;
  float* s;
  float lr, eps;
};

template <typename WT, bool ADAGRAD>
__device__ __forceinline__ void update_element(const EmitUpdate<WT>& u, uint32_t m, float g) {
  if (g == 0.f) return;  // untouched in value: keep the exact bits
  float upd;
  if (ADAGRAD) {
    const float sn = u.s[m] + g * g;
    u.s[m] = sn;
    upd = u.lr * g / (sqrtf(sn) + u.eps);
  } else {
    upd = u.lr * g;
  }
  if constexpr (sizeof(WT) == 4) {
    u.w[m] = u.w[m] - upd;
  } else {
    u.w[m] = f32_to_bf16_rne(bf16_to_f32(u.w[m]) - upd);
  }
}

constexpr int kWalk = 4;     // covering records summed per round of a walk
constexpr int kStage = 384;  // records a wavefront stages in LDS

// Sum, for element m, of the run-sum entries of the records covering it,
// walking from record `y0` backwards in walk order.  Rec(y) gives
// (base, id | sign) of record y; the walk stops at the first record whose
// span ends at or before m, or below record `ylo`.
template <typename Rec>
__device__ __forceinline__ float walk_sum(const KParams& p, const float* __restrict__ rs,
                                          const uint32_t rsC, const uint32_t rsD, int64_t m,
                                          int64_t y0, int64_t ylo, Rec rec_of) {
  const int64_t Z = p.Z;
  float v = 0.f;
  for (int64_t y = y0; y >= ylo; y -= kWalk) {
    int64_t by[kWalk];
    uint32_t rec[kWalk];
    bool ok[kWalk];
#pragma unroll
    for (int u = 0; u < kWalk; ++u) {
      ok[u] = y - u >= ylo;
      by[u] = 0;
      rec[u] = 0;
      if (ok[u]) rec_of(y - u, by[u], rec[u]);
      ok[u] = ok[u] && by[u] + Z > m;
    }
    float xv[kWalk];
#pragma unroll
    for (int u = 0; u < kWalk; ++u) {
      const uint32_t id = rec[u] & 0x7fffffffu;
      const uint32_t run = id / rsC, j = id - run * rsC;
      xv[u] = ok[u] ? rs[static_cast<uint64_t>(run) * rsD + j * p.Z +
                         static_cast<uint32_t>(m - by[u])]
                    : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kWalk; ++u)
      if (ok[u]) v += (rec[u] >> 31) ? -xv[u] : xv[u];
    if (!ok[kWalk - 1]) break;
  }
  return v;
}

template <int MODE, typename WT, bool ADAGRAD>
__global__ __launch_bounds__(kBlockThreads) void emit_kernel(
    const KParams p, const uint32_t* __restrict__ cb, const uint32_t* __restrict__ cv,
    const uint32_t* __restrict__ info, const uint32_t* __restrict__ slot,
    const uint32_t* __restrict__ total, const float* __restrict__ rs, const uint32_t rsC,
    const uint32_t rsD, const EmitList list, const EmitUpdate<WT> upd) {
  __shared__ int32_t sbase_all[kWavesPerBlock][kStage];
  __shared__ uint32_t srec_all[kWavesPerBlock][kStage];
  int32_t* sbase = sbase_all[threadIdx.x >> 6];
  uint32_t* srec = srec_all[threadIdx.x >> 6];
  const int lane = threadIdx.x & (kWave - 1);
  const ExtList el{cb, info[0], info[1], p.M};
  const int64_t L = el.len();
  const uint32_t U = *total;
  const int64_t chunks = (L + kWave - 1) / kWave;
  const int64_t wave0 = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + (threadIdx.x >> 6);
  const int64_t nwaves = static_cast<int64_t>(gridDim.x) * kWavesPerBlock;
  const int64_t Z = p.Z;
  for (int64_t chunk = wave0; chunk < chunks; chunk += nwaves) {
    const int64_t x0 = chunk * kWave;
    const int64_t x = x0 + lane;
    uint32_t o = 0, first = 0;
    int64_t lo = 0;
    if (x < L) {
      first = slot[x];
      o = (x + 1 < L ? slot[x + 1] : U) - first;
      const int64_t b = el.base(static_cast<uint32_t>(x));
      lo = b < 0 ? 0 : b;
    }
    // exclusive prefix of o over the lanes
    uint32_t incl = o;
#pragma unroll
    for (int sh = 1; sh < kWave; sh <<= 1) {
      const uint32_t y = __shfl_up(incl, sh);
      if (lane >= sh) incl += y;
    }
    const uint32_t pre = incl - o;
    const uint32_t T = __shfl(incl, kWave - 1);
    if (T == 0) continue;
    // Records before x0 that can still cover an element owned here: every
    // such element is >= base(x0), so they are those with base > base(x0) - Z
    // (a contiguous run ending at x0 - 1, bases being in ascending order).
    const int64_t b0 = el.base(static_cast<uint32_t>(x0));
    const int64_t xend = x0 + kWave < L ? x0 + kWave : L;
    int64_t ymin = x0;
    bool fits = true;
    while (ymin > 0) {
      const int64_t y = ymin - 1 - lane;
      const bool cov = y >= 0 && el.base(static_cast<uint32_t>(y)) + Z > b0;
      const uint64_t stop = __ballot(!cov);
      if (stop == 0) {  // all 64 records before ymin cover: keep going back
        ymin -= kWave;
        if (xend - ymin > kStage) {  // too many to stage: walk from memory
          fits = false;
          break;
        }
        continue;
      }
      ymin -= __builtin_ctzll(stop);
      break;
    }
    const bool staged = fits && xend - ymin <= kStage;
    if (staged) {
      // the previous chunk's reads of this wave's LDS rows are complete
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      for (int64_t i = lane; i < xend - ymin; i += kWave) {
        sbase[i] = static_cast<int32_t>(el.base(static_cast<uint32_t>(ymin + i)));
        srec[i] = cv[el.sorted_index(static_cast<uint32_t>(ymin + i))];
      }
      __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
      __builtin_amdgcn_wave_barrier();
    }
    for (uint32_t b0e = 0; b0e < T; b0e += kWave) {
      const uint32_t e = b0e + static_cast<uint32_t>(lane);
      // record of element e: the largest lane r with pre[r] <= e
      int r = 0;
#pragma unroll
      for (int step = kWave / 2; step >= 1; step >>= 1) {
        const int probe = r + step;
        if (__shfl(pre, probe) <= e) r = probe;
      }
      const uint32_t off = e - __shfl(pre, r);
      const int64_t xr = x0 + r;
      const int64_t m = __shfl(lo, r) + off;
      const uint32_t k = __shfl(first, r) + off;
      if (e >= T) continue;
      float v;
      if (staged) {
        v = walk_sum(p, rs, rsC, rsD, m, xr - ymin, 0, [&](int64_t y, int64_t& by, uint32_t& rec) {
          by = sbase[y];
          rec = srec[y];
        });
      } else {
        v = walk_sum(p, rs, rsC, rsD, m, xr, 0, [&](int64_t y, int64_t& by, uint32_t& rec) {
          by = el.base(static_cast<uint32_t>(y));
          rec = cv[el.sorted_index(static_cast<uint32_t>(y))];
        });
      }
      if (MODE == 0) {
        if (static_cast<int64_t>(k) < list.capacity) {
          list.locations[k] = static_cast<uint32_t>(m);
          list.values[k] = v;
        }
      } else {
        update_element<WT, ADAGRAD>(upd, static_cast<uint32_t>(m), v);
      }
    }
  }
  (void)Z;
}

// ---------------------------------------------------------------------------
// pre-merge of records that share a base
// ---------------------------------------------------------------------------
// Records with one base cover the same Z elements: their signed run-sum
// pieces are summed once per base (in record order) before the ownership
// and emit steps, so that an element's walk meets at most Z records however
// many chunks hash to its neighbourhood.
constexpr uint32_t kNoBase = 0xffffffffu;

// hd[x] = 1 where record x starts a new base (records before the sentinels).
__global__ __launch_bounds__(kBlockThreads) void merge_heads_kernel(
    const uint32_t* __restrict__ cb, const uint32_t* __restrict__ num_runs, const uint32_t C,
    uint32_t* __restrict__ hd) {
  const int64_t rc = static_cast<int64_t>(*num_runs) * C;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlockThreads;
  for (int64_t x = static_cast<int64_t>(blockIdx.x) * kBlockThreads + threadIdx.x; x < rc;
       x += stride) {
    const uint32_t b = cb[x];
    hd[x] = b != kNoBase && (x == 0 || cb[x - 1] != b) ? 1u : 0u;
  }
}

// After the scan of hd: hpos[u] = position of the u-th head; the records of
// base u are [hpos[u], hpos[u + 1]), hpos[U] = first sentinel position.
__global__ __launch_bounds__(kBlockThreads) void merge_positions_kernel(
    const uint32_t* __restrict__ cb, const uint32_t* __restrict__ num_runs, const uint32_t C,
    const uint32_t* __restrict__ hd, const uint32_t* __restrict__ num_bases,
    uint32_t* __restrict__ hpos) {
  const int64_t rc = static_cast<int64_t>(*num_runs) * C;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlockThreads;
  for (int64_t x = static_cast<int64_t>(blockIdx.x) * kBlockThreads + threadIdx.x; x < rc;
       x += stride) {
    const uint32_t b = cb[x];
    const uint32_t prev = x > 0 ? cb[x - 1] : kNoBase;
    if (b != kNoBase && (x == 0 || prev != b)) hpos[hd[x]] = static_cast<uint32_t>(x);
    // the end of the last base: the first sentinel, or rc
    if ((b == kNoBase && (x == 0 || prev != kNoBase)) || (b != kNoBase && x + 1 == rc))
      hpos[*num_bases] = static_cast<uint32_t>(b == kNoBase ? x : rc);
  }
}

// One wavefront per base u: mrs[u * Z + k] = sum over its records of the
// signed run-sum entry k; mb[u] = base, mv[u] = u.  Record ids are
// requested 64 at a time and their entries kMergeBatch at a time.
constexpr int kMergeBatch = 8;
__global__ __launch_bounds__(kBlockThreads) void merge_sums_kernel(
    const KParams p, const uint32_t* __restrict__ cb, const uint32_t* __restrict__ cv,
    const uint32_t* __restrict__ hpos, const uint32_t* __restrict__ num_bases,
    const float* __restrict__ rs, float* __restrict__ mrs, uint32_t* __restrict__ mb,
    uint32_t* __restrict__ mv) {
  const int lane = threadIdx.x & (kWave - 1);
  const uint32_t U = *num_bases;
  const uint64_t nwaves = static_cast<uint64_t>(gridDim.x) * kWavesPerBlock;
  for (uint64_t u = static_cast<uint64_t>(blockIdx.x) * kWavesPerBlock + (threadIdx.x >> 6); u < U;
       u += nwaves) {
    const uint32_t lo = hpos[u], hi = hpos[u + 1];
    for (uint32_t k0 = 0; k0 < p.Z; k0 += kWave) {
      const uint32_t k = k0 + lane;
      float acc = 0.f;
      for (uint32_t x0 = lo; x0 < hi; x0 += kWave) {
        const uint32_t nx = hi - x0 < static_cast<uint32_t>(kWave) ? hi - x0 : kWave;
        const uint32_t myid = static_cast<uint32_t>(lane) < nx ? cv[x0 + lane] : 0u;
        for (uint32_t q0 = 0; q0 < nx; q0 += kMergeBatch) {
          float v[kMergeBatch];
#pragma unroll
          for (int t = 0; t < kMergeBatch; ++t) {
            const uint32_t q = q0 + t < nx ? q0 + t : nx - 1;
            const uint32_t id = readlane_u32(myid, static_cast<int>(q));
            const uint32_t run = (id & 0x7fffffffu) / p.C, j = (id & 0x7fffffffu) - run * p.C;
            const float x = k < p.Z ? rs[static_cast<uint64_t>(run) * p.d + j * p.Z + k] : 0.f;
            v[t] = (id >> 31) ? -x : x;
          }
#pragma unroll
          for (int t = 0; t < kMergeBatch; ++t)
            if (q0 + t < nx) acc += v[t];
        }
      }
      if (k < p.Z) mrs[u * p.Z + k] = acc;
    }
    if (lane == 0) {
      mb[u] = cb[lo];
      mv[u] = static_cast<uint32_t>(u);
    }
  }
}

// tail_count for the merged list: U bases, no sentinels.
__global__ void tail_count_merged_kernel(const KParams p, const uint32_t* __restrict__ mb,
                                         const uint32_t* __restrict__ num_bases,
                                         uint32_t* __restrict__ info) {
  const uint64_t rc = *num_bases;
  uint64_t lo = 0, hi = rc;
  const uint32_t lim = p.M - p.Z;
  while (lo < hi) {
    const uint64_t mid = (lo + hi) / 2;
    if (mb[mid] > lim) hi = mid; else lo = mid + 1;
  }
  info[0] = static_cast<uint32_t>(rc);
  info[1] = static_cast<uint32_t>(rc - lo);
  info[3] = static_cast<uint32_t>(rc + (rc - lo));
}

__global__ void store_count_kernel(const uint32_t* __restrict__ total, int64_t* __restrict__ out) {
  *out = *total;
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------

// Records have 31-bit ids (bit 31 carries the sign): N*C must stay below 2^31.
static int64_t record_cap(const KParams& p) { return p.N * static_cast<int64_t>(p.C); }

// Pre-merge when the chunk records average at least 16 per base of the
// array (N * C >= 16 * M, an upper bound: runs are at most lookups).
// Measured on post-hoc compression of 10^7 x 128 entries (Z = 32): 1000x
// 51.6 -> 6.5 ms, 10000x 142 -> 6.1 ms; at 100x (3 records per base) even,
// at 10x 3.4x slower, and 1.3-2x slower on the benchmark batches (2.7-4.3
// records per base), whose walks are already short.
static bool sparse_merges(const KParams& p) {
  return record_cap(p) >= 16 * static_cast<int64_t>(p.M);
}

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
  if (sparse_merges(p)) {
    const int64_t ub = cap < static_cast<int64_t>(p.M) ? cap : static_cast<int64_t>(p.M);
    s += static_cast<size_t>(cap) * 4 + scan_scratch_bytes(cap) + static_cast<size_t>(cap + 1) * 4 +
         static_cast<size_t>(ub) * (p.Z + 2) * 4 + 64;  // pre-merge
  }
  if (p.mean) s += static_cast<size_t>(p.num_bags) * 4;  // 1 / |bag| per pooled row
  return s + 72 * 16;  // alignment slack
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

// Blocks of a grid-stride launch over at most n items.
static uint32_t grid_stride_blocks(int64_t n) {
  const int64_t b = (n + kBlockThreads - 1) / kBlockThreads;
  return static_cast<uint32_t>(b < 1 ? 1 : (b > 8192 ? 8192 : b));
}

static uint32_t emit_blocks(int64_t cap2) {
  const int64_t waves = (cap2 + kWave - 1) / kWave;
  const int64_t want = (waves + kWavesPerBlock - 1) / kWavesPerBlock;
  return static_cast<uint32_t>(want < 1 ? 1 : (want > 16384 ? 16384 : want));
}

// Everything up to the scanned ownership; returns the buffers the emit
// step reads.
struct SparseState {
  const uint32_t *cb, *cv, *info, *own;
  const float* rs;
  uint32_t rsC, rsD;  // record id -> rs entry: (id / rsC) * rsD + (id % rsC) * Z + offset
  int64_t cap2;
};

static hipError_t sparse_prepare(const KParams& p, const void* indices, const void* offsets,
                                 const void* grad, void* workspace, uint32_t* num_unique32,
                                 SparseState* st, hipStream_t stream) {
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
  const bool merge = sparse_merges(p);
  const int64_t ub = cap < static_cast<int64_t>(p.M) ? cap : static_cast<int64_t>(p.M);
  uint32_t* hd = merge ? carve<uint32_t>(cur, cap) : nullptr;
  uint32_t* hscr = merge ? carve<uint32_t>(cur, scan_scratch_bytes(cap) / 4 + 1) : nullptr;
  uint32_t* hpos = merge ? carve<uint32_t>(cur, cap + 1) : nullptr;
  uint32_t* num_bases = merge ? carve<uint32_t>(cur, 4) : nullptr;
  float* mrs = merge ? carve<float>(cur, static_cast<size_t>(ub) * p.Z) : nullptr;
  uint32_t* mb = merge ? carve<uint32_t>(cur, ub) : nullptr;
  uint32_t* mv = merge ? carve<uint32_t>(cur, ub) : nullptr;

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
  hipLaunchKernelGGL(chunk_records_kernel, dim3(grid_stride_blocks(cap)), dim3(kBlockThreads), 0,
                     stream, p, rk, num_runs, cap, cb, cv, info);
  e = hipGetLastError();
  uint32_t* cbs = cb;
  uint32_t* cvs = cv;
  // only the runs * C records that exist are sorted, owned and scanned
  if (e == hipSuccess)
    e = radix_sort_pairs(cbs, cvs, cb1, cv1, cap, base_bits(p.M), cscr, stream, info + 2);
  if (e != hipSuccess) return e;
  if (!merge) {
    hipLaunchKernelGGL(tail_count_kernel, dim3(1), dim3(1), 0, stream, p, cbs, num_runs, info);
    hipLaunchKernelGGL(own_kernel, dim3(grid_stride_blocks(cap2)), dim3(kBlockThreads), 0, stream,
                       p, cbs, info, own);
    e = exclusive_scan(own, cap2, oscr, num_unique32, stream, info + 3);
    if (e != hipSuccess) return e;
    *st = SparseState{cbs, cvs, info, own, rs, p.C, p.d, cap2};
    return hipSuccess;
  }
  // pre-merge: one record per distinct base
  hipLaunchKernelGGL(merge_heads_kernel, dim3(grid_stride_blocks(cap)), dim3(kBlockThreads), 0,
                     stream, cbs, num_runs, p.C, hd);
  e = exclusive_scan(hd, cap, hscr, num_bases, stream, info + 2);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(merge_positions_kernel, dim3(grid_stride_blocks(cap)), dim3(kBlockThreads), 0,
                     stream, cbs, num_runs, p.C, hd, num_bases, hpos);
  {
    const int64_t want = (ub + kWavesPerBlock - 1) / kWavesPerBlock;  // a wavefront per base
    const uint32_t mblocks = static_cast<uint32_t>(want < 1 ? 1 : (want > 65536 ? 65536 : want));
    hipLaunchKernelGGL(merge_sums_kernel, dim3(mblocks), dim3(kBlockThreads), 0, stream, p, cbs,
                       cvs, hpos, num_bases, rs, mrs, mb, mv);
  }
  hipLaunchKernelGGL(tail_count_merged_kernel, dim3(1), dim3(1), 0, stream, p, mb, num_bases, info);
  hipLaunchKernelGGL(own_kernel, dim3(grid_stride_blocks(cap2)), dim3(kBlockThreads), 0, stream, p,
                     mb, info, own);
  e = exclusive_scan(own, cap2, oscr, num_unique32, stream, info + 3);
  if (e != hipSuccess) return e;
  *st = SparseState{mb, mv, info, own, mrs, 1u, p.Z, cap2};
  return hipSuccess;
}

hipError_t launch_gradient_sparse(const KParams& p, const void* indices, const void* offsets,
                                  const void* grad, void* workspace, uint32_t* locations,
                                  float* values, int64_t capacity, uint32_t* num_unique32,
                                  hipStream_t stream) {
  SparseState st;
  hipError_t e = sparse_prepare(p, indices, offsets, grad, workspace, num_unique32, &st, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((emit_kernel<0, float, false>), dim3(emit_blocks(st.cap2)), dim3(kBlockThreads),
                     0, stream, p, st.cb, st.cv, st.info, st.own, num_unique32, st.rs, st.rsC,
                     st.rsD, EmitList{locations, values, capacity},
                     EmitUpdate<float>{nullptr, nullptr, 0.f, 0.f});
  return hipGetLastError();
}

template <typename WT>
static void launch_emit_update(const KParams& p, const SparseState& st, const uint32_t* total,
                               WT* w, float* state, float lr, float eps, hipStream_t stream) {
  const EmitList none{nullptr, nullptr, 0};
  const EmitUpdate<WT> u{w, state, lr, eps};
  if (state)
    hipLaunchKernelGGL((emit_kernel<1, WT, true>), dim3(emit_blocks(st.cap2)), dim3(kBlockThreads), 0,
                       stream, p, st.cb, st.cv, st.info, st.own, total, st.rs, st.rsC, st.rsD,
                       none, u);
  else
    hipLaunchKernelGGL((emit_kernel<1, WT, false>), dim3(emit_blocks(st.cap2)), dim3(kBlockThreads), 0,
                       stream, p, st.cb, st.cv, st.info, st.own, total, st.rs, st.rsC, st.rsD,
                       none, u);
}

hipError_t launch_sparse_update(const KParams& p, const void* indices, const void* offsets,
                                const void* grad, void* workspace, uint32_t* num_unique32, void* w,
                                bool bf16, float* state, float lr, float eps, hipStream_t stream) {
  SparseState st;
  hipError_t e = sparse_prepare(p, indices, offsets, grad, workspace, num_unique32, &st, stream);
  if (e != hipSuccess) return e;
  if (bf16)
    launch_emit_update(p, st, num_unique32, static_cast<uint16_t*>(w), state, lr, eps, stream);
  else
    launch_emit_update(p, st, num_unique32, static_cast<float*>(w), state, lr, eps, stream);
  return hipGetLastError();
}

hipError_t launch_store_count(const uint32_t* total, int64_t* out, hipStream_t stream) {
  hipLaunchKernelGGL(store_count_kernel, dim3(1), dim3(1), 0, stream, total, out);
  return hipGetLastError();
}

}  // namespace pss
