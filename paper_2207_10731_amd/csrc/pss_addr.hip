// Address-sorted deposit: Alg. 1's scatter_add with the contributions
// ordered by address instead of added with atomics.
//
// Made for the regime where lookups rarely repeat and a chunk is shorter
// than a memory line (the per-element hashing trick on an array held in HBM):
// grouping by token then removes nothing, and every contribution would be a
// float atomic to a different line, carried out at the memory side.  Here
// each contribution becomes a record and each tile of the array is written
// once:
//
//   records  item e, dim c -> (address (h(i, j) + k) mod M, scale * s * grad),
//            at position e*d + c (the gradient rows are read in bag order);
//            a chunk of factor 0 gives -0.0, which changes nothing
//   sort     LSD radix sort of the records by address tile (the address bits
//            from kAddrTileShift up; 8-bit digits, stable)
//   starts   first record of every tile: a binary search of the sorted
//            addresses per tile
//   apply    one workgroup per tile of 2^kAddrTileShift elements: the tile's
//            records are summed into an LDS copy of the tile (LDS float
//            atomics, initialised to -0.0 so that an element without records
//            keeps its bits), then the tile is added to dst in one streaming
//            pass (fused SGD) or stored as the tile of a float32 gradient
//            buffer (every element of it, so the buffer needs no zero-fill).
//
// Run sums by address (chunks of 64 elements or more, updates through G):
// the lookups are first grouped by token as for the grouped deposit, and
// each run's summed gradient row becomes the contribution: one record per
// run and chunk, (chunk base, payload row of Z values).  The records are
// radix-sorted by the tile of their base, and one workgroup per tile sums
// the payloads of every chunk that reaches the tile (its own, the previous
// tile's spilling over the boundary and, for tile 0, those wrapping past M)
// in LDS, each wavefront owning a range of the tile and adding in record
// order, then applies SGD or Adagrad to the tile's elements in place: no
// atomics at all, no G buffer, no dense optimizer pass, and every sum taken
// in a fixed order (the update is bit-identical run to run).  Opt-in: with
// chunks this long the atomic deposit moves whole lines and is faster.
#include "pss_launch.hpp"

namespace pss {

constexpr uint32_t kAddrTile = 1u << kAddrTileShift;  // elements per tile
constexpr int kApplyThreads = 512;

// Records of the items of one 64-bag tile (one wavefront): lanes over the
// dims (c = lane + 64 s), U items' gradient rows requested before any of
// their records is written.
template <int EPL, int U, bool SIGN, typename GT>
__global__ __launch_bounds__(kBlockThreads) void addr_records_kernel(
    const KParams p, const void* __restrict__ indices, const void* __restrict__ offsets,
    const GT* __restrict__ grad, const float scale, uint32_t* __restrict__ keys,
    uint32_t* __restrict__ vals) {
  const int lane = threadIdx.x & (kWave - 1);
  const uint64_t wave = static_cast<uint64_t>(blockIdx.x) * kWavesPerBlock + (threadIdx.x >> 6);
  const uint64_t g0 = wave * kTileBags;
  if (g0 >= p.num_bags) return;
  const Tile tl = load_tile(p, offsets, g0, lane);
  // pooled row r = b*T + t of bag g0 + lane
  const uint64_t g = g0 + static_cast<uint64_t>(lane < tl.nb ? lane : 0);
  const uint32_t t = static_cast<uint32_t>(g / p.B);
  const uint32_t rr = static_cast<uint32_t>(g - static_cast<uint64_t>(t) * p.B) * p.T + t;

  uint32_t step[EPL], step2[EPL], kk[EPL], cc[EPL];
  bool act[EPL];
#pragma unroll
  for (int s = 0; s < EPL; ++s) {
    const uint32_t c = static_cast<uint32_t>(lane) + kWave * s;
    act[s] = c < p.d;
    cc[s] = act[s] ? c : 0u;
    const uint32_t j = cc[s] / p.Z;
    kk[s] = cc[s] - j * p.Z;
    step[s] = chunk_step(p.a, j);
    step2[s] = SIGN ? chunk_step(p.a2, j) : 0u;
  }

  for (int64_t blk = tl.E0; blk < tl.E1; blk += kWave) {
    const int64_t rem = tl.E1 - blk;
    const int n = rem < kWave ? static_cast<int>(rem) : kWave;
    const int64_t e = blk + lane;
    const int bag = bag_of_item(tl, e);
    const uint32_t tC = __shfl(tl.tC, bag);
    const uint32_t r_l = __shfl(rr, bag);
    uint32_t h0 = 0;
    if (lane < n) h0 = item_hash(load_index(indices, e, p.idx32), tC, p.TC, p.a, p.b);
    float il_l = 1.f;
    if (p.mean) {
      const uint32_t len = __shfl(tl.len, bag);
      il_l = len ? 1.f / static_cast<float>(len) : 1.f;
    }
    for (int q0 = 0; q0 < n; q0 += U) {
      float x[U][EPL];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int q = q0 + u < n ? q0 + u : n - 1;  // past the end: repeat the last item
        const GT* row = grad + static_cast<uint64_t>(readlane_u32(r_l, q)) * p.d;
#pragma unroll
        for (int s = 0; s < EPL; ++s) x[u][s] = load_row(row, cc[s]);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (q0 + u >= n) break;
        const int q = q0 + u;
        const uint32_t h = readlane_u32(h0, q);
        const float f = scale * (p.mean ? __builtin_bit_cast(float, readlane_u32(
                                                                  __builtin_bit_cast(uint32_t, il_l), q))
                                        : 1.f);
        const uint32_t h20 = SIGN ? sign_hash0(h, p.s_alpha, p.s_beta) : 0u;
        const uint64_t rec = static_cast<uint64_t>(blk + q) * p.d;
#pragma unroll
        for (int s = 0; s < EPL; ++s) {
          if (!act[s]) continue;
          const uint32_t ent =
              chunk_entry<SIGN>(fast_mod(add_mod_p(h, step[s]), p.fm_c, p.M), add_mod_p(h20, step2[s]), p);
          const Elem el = elem_of<SIGN>(ent, kk[s], p.M);
          float v = f * x[u][s];
          if (SIGN) v = el.read ? __uint_as_float(__float_as_uint(v) ^ el.neg) : -0.f;
          keys[rec + cc[s]] = el.m;
          vals[rec + cc[s]] = __float_as_uint(v);
        }
      }
    }
  }
}

// starts[x] = first record of tile x (records sorted by tile), for x in
// [0, ntiles]; starts[ntiles] = the number of records with an address.  One thread per entry: a binary search
// for the first record whose tile is at least x.
__global__ __launch_bounds__(kBlockThreads) void addr_starts_kernel(const uint32_t* __restrict__ keys,
                                                                    const uint32_t n, const uint32_t ntiles,
                                                                    uint32_t* __restrict__ starts) {
  const uint32_t x = blockIdx.x * kBlockThreads + threadIdx.x;
  if (x > ntiles) return;
  uint32_t lo = 0, hi = n;
  while (lo < hi) {
    const uint32_t mid = lo + ((hi - lo) >> 1);
    uint32_t t = keys[mid] >> kAddrTileShift;
    t = t > ntiles ? ntiles : t;  // records without an address (kNoRecord) sort last
    if (t < x) lo = mid + 1; else hi = mid;
  }
  starts[x] = lo;
}

// One workgroup per tile of the array: sum the tile's records in LDS, then
// apply the tile to dst once.
__global__ __launch_bounds__(kApplyThreads) void addr_apply_kernel(
    float* __restrict__ dst, const uint32_t assign, const uint32_t M,
    const uint32_t* __restrict__ keys, const uint32_t* __restrict__ vals,
    const uint32_t* __restrict__ starts) {
  __shared__ float tile[kAddrTile];
  const uint32_t x = blockIdx.x;
  const uint64_t base = static_cast<uint64_t>(x) << kAddrTileShift;
  const uint32_t len = M - base < kAddrTile ? static_cast<uint32_t>(M - base) : kAddrTile;
  for (uint32_t i = threadIdx.x; i < kAddrTile; i += kApplyThreads) tile[i] = -0.f;
  __syncthreads();
  const uint32_t lo = starts[x], hi = starts[x + 1];
  for (uint32_t r = lo + threadIdx.x; r < hi; r += kApplyThreads)
    atomicAdd(&tile[keys[r] & (kAddrTile - 1)], __uint_as_float(vals[r]));
  __syncthreads();
  float* out = dst + base;
  if (len == kAddrTile) {
    float4* o4 = reinterpret_cast<float4*>(out);
    const float4* t4 = reinterpret_cast<const float4*>(tile);
    for (uint32_t i = threadIdx.x; i < kAddrTile / 4; i += kApplyThreads) {
      float4 v = t4[i];
      if (!assign) {
        const float4 w = o4[i];
        v = make_float4(w.x + v.x, w.y + v.y, w.z + v.z, w.w + v.w);
      }
      o4[i] = v;
    }
  } else {
    for (uint32_t i = threadIdx.x; i < len; i += kApplyThreads) out[i] = assign ? tile[i] : out[i] + tile[i];
  }
}

static uint32_t addr_tiles(const KParams& p) {
  return static_cast<uint32_t>((static_cast<uint64_t>(p.M) + kAddrTile - 1) >> kAddrTileShift);
}

size_t addr_workspace_bytes(const KParams& p) {
  const uint64_t n = static_cast<uint64_t>(p.N) * p.d;
  return n * 16 + radix_scratch_bytes(static_cast<int64_t>(n)) +
         (static_cast<size_t>(addr_tiles(p)) + 1) * 4 + 256;
}

template <int EPL, int U, bool SIGN, typename GT>
static void launch_records_t(const KParams& p, const void* indices, const void* offsets,
                             const GT* grad, float scale, uint32_t* keys, uint32_t* vals,
                             hipStream_t stream) {
  const uint64_t tiles = (p.num_bags + kTileBags - 1) / kTileBags;
  const uint64_t blocks = (tiles + kWavesPerBlock - 1) / kWavesPerBlock;
  hipLaunchKernelGGL((addr_records_kernel<EPL, U, SIGN, GT>), dim3(static_cast<uint32_t>(blocks)),
                     dim3(kBlockThreads), 0, stream, p, indices, offsets, grad, scale, keys, vals);
}

template <bool SIGN, typename GT>
static void launch_records_s(const KParams& p, const void* indices, const void* offsets,
                             const GT* grad, float scale, uint32_t* keys, uint32_t* vals,
                             hipStream_t stream) {
  if (p.d <= 64) return launch_records_t<1, 8, SIGN>(p, indices, offsets, grad, scale, keys, vals, stream);
  if (p.d <= 128) return launch_records_t<2, 8, SIGN>(p, indices, offsets, grad, scale, keys, vals, stream);
  if (p.d <= 256) return launch_records_t<4, 4, SIGN>(p, indices, offsets, grad, scale, keys, vals, stream);
  if (p.d <= 1024) return launch_records_t<16, 1, SIGN>(p, indices, offsets, grad, scale, keys, vals, stream);
  return launch_records_t<64, 1, SIGN>(p, indices, offsets, grad, scale, keys, vals, stream);
}

template <typename GT>
static void launch_records_g(const KParams& p, const void* indices, const void* offsets,
                             const GT* grad, float scale, uint32_t* keys, uint32_t* vals,
                             hipStream_t stream) {
  if (p.sign_mode) return launch_records_s<true>(p, indices, offsets, grad, scale, keys, vals, stream);
  return launch_records_s<false>(p, indices, offsets, grad, scale, keys, vals, stream);
}

hipError_t launch_deposit_addr(float* dst, bool assign, float scale, const KParams& p,
                               const void* indices, const void* offsets, const void* grad,
                               void* workspace, hipStream_t stream) {
  const uint64_t n = static_cast<uint64_t>(p.N) * p.d;
  if (n >= (1ull << 31)) return hipErrorInvalidValue;
  const uint32_t ntiles = addr_tiles(p);
  uint32_t* k0 = static_cast<uint32_t*>(workspace);
  uint32_t* v0 = k0 + n;
  uint32_t* k1 = v0 + n;
  uint32_t* v1 = k1 + n;
  uint32_t* scratch = v1 + n;
  uint32_t* starts = reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(scratch) +
                                                 radix_scratch_bytes(static_cast<int64_t>(n)));
  if (n > 0) {
    if (p.rows_bf16)
      launch_records_g(p, indices, offsets, static_cast<const uint16_t*>(grad), scale, k0, v0, stream);
    else
      launch_records_g(p, indices, offsets, static_cast<const float*>(grad), scale, k0, v0, stream);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // tile bits of the addresses (0 when the whole array is one tile)
    int bits = 0;
    while ((1ull << bits) < ntiles) ++bits;
    e = radix_sort_pairs(k0, v0, k1, v1, static_cast<int64_t>(n), bits, scratch, stream, nullptr,
                         false, kAddrTileShift);
    if (e != hipSuccess) return e;
  }
  const uint32_t sgrid = (ntiles + 1 + kBlockThreads - 1) / kBlockThreads;
  hipLaunchKernelGGL(addr_starts_kernel, dim3(sgrid), dim3(kBlockThreads), 0, stream, k0,
                     static_cast<uint32_t>(n), ntiles, starts);
  hipLaunchKernelGGL(addr_apply_kernel, dim3(ntiles), dim3(kApplyThreads), 0, stream, dst,
                     assign ? 1u : 0u, p.M, k0, v0, starts);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Run sums by address
// ---------------------------------------------------------------------------
constexpr int kRunsApplyThreads = 1024;
constexpr int kRunsBatch = 8;  // records whose payload pieces are requested together
constexpr int kRunsOpt = 4;    // elements per lane updated together
constexpr uint32_t kRunsStage = 1024;  // records staged in LDS at a time

// Whether the chunk of Z elements from `base` (wrapping past M) has an
// element in [x0, x0 + len).
__device__ __forceinline__ bool chunk_reaches(uint32_t base, uint32_t Z, uint32_t M, uint32_t x0,
                                              uint32_t len) {
  const uint64_t last = static_cast<uint64_t>(base) + Z - 1;
  if (last < M) return base < x0 + len && last >= x0;
  return base < x0 + len || x0 <= last - M;  // [base, M) and [0, last - M]
}

// One workgroup per tile of the array, each of its wavefronts owning a
// range of kRunsRange consecutive elements of the tile in LDS.  Records are
// (base, slot): the chunk covers elements (base + k) mod M, k < Z, with
// values payload[slot * Z + k].  Every wavefront walks the records of the
// tiles whose chunks can reach this one and adds the part of each chunk
// that falls in its own range with plain LDS read-add-writes: no two
// wavefronts touch one element, and a wavefront adds one chunk at a time
// (its lanes on distinct elements), so no atomics are needed and each
// element's sum is taken in the records' sorted order.  The wavefront then
// applies the update to its range.
constexpr uint32_t kRunsRange = kAddrTile / (kRunsApplyThreads / kWave);  // 1024

template <typename WT, bool ADAGRAD>
__global__ __launch_bounds__(kRunsApplyThreads) void runs_apply_kernel(
    WT* __restrict__ w, float* __restrict__ s, const uint32_t M, const uint32_t Z,
    const uint32_t ntiles, const uint32_t* __restrict__ keys, const uint32_t* __restrict__ slots,
    const uint32_t* __restrict__ starts, const float* __restrict__ payload, const float lr,
    const float eps) {
  __shared__ float tile[kAddrTile];
  const uint32_t x = blockIdx.x;
  const uint32_t x0 = x << kAddrTileShift;
  const uint32_t len = M - x0 < kAddrTile ? M - x0 : kAddrTile;
  // Tiles whose chunks can reach this one: itself; the previous tile (a
  // chunk of at most 4096 elements crosses at most one boundary of a full
  // tile); for tile 0 the last two (chunks wrapping past M, the last tile
  // possibly shorter than a chunk).
  uint32_t src[3];
  int nsrc = 0;
  src[nsrc++] = x;
  if (x >= 1) src[nsrc++] = x - 1;
  if (x == 0 && ntiles >= 2) src[nsrc++] = ntiles - 1;
  if (x == 0 && ntiles >= 3) src[nsrc++] = ntiles - 2;
  uint32_t total = 0;
  for (int i = 0; i < nsrc; ++i) total += starts[src[i] + 1] - starts[src[i]];
  if (total == 0) return;  // whole workgroup: G = 0 on this tile, nothing changes
  __shared__ uint32_t sbase[kRunsStage], sslot[kRunsStage];
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & (kWave - 1);
  // this wavefront's elements: [r0, r0 + rlen) of the array
  const uint32_t r0 = x0 + wv * kRunsRange;
  const uint32_t rend = x0 + len;
  const uint32_t rlen = r0 >= rend ? 0u : (rend - r0 < kRunsRange ? rend - r0 : kRunsRange);
  float* acc = tile + wv * kRunsRange;
  for (uint32_t i = lane; i < kRunsRange; i += kWave) acc[i] = 0.f;
  bool touched = false;
  for (int i = 0; i < nsrc; ++i) {
    const uint32_t lo = starts[src[i]], hi = starts[src[i] + 1];
    for (uint32_t c0 = lo; c0 < hi; c0 += kRunsStage) {
      // the workgroup stages up to kRunsStage records in LDS; every
      // wavefront then picks those reaching its range
      const uint32_t cn = hi - c0 < kRunsStage ? hi - c0 : kRunsStage;
      __syncthreads();  // the previous stage has been read
      for (uint32_t j = threadIdx.x; j < cn; j += kRunsApplyThreads) {
        sbase[j] = keys[c0 + j];
        sslot[j] = slots[c0 + j];
      }
      __syncthreads();
      if (rlen == 0) continue;  // past the end of a short last tile
      for (uint32_t b0 = 0; b0 < cn; b0 += kWave) {
        uint32_t base = 0, slot = 0;
        bool reach = false;
        if (b0 + lane < cn) {
          base = sbase[b0 + lane];
          slot = sslot[b0 + lane];
          reach = chunk_reaches(base, Z, M, r0, rlen);
        }
        uint64_t todo = __ballot(reach);
        touched |= todo != 0;
        while (todo) {
          // up to kRunsBatch records: their payload pieces are requested
          // before any is added
          uint32_t qs[kRunsBatch];
          int nq = 0;
#pragma unroll
          for (int u = 0; u < kRunsBatch; ++u) {
            qs[u] = todo ? static_cast<uint32_t>(__builtin_ctzll(todo)) : qs[0];
            if (todo) {
              todo &= todo - 1;
              ++nq;
            }
          }
          for (uint32_t k0 = 0; k0 < Z; k0 += kWave) {
            const uint32_t k = k0 + lane;
            float v[kRunsBatch];
            uint32_t off[kRunsBatch];
#pragma unroll
            for (int u = 0; u < kRunsBatch; ++u) {
              const uint32_t bq = readlane_u32(base, qs[u]);
              uint32_t m = bq + k;  // bq < M and k < Z <= M: no overflow
              if (m >= M) m -= M;
              off[u] = m - r0;  // below rlen exactly when m is in the range
              v[u] = 0.f;
              if (u < nq && k < Z && off[u] < rlen)
                v[u] = payload[static_cast<uint64_t>(readlane_u32(slot, qs[u])) * Z + k];
            }
#pragma unroll
            for (int u = 0; u < kRunsBatch; ++u)
              if (u < nq && k < Z && off[u] < rlen) acc[off[u]] += v[u];
          }
        }
      }
    }
  }
  if (rlen == 0) return;
  if (!touched) return;  // no chunk reaches this range: G = 0 on it
  // Each element was written by this wavefront only (its own LDS writes are
  // visible to it in program order).  The range's weights (and states) are
  // read whole, kRunsOpt elements per lane at a time, then updated where
  // G != 0 (elements with G == 0, and lanes past the range's end, store
  // nothing).
  for (uint32_t i0 = 0; i0 < rlen; i0 += kRunsOpt * kWave) {
    float g[kRunsOpt];
#pragma unroll
    for (int u = 0; u < kRunsOpt; ++u) {
      const uint32_t i = i0 + u * kWave + lane;
      g[u] = i < rlen ? acc[i] : 0.f;
    }
    float wo[kRunsOpt], so[kRunsOpt];
#pragma unroll
    for (int u = 0; u < kRunsOpt; ++u) {
      const uint32_t i = i0 + u * kWave + lane;
      const int64_t m = static_cast<int64_t>(r0) + (i < rlen ? i : 0u);
      wo[u] = load_weight64(w, m);
      so[u] = ADAGRAD ? s[m] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kRunsOpt; ++u)
      if (g[u] != 0.f)
        update_loaded<WT, ADAGRAD>(w, s, static_cast<int64_t>(r0) + i0 + u * kWave + lane, g[u],
                                   wo[u], so[u], lr, eps);
  }
}

static int runs_sort_bits(uint32_t ntiles) {
  int bits = 0;  // 2^bits > ntiles: kNoRecord's tile field lies past every tile
  while ((1u << bits) <= ntiles) ++bits;
  return bits;
}

size_t runs_workspace_bytes(const KParams& p) {
  const uint64_t n = static_cast<uint64_t>(p.N) * p.C;
  const uint64_t payload = (static_cast<uint64_t>(p.N) * p.d * 4 + 255) & ~uint64_t(255);
  return payload + n * 16 + radix_scratch_bytes(static_cast<int64_t>(n)) +
         (static_cast<size_t>(addr_tiles(p)) + 1) * 4 + 256;
}

hipError_t launch_deposit_runs(void* w, bool bf16, float* state, float lr, float eps,
                               const KParams& p, const GroupedPairs& g, const void* grad,
                               void* workspace, hipStream_t stream) {
  const uint64_t n = static_cast<uint64_t>(p.N) * p.C;
  if (n >= (1ull << 31) || p.Z > 4096) return hipErrorInvalidValue;
  const uint32_t ntiles = addr_tiles(p);
  float* payload = static_cast<float*>(workspace);
  uint32_t* k0 = reinterpret_cast<uint32_t*>(
      static_cast<char*>(workspace) +
      ((static_cast<uint64_t>(p.N) * p.d * 4 + 255) & ~uint64_t(255)));
  uint32_t* v0 = k0 + n;
  uint32_t* k1 = v0 + n;
  uint32_t* v1 = k1 + n;
  uint32_t* scratch = v1 + n;
  uint32_t* starts = reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(scratch) +
                                                 radix_scratch_bytes(static_cast<int64_t>(n)));
  if (n == 0) return hipSuccess;
  hipError_t e = launch_reduce_records(payload, 1.f, p, g, grad, k0, v0, stream);
  if (e != hipSuccess) return e;
  e = radix_sort_pairs(k0, v0, k1, v1, static_cast<int64_t>(n), runs_sort_bits(ntiles), scratch,
                       stream, nullptr, false, kAddrTileShift);
  if (e != hipSuccess) return e;
  const uint32_t sgrid = (ntiles + 1 + kBlockThreads - 1) / kBlockThreads;
  hipLaunchKernelGGL(addr_starts_kernel, dim3(sgrid), dim3(kBlockThreads), 0, stream, k0,
                     static_cast<uint32_t>(n), ntiles, starts);
  const dim3 grid(ntiles), block(kRunsApplyThreads);
  if (bf16) {
    uint16_t* wb = static_cast<uint16_t*>(w);
    if (state)
      hipLaunchKernelGGL((runs_apply_kernel<uint16_t, true>), grid, block, 0, stream, wb, state,
                         p.M, p.Z, ntiles, k0, v0, starts, payload, lr, eps);
    else
      hipLaunchKernelGGL((runs_apply_kernel<uint16_t, false>), grid, block, 0, stream, wb, state,
                         p.M, p.Z, ntiles, k0, v0, starts, payload, lr, eps);
  } else {
    float* wf = static_cast<float*>(w);
    if (state)
      hipLaunchKernelGGL((runs_apply_kernel<float, true>), grid, block, 0, stream, wf, state, p.M,
                         p.Z, ntiles, k0, v0, starts, payload, lr, eps);
    else
      hipLaunchKernelGGL((runs_apply_kernel<float, false>), grid, block, 0, stream, wf, state,
                         p.M, p.Z, ntiles, k0, v0, starts, payload, lr, eps);
  }
  return hipGetLastError();
}

}  // namespace pss
