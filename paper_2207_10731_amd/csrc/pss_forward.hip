// Forward of the PSS layer: hash -> chunk gather -> sum-pool (paper Sec. 2.4
// forward(i) = (S e_i)^T M with the ROBE-Z mapping of Sec. 2.5).
//
// One wavefront per tile of 64 bags.  Hashing: with C = d/Z <= 16 chunks,
// each lane evaluates the C chunk bases of one item of the current 64-item
// block into a wave-private LDS table and the gathers read their base from
// it (one modular reduction per chunk instead of one per dim); with more
// chunks each lane hashes its own dims (item part on the scalar unit).  U items are gathered before any is consumed so
// that U * EPL loads per lane are in flight.  Pooling runs in registers in
// item order; a finished bag's row is written with non-temporal stores (the
// 4 bytes/dim output stream must not evict the shared array from L2/MALL).
// On gfx9 stores and loads share one wait counter, so the kernel issues all
// U gathers of a batch before any store of that batch: a store is never
// followed by a wait for a load issued after it.
//
// Options: SIGN (template) multiplies each chunk by its sign factor and skips
// chunks of factor 0; mean pooling divides a finished row by the bag's item
// count; rows may be stored as bfloat16 (round to nearest even); indices and
// offsets may be int32.
#include "pss_launch.hpp"

namespace pss {

// Shared arrays larger than the chip's aggregate L2 (8 x 4 MiB) get their
// tiles partitioned over the XCDs (see forward_kernel).  Measured: the
// multi-hot forward on a 64 MB array 1053 -> 867 us, the row-hash forward
// on a 128 MB array 852 -> 832 us; on a 10 MB array the split is neutral
// alone and slower beside a concurrent backward grouping.
constexpr uint64_t kXcdSplitBytes = 32ull << 20;

__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int lane) {
  const uint32_t lo = readlane_u32(static_cast<uint32_t>(v), lane);
  const uint32_t hi = readlane_u32(static_cast<uint32_t>(v >> 32), lane);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Pooled value k of the output: float32, or bfloat16 rounded to nearest even.
__device__ __forceinline__ void store_out(void* out, uint64_t k, float v, uint32_t bf16) {
  if (bf16)
    __builtin_nontemporal_store(f32_to_bf16_rne(v), static_cast<uint16_t*>(out) + k);
  else
    __builtin_nontemporal_store(v, static_cast<float*>(out) + k);
}

// One-hot tile: item l of the tile is bag l.  The (h0, bag) pairs are sorted
// across the lanes; every run of equal h0 is one token, gathered once (U runs
// in flight) and stored to the rows of all its bags.
template <typename WT, int EPL, int U, bool SIGN>
__device__ __forceinline__ void forward_onehot_tile(
    const WT* __restrict__ w, const KParams& p, const Tile& tl, const void* __restrict__ indices,
    void* __restrict__ out, uint32_t* tab, int lane, uint32_t c0, const uint32_t* jj,
    const uint32_t* kk, const bool* act, uint32_t spec) {
  const int nb = tl.nb;
  uint32_t key = 0xffffffffu;  // empty lanes sort last
  uint32_t bag = static_cast<uint32_t>(lane);
  const bool hit = tl.E0 == static_cast<int64_t>(tl.g0);
  if (lane < nb) {
    const uint32_t i = hit ? spec : load_index(indices, tl.E0 + lane, p.idx32);
    key = item_hash(i, tl.tC, p.TC, p.a, p.b);
  }
  wave_sort_pairs(key, bag, lane);
  fill_base_table<SIGN>(tab, key, p, lane);
  const uint32_t prev = __shfl_up(key, 1);
  uint64_t starts = __ballot(lane < nb && (lane == 0 || prev != key));
  while (starts) {
    // next U runs: first positions pos[u], run u covers [pos[u], pos[u+1])
    int pos[U + 1];
#pragma unroll
    for (int u = 0; u <= U; ++u) {
      if (starts) {
        pos[u] = __builtin_ctzll(starts);
        if (u < U) starts &= starts - 1;
      } else {
        pos[u] = nb;
      }
    }
    float v[U][EPL];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int pu = pos[u] < nb ? pos[u] : pos[0];
#pragma unroll
      for (int r = 0; r < EPL; ++r) {
        const Elem el = elem_of<SIGN>(tab[pu * kTabStride + jj[r]], kk[r], p.M);
        const float x = load_weight(w, act[r] ? el.m : 0u);
        v[u][r] = SIGN ? apply_sign(x, el) : x;
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      for (int q = pos[u]; q < pos[u + 1]; ++q) {
        const int b = static_cast<int>(readlane_u32(bag, q));
        const uint64_t ro = readlane_u64(tl.row_off, b) + c0 + lane;
#pragma unroll
        for (int r = 0; r < EPL; ++r)
          if (act[r]) store_out(out, ro + kWave * r, v[u][r], p.rows_bf16);
      }
    }
  }
}

template <typename WT, int EPL, int U, bool TAB, bool SIGN>
__global__ __launch_bounds__(kBlockThreads) void forward_kernel(
    const WT* __restrict__ w, const KParams p, const void* __restrict__ indices,
    const void* __restrict__ offsets, void* __restrict__ out, const uint32_t xcd_split) {
  const int lane = threadIdx.x & (kWave - 1);
  // Workgroups are dispatched round-robin over the chip's XCDs (workgroup b
  // on XCD b mod kXcds), each with an L2 of its own.  Tiles are table-major,
  // so with xcd_split XCD x takes a contiguous share of the tiles and its L2
  // holds the hot tokens of about 1/kXcds of the tables (grid.x is then a
  // multiple of kXcds; any other dispatch order only changes which L2 sees
  // which tile).
  const uint64_t per_xcd = gridDim.x / kXcds;
  const uint64_t blk =
      xcd_split ? (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds : blockIdx.x;
  const uint64_t wave = blk * kWavesPerBlock + (threadIdx.x >> 6);
  const uint64_t g0 = wave * kTileBags;
  if (g0 >= p.num_bags) return;
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

  // One-hot batches: item g0 + lane is usually bag g0 + lane's item; its
  // index is requested together with the offsets.
  uint32_t spec = 0;
  if (TAB && static_cast<int64_t>(g0) + lane < p.N) spec = load_index(indices, g0 + lane, p.idx32);
  const Tile tl = load_tile(p, offsets, g0, lane);

  if (TAB) {
    // One-hot tile (every bag exactly one item): gather each distinct token
    // of the tile once and store its row to every bag that reads it.
    if (__ballot(lane >= tl.nb || tl.len == 1) == ~0ull) {
      forward_onehot_tile<WT, EPL, U, SIGN>(w, p, tl, indices, out, tab, lane, c0, jj, kk, act, spec);
      return;
    }
  }

  float acc[EPL];
#pragma unroll
  for (int r = 0; r < EPL; ++r) acc[r] = 0.f;
  int cur = -1;  // local bag being pooled (wave-uniform)

  auto store_row = [&](int bag, bool zero) {
    const uint64_t ro = readlane_u64(tl.row_off, bag) + c0 + lane;
    float div = 1.f;
    if (p.mean && !zero) div = static_cast<float>(readlane_u32(tl.len, bag));
#pragma unroll
    for (int r = 0; r < EPL; ++r) {
      if (act[r]) {
        const float x = zero ? 0.f : (p.mean ? acc[r] / div : acc[r]);
        store_out(out, ro + kWave * r, x, p.rows_bf16);
      }
    }
  };

  for (int64_t blk = tl.E0; blk < tl.E1; blk += kWave) {
    const int64_t rem = tl.E1 - blk;
    const int n = rem < kWave ? static_cast<int>(rem) : kWave;
    const int64_t e = blk + lane;
    uint32_t idx = 0;
    if (lane < n) idx = load_index(indices, e, p.idx32);
    const int bag = bag_of_item(tl, e);
    const uint32_t tC = __shfl(tl.tC, bag);
    if (TAB) fill_base_table<SIGN>(tab, item_hash(idx, tC, p.TC, p.a, p.b), p, lane);

    for (int q = 0; q < n; q += U) {
      // Gather phase: straight-line, U items x EPL loads in flight.  Items
      // past the end of the block re-read the last item (clamped index) and
      // inactive dims read element 0, so no load sits behind a branch.
      float v[U][EPL];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int uu = q + u < n ? q + u : n - 1;
        uint32_t h0 = 0, h20 = 0;
        if (!TAB) {
          h0 = item_hash(readlane_u32(idx, uu), readlane_u32(tC, uu), p.TC, p.a, p.b);
          if (SIGN) h20 = sign_hash0(h0, p.s_alpha, p.s_beta);
        }
#pragma unroll
        for (int r = 0; r < EPL; ++r) {
          const uint32_t ent =
              TAB ? tab[uu * kTabStride + jj[r]]
                  : chunk_entry<SIGN>(fast_mod(add_mod_p(h0, step[r]), p.fm_c, p.M),
                                      add_mod_p(h20, step2[r]), p);
          const Elem el = elem_of<SIGN>(ent, kk[r], p.M);
          const float x = load_weight(w, act[r] ? el.m : 0u);
          v[u][r] = SIGN ? apply_sign(x, el) : x;
        }
      }
      // Pool phase: stores only here, after every gather of the batch was
      // issued (a store counts in the same wait counter as the gathers).
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (q + u < n) {
          const int bg = static_cast<int>(readlane_u32(static_cast<uint32_t>(bag), q + u));
          if (bg != cur) {
            if (cur >= 0) store_row(cur, false);
            for (int z = cur + 1; z < bg; ++z) store_row(z, true);
            cur = bg;
#pragma unroll
            for (int r = 0; r < EPL; ++r) acc[r] = 0.f;
          }
#pragma unroll
          for (int r = 0; r < EPL; ++r) acc[r] += v[u][r];
        }
      }
    }
  }
  if (cur >= 0) store_row(cur, false);
  for (int z = cur + 1; z < tl.nb; ++z) store_row(z, true);
}

template <typename WT, int EPL, int U, bool TAB, bool SIGN>
static hipError_t launch_fwd_t(const WT* w, const KParams& p, const void* indices,
                               const void* offsets, void* out, hipStream_t stream) {
  const uint64_t tiles = (p.num_bags + kTileBags - 1) / kTileBags;
  const uint64_t blocks = (tiles + kWavesPerBlock - 1) / kWavesPerBlock;
  const uint32_t slabs = (p.d + kWave * EPL - 1) / (kWave * EPL);
  if (blocks > 0x7fffffffull - kXcds) return hipErrorInvalidConfiguration;
  const uint32_t xcd_split = static_cast<uint64_t>(p.M) * sizeof(WT) > kXcdSplitBytes ? 1u : 0u;
  // with the split, grid.x is rounded up to a multiple of kXcds (the extra
  // workgroups' tiles lie past the last bag: they exit at once)
  const uint64_t grid_x = xcd_split ? (blocks + kXcds - 1) / kXcds * kXcds : blocks;
  dim3 grid(static_cast<uint32_t>(grid_x), slabs);
  hipLaunchKernelGGL((forward_kernel<WT, EPL, U, TAB, SIGN>), grid, dim3(kBlockThreads), 0, stream,
                     w, p, indices, offsets, out, xcd_split);
  return hipGetLastError();
}

template <typename WT, bool TAB, bool SIGN>
static hipError_t launch_fwd_c(const WT* w, const KParams& p, const void* indices,
                               const void* offsets, void* out, hipStream_t stream) {
  if (p.d <= 64) return launch_fwd_t<WT, 1, 16, TAB, SIGN>(w, p, indices, offsets, out, stream);
  if (p.d <= 128) return launch_fwd_t<WT, 2, 8, TAB, SIGN>(w, p, indices, offsets, out, stream);
  if (p.d <= 256) return launch_fwd_t<WT, 4, 4, TAB, SIGN>(w, p, indices, offsets, out, stream);
  return launch_fwd_t<WT, 8, 2, TAB, SIGN>(w, p, indices, offsets, out, stream);
}

template <typename WT, bool SIGN>
static hipError_t launch_fwd_s(const WT* w, const KParams& p, const void* indices,
                               const void* offsets, void* out, hipStream_t stream) {
  if (p.C <= static_cast<uint32_t>(kTabChunks))
    return launch_fwd_c<WT, true, SIGN>(w, p, indices, offsets, out, stream);
  return launch_fwd_c<WT, false, SIGN>(w, p, indices, offsets, out, stream);
}

template <typename WT>
static hipError_t launch_fwd_w(const WT* w, const KParams& p, const void* indices,
                               const void* offsets, void* out, hipStream_t stream) {
  if (p.sign_mode) return launch_fwd_s<WT, true>(w, p, indices, offsets, out, stream);
  return launch_fwd_s<WT, false>(w, p, indices, offsets, out, stream);
}

hipError_t launch_forward(const void* w, bool bf16, const KParams& p, const void* indices,
                          const void* offsets, void* out, hipStream_t stream) {
  if (bf16)
    return launch_fwd_w(static_cast<const uint16_t*>(w), p, indices, offsets, out, stream);
  return launch_fwd_w(static_cast<const float*>(w), p, indices, offsets, out, stream);
}

}  // namespace pss
