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
#include "pss_launch.hpp"

namespace pss {

__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int lane) {
  const uint32_t lo = readlane_u32(static_cast<uint32_t>(v), lane);
  const uint32_t hi = readlane_u32(static_cast<uint32_t>(v >> 32), lane);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

// One-hot tile: item l of the tile is bag l.  The (h0, bag) pairs are sorted
// across the lanes; every run of equal h0 is one token, gathered once (U runs
// in flight) and stored to the rows of all its bags.
template <typename WT, int EPL, int U>
__device__ __forceinline__ void forward_onehot_tile(
    const WT* __restrict__ w, const KParams& p, const Tile& tl,
    const int64_t* __restrict__ indices, float* __restrict__ out, uint32_t* tab, int lane,
    uint32_t c0, const uint32_t* jj, const uint32_t* kk, const bool* act) {
  const int nb = tl.nb;
  uint32_t key = 0xffffffffu;  // empty lanes sort last
  uint32_t bag = static_cast<uint32_t>(lane);
  if (lane < nb) {
    const uint32_t i = static_cast<uint32_t>(__builtin_nontemporal_load(indices + tl.E0 + lane));
    key = item_hash(i, tl.tC, p.TC, p.a, p.b);
  }
  wave_sort_pairs(key, bag, lane);
  fill_base_table(tab, key, p, lane);
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
        const uint32_t m = act[r] ? wrap_add(tab[pu * kTabStride + jj[r]], kk[r], p.M) : 0u;
        v[u][r] = load_weight(w, m);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      for (int q = pos[u]; q < pos[u + 1]; ++q) {
        const int b = static_cast<int>(readlane_u32(bag, q));
        const uint64_t ro = readlane_u64(tl.row_off, b) + c0 + lane;
#pragma unroll
        for (int r = 0; r < EPL; ++r)
          if (act[r]) __builtin_nontemporal_store(v[u][r], out + ro + kWave * r);
      }
    }
  }
}

template <typename WT, int EPL, int U, bool TAB>
__global__ __launch_bounds__(kBlockThreads) void forward_kernel(
    const WT* __restrict__ w, const KParams p, const int64_t* __restrict__ indices,
    const int64_t* __restrict__ offsets, float* __restrict__ out) {
  const int lane = threadIdx.x & (kWave - 1);
  const uint64_t wave = static_cast<uint64_t>(blockIdx.x) * kWavesPerBlock + (threadIdx.x >> 6);
  const uint64_t g0 = wave * kTileBags;
  if (g0 >= p.num_bags) return;
  const uint32_t c0 = blockIdx.y * (kWave * EPL);

  __shared__ uint32_t tab_all[TAB ? kWavesPerBlock * kWave * kTabStride : 1];
  uint32_t* tab = tab_all + (TAB ? (threadIdx.x >> 6) * kWave * kTabStride : 0);

  uint32_t step[EPL], kk[EPL], jj[EPL];
  bool act[EPL];
#pragma unroll
  for (int r = 0; r < EPL; ++r) {
    const uint32_t c = c0 + lane + kWave * r;
    act[r] = c < p.d;
    const uint32_t cc = act[r] ? c : 0;
    jj[r] = cc / p.Z;
    kk[r] = cc - jj[r] * p.Z;
    step[r] = TAB ? 0u : chunk_step(p.a, jj[r]);
  }

  const Tile tl = load_tile(p, offsets, g0, lane);

  if (TAB) {
    // One-hot tile (every bag exactly one item): gather each distinct token
    // of the tile once and store its row to every bag that reads it.
    const int64_t nxt = __shfl_down(tl.start, 1);
    const int64_t end = lane == tl.nb - 1 ? tl.E1 : nxt;
    if (__ballot(lane >= tl.nb || end - tl.start == 1) == ~0ull) {
      forward_onehot_tile<WT, EPL, U>(w, p, tl, indices, out, tab, lane, c0, jj, kk, act);
      return;
    }
  }

  float acc[EPL];
#pragma unroll
  for (int r = 0; r < EPL; ++r) acc[r] = 0.f;
  int cur = -1;  // local bag being pooled (wave-uniform)

  auto store_row = [&](int bag, bool zero) {
    const uint64_t ro = readlane_u64(tl.row_off, bag) + c0 + lane;
#pragma unroll
    for (int r = 0; r < EPL; ++r)
      if (act[r]) __builtin_nontemporal_store(zero ? 0.f : acc[r], out + ro + kWave * r);
  };

  for (int64_t blk = tl.E0; blk < tl.E1; blk += kWave) {
    const int64_t rem = tl.E1 - blk;
    const int n = rem < kWave ? static_cast<int>(rem) : kWave;
    const int64_t e = blk + lane;
    uint32_t idx = 0;
    if (lane < n) idx = static_cast<uint32_t>(__builtin_nontemporal_load(indices + e));
    const int bag = bag_of_item(tl, e);
    const uint32_t tC = __shfl(tl.tC, bag);
    if (TAB) fill_base_table(tab, item_hash(idx, tC, p.TC, p.a, p.b), p, lane);

    for (int q = 0; q < n; q += U) {
      // Gather phase: straight-line, U items x EPL loads in flight.  Items
      // past the end of the block re-read the last item (clamped index) and
      // inactive dims read element 0, so no load sits behind a branch.
      float v[U][EPL];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int uu = q + u < n ? q + u : n - 1;
        uint32_t h0 = 0;
        if (!TAB) h0 = item_hash(readlane_u32(idx, uu), readlane_u32(tC, uu), p.TC, p.a, p.b);
#pragma unroll
        for (int r = 0; r < EPL; ++r) {
          const uint32_t base = TAB ? tab[uu * kTabStride + jj[r]]
                                    : fast_mod(add_mod_p(h0, step[r]), p.fm_c, p.M);
          const uint32_t m = act[r] ? wrap_add(base, kk[r], p.M) : 0u;
          v[u][r] = load_weight(w, m);
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

template <typename WT, int EPL, int U, bool TAB>
static hipError_t launch_fwd_t(const WT* w, const KParams& p, const int64_t* indices,
                               const int64_t* offsets, float* out, hipStream_t stream) {
  const uint64_t tiles = (p.num_bags + kTileBags - 1) / kTileBags;
  const uint64_t blocks = (tiles + kWavesPerBlock - 1) / kWavesPerBlock;
  const uint32_t slabs = (p.d + kWave * EPL - 1) / (kWave * EPL);
  if (blocks > 0x7fffffffull) return hipErrorInvalidConfiguration;
  dim3 grid(static_cast<uint32_t>(blocks), slabs);
  hipLaunchKernelGGL((forward_kernel<WT, EPL, U, TAB>), grid, dim3(kBlockThreads), 0, stream, w, p,
                     indices, offsets, out);
  return hipGetLastError();
}

template <typename WT, bool TAB>
static hipError_t launch_fwd_c(const WT* w, const KParams& p, const int64_t* indices,
                               const int64_t* offsets, float* out, hipStream_t stream) {
  if (p.d <= 64) return launch_fwd_t<WT, 1, 16, TAB>(w, p, indices, offsets, out, stream);
  if (p.d <= 128) return launch_fwd_t<WT, 2, 8, TAB>(w, p, indices, offsets, out, stream);
  if (p.d <= 256) return launch_fwd_t<WT, 4, 4, TAB>(w, p, indices, offsets, out, stream);
  return launch_fwd_t<WT, 8, 2, TAB>(w, p, indices, offsets, out, stream);
}

template <typename WT>
static hipError_t launch_fwd_w(const WT* w, const KParams& p, const int64_t* indices,
                               const int64_t* offsets, float* out, hipStream_t stream) {
  if (p.C <= static_cast<uint32_t>(kTabChunks))
    return launch_fwd_c<WT, true>(w, p, indices, offsets, out, stream);
  return launch_fwd_c<WT, false>(w, p, indices, offsets, out, stream);
}

hipError_t launch_forward(const void* w, bool bf16, const KParams& p, const int64_t* indices,
                          const int64_t* offsets, float* out, hipStream_t stream) {
  if (bf16)
    return launch_fwd_w(static_cast<const uint16_t*>(w), p, indices, offsets, out, stream);
  return launch_fwd_w(static_cast<const float*>(w), p, indices, offsets, out, stream);
}

}  // namespace pss
