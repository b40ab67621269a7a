// Forward of the PSS layer: hash -> chunk gather -> sum-pool (paper Sec. 2.4
// forward(i) = (S e_i)^T M with the ROBE-Z mapping of Sec. 2.5).
//
// Two kernels.  Batches of one item per bag with d in {64, 128, 256},
// Z % 4 == 0 and an array within the aggregate L2 take the streamed forward
// (end of this file), which writes the output in row order.  Every other
// batch takes the tiled kernel: one wavefront per tile of 64 bags of one
// table.  Hashing: with C = d/Z <= 16 chunks, each lane evaluates the C chunk
// bases of one item of the current 64-item block into a wave-private LDS
// table and the gathers read their base from it (one modular reduction per
// chunk instead of one per dim); with more chunks each lane hashes its own
// dims (item part on the scalar unit).  U items are gathered before any is
// consumed so that U * EPL loads per lane are in flight.  Pooling runs in registers in
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
#include <atomic>

#include "pss_keygen.hpp"
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

// ---------------------------------------------------------------------------
// Streamed forward for batches with one item per bag.
//
// HBM takes writes fastest when the stores in flight across the chip cover a
// narrow window of addresses that advances through the array; the tiled
// kernel above writes 512-byte row pieces spread over the whole output.  Here
// a persistent grid of one wavefront per SIMD writes the output in row order:
// at step s every wavefront stores one 1 KB unit (64 lanes x 4 elements: PPU =
// 256/d row pieces of d elements), and the units of one step lie within about
// 1 MB of rows.  Each lane gathers its 4 elements with one 16-byte load (a
// chunk of Z % 4 == 0 elements never splits a lane's 4 elements).
//
// Which pieces a wavefront takes (StreamMap): each XCD (workgroups are
// dispatched round-robin over the XCDs) owns a fixed share of the tables, so
// that its L2 holds the hot tokens of a few tables instead of all of them,
// while every XCD walks the rows at the same pace.
//
// Pipelining (loads and stores share one in-order wait counter on gfx9): a
// wavefront works in groups of D steps (32 for d >= 128, using all 64 lanes
// for the group's bags).  Three item sets rotate: while group n is stored and
// group n + 1 gathered, the offsets and index of group n + 3 are requested, so
// neither the index loads nor the gathers wait for a recent store.  Index and
// offset loads are ordinary (cached) loads: one 64-byte line of indices serves
// 8 rows of a table, which wavefronts of the same XCD read at about the same
// time.
//
// A bag that is not exactly one item at position offsets[g] == g (an empty
// bag, a bag of several items, or a permuted layout) is pooled by a slow path
// that walks its items; the fast path applies to every bag of a one-hot batch.
// ---------------------------------------------------------------------------
// Steps per group: D * PPU bags fit one wavefront's lanes.
template <int PPU> constexpr int stream_group() { return PPU >= 4 ? 16 : 32; }
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4u __attribute__((ext_vector_type(4), aligned(4)));  // 4-byte aligned
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

struct StreamItems {
  uint32_t idx;      // index of the bag's (speculated) item
  int64_t o0, o1;    // offsets[g], offsets[g + 1]
  uint32_t g;        // bag
  uint32_t t;        // its table
  uint32_t o4;       // first element of its row piece in out, / 4
  bool valid;        // lane holds a bag of the batch
};

// Placement of row pieces: the XCD groups (8 when the grid is a multiple of
// 8, else 1) each take a fixed share of the tables.  Rows go in periods of L
// rows (T*L divisible by the group count); the T*L pieces of a period, in
// table-major order, are split into equal runs of K, one run per group, so a
// group meets the same few tables throughout while all groups advance
// through the rows together.
struct StreamMap {
  uint32_t nw;   // wavefronts of this XCD group
  uint32_t w;    // this wavefront's rank in the group
  uint32_t x;    // the group
  uint32_t L;    // rows per period
  uint32_t K;    // pieces per group and period
  uint64_t Kx;   // pieces of the group: K * ceil(B / L)
};

template <bool I32>
__device__ __forceinline__ uint32_t load_index_cached(const void* idx, uint64_t e) {
  if constexpr (I32) return static_cast<uint32_t>(static_cast<const int32_t*>(idx)[e]);
  else return static_cast<uint32_t>(static_cast<const int64_t*>(idx)[e]);
}
template <bool I32>
__device__ __forceinline__ int64_t load_offset_cached(const void* off, uint64_t g) {
  if constexpr (I32) return static_cast<int64_t>(static_cast<const int32_t*>(off)[g]);
  else return static_cast<const int64_t*>(off)[g];
}

// Lane i < D * PPU requests the bag of group n's step i / PPU, row piece
// i % PPU of that step's unit.  Bags, and so row pieces, number fewer than
// 2^32; its piece's first output element is below 2^34 (o4 fits 32 bits).
template <int PPU, bool I32>
__device__ __forceinline__ void stream_items(StreamItems& it, const KParams& p,
                                             const void* __restrict__ indices,
                                             const void* __restrict__ offsets, uint64_t n,
                                             const StreamMap& sm, int lane) {
  constexpr int D = stream_group<PPU>();
  const uint64_t unit = (n * D + static_cast<uint64_t>(lane / PPU)) * sm.nw + sm.w;
  const uint64_t piece = unit * PPU + static_cast<uint64_t>(lane % PPU);
  bool valid = lane < D * PPU && piece < sm.Kx;
  const uint32_t pc = valid ? static_cast<uint32_t>(piece) : 0u;  // Kx < 2^32
  const uint32_t Q = pc / sm.K, k = pc - Q * sm.K;
  const uint32_t q = sm.x * sm.K + k;  // < T * L
  const uint32_t tq = q / sm.L;
  const uint32_t r = Q * sm.L + (q - tq * sm.L);
  valid = valid && r < p.B;
  it.valid = valid;
  it.t = valid ? tq : 0u;
  const uint32_t rr = valid ? r : 0u;
  it.g = it.t * p.B + rr;  // < T*B <= 2^32 - 1
  it.o4 = static_cast<uint32_t>(
      (static_cast<uint64_t>(rr) * p.row_stride + static_cast<uint64_t>(it.t) * p.d) >> 2);
  // out-of-batch lanes read bag 0 (offsets has T*B + 1 >= 2 entries)
  const uint32_t g = it.g;
  it.o0 = load_offset_cached<I32>(offsets, g);
  it.o1 = load_offset_cached<I32>(offsets, static_cast<uint64_t>(g) + 1);
  // the index of item g, which is the bag's item in a one-hot layout
  const uint64_t e = static_cast<int64_t>(g) < p.N ? g : 0u;
  it.idx = p.N > 0 ? load_index_cached<I32>(indices, e) : 0u;
}

// Elements kk .. kk+3 of the chunk of table entry `ent` (a chunk base, with
// the sign bits of chunk_entry when SIGN), widened to float and signed.  One
// 16-byte load (4-byte aligned) unless the 4 elements run past the end of
// the array, where each wraps on its own.
template <typename WT, bool SIGN>
__device__ __forceinline__ f32x4 gather4(const WT* __restrict__ w, uint32_t ent, uint32_t kk,
                                         uint32_t M) {
  bool read = true;
  uint32_t neg = 0, base = ent;
  if (SIGN) {
    read = ent != kSkip;
    neg = ent & 0x80000000u;
    base = read ? ent & 0x7fffffffu : 0u;
  }
  const uint32_t m = base + kk;  // < 2M <= 2^32
  const bool wrap = m + 3 >= M;
  const uint32_t mv = wrap ? 0u : m;  // M >= Z >= 4: elements 0..3 exist
  f32x4 x;
  if constexpr (sizeof(WT) == 4) {
    x = *reinterpret_cast<const f32x4u*>(reinterpret_cast<const float*>(w) + mv);
  } else {
    x = f32x4{load_weight(w, mv), load_weight(w, mv + 1), load_weight(w, mv + 2),
              load_weight(w, mv + 3)};
  }
  if (wrap) {
    x = f32x4{load_weight(w, wrap_add(base, kk, M)), load_weight(w, wrap_add(base, kk + 1, M)),
              load_weight(w, wrap_add(base, kk + 2, M)), load_weight(w, wrap_add(base, kk + 3, M))};
  }
  if (SIGN) {
    if (!read) return f32x4{0.f, 0.f, 0.f, 0.f};
    x = f32x4{__uint_as_float(__float_as_uint(x.x) ^ neg), __uint_as_float(__float_as_uint(x.y) ^ neg),
              __uint_as_float(__float_as_uint(x.z) ^ neg), __uint_as_float(__float_as_uint(x.w) ^ neg)};
  }
  return x;
}

// Chunk entry, for the lane's chunk (hash steps stepj, step2j), of the item
// whose item hash is h.
template <bool SIGN>
__device__ __forceinline__ uint32_t stream_entry(uint32_t h, uint32_t stepj, uint32_t step2j,
                                                 const KParams& p) {
  const uint32_t base = fast_mod(add_mod_p(h, stepj), p.fm_c, p.M);
  if (!SIGN) return base;
  return chunk_entry<SIGN>(base, add_mod_p(sign_hash0(h, p.s_alpha, p.s_beta), step2j), p);
}

// Item hash of the bag of step d, row piece pcl (hashed by lane d * PPU + pcl).
template <int PPU>
__device__ __forceinline__ uint32_t pick_hash(uint32_t h0, int d, uint32_t pcl) {
  uint32_t h = readlane_u32(h0, d * PPU);
#pragma unroll
  for (int q = 1; q < PPU; ++q) {
    const uint32_t hq = readlane_u32(h0, d * PPU + q);
    h = pcl == static_cast<uint32_t>(q) ? hq : h;
  }
  return h;
}

__device__ __forceinline__ int64_t readlane_i64(int64_t v, int lane) {
  const uint32_t lo = readlane_u32(static_cast<uint32_t>(v), lane);
  const uint32_t hi = readlane_u32(static_cast<uint32_t>(static_cast<uint64_t>(v) >> 32), lane);
  return static_cast<int64_t>((static_cast<uint64_t>(hi) << 32) | lo);
}

template <typename WT, int PPU, bool SIGN, bool I32>
__global__ __launch_bounds__(kBlockThreads) void forward_stream_kernel(
    const WT* __restrict__ w, const KParams p, const void* __restrict__ indices,
    const void* __restrict__ offsets, void* __restrict__ out, const uint32_t nx,
    const KeygenOut kg) {
  constexpr int D = stream_group<PPU>();
  const int lane = threadIdx.x & (kWave - 1);
  // Workgroups go round-robin to the XCDs (grid.x is a multiple of nx).
  StreamMap sm;
  sm.x = blockIdx.x % nx;
  sm.nw = (gridDim.x / nx) * kWavesPerBlock;
  sm.w = (blockIdx.x / nx) * kWavesPerBlock + (threadIdx.x >> 6);
  sm.L = 1;
  while ((p.T * sm.L) % nx != 0) ++sm.L;  // nx <= 8
  sm.K = p.T * sm.L / nx;
  sm.Kx = static_cast<uint64_t>(sm.K) * ((p.B + sm.L - 1) / sm.L);
  const uint64_t units = (sm.Kx + PPU - 1) / PPU;
  const uint64_t steps = (units + sm.nw - 1) / sm.nw;
  const uint64_t groups = (steps + D - 1) / D;

  // Prefetch.  Each group's index and offset entries (the contiguous range of
  // its tables) are read once, in whole 16-byte pieces lying inside the
  // arrays, before the loop: the loop's item loads then find them in the
  // caches instead of sending scattered reads to HBM in the middle of the
  // write stream.  In a training step (entries not cached after the
  // backward) this took the headline forward from 189 to 171 us.
  //
  // With kg (the backward's grouping prepared by this forward), the same
  // entries are read by the grouping's keygen instead (keygen_process: the
  // (h0, row) pairs and the first radix pass's digit counts of every sort
  // tile), which then serves as the prefetch.  XCD x's workgroups take the
  // contiguous x-th eighth of the sort tiles, about the tables it owns.
  uint32_t pf = 0;
  __shared__ KeygenLds kg_lds;
  if (kg.keys != nullptr) {
    const uint32_t per_x = (kg.nblocks + nx - 1) / nx;
    const uint32_t lo = sm.x * per_x;
    const uint32_t hi = lo + per_x < kg.nblocks ? lo + per_x : kg.nblocks;
    const uint32_t wgs = gridDim.x / nx, rank = blockIdx.x / nx;
    // the next tile's entries are requested before the current tile is
    // worked (two input sets take turns)
    KeygenIn ka, kb;
    uint32_t tile = lo + rank;
    if (tile < hi) keygen_load<I32, false>(p, indices, offsets, tile, ka);
    while (tile < hi) {
      const uint32_t t2 = tile + wgs;
      if (t2 < hi) keygen_load<I32, false>(p, indices, offsets, t2, kb);
      keygen_process<I32, false>(p, offsets, kg.keys, kg.rows, kg.inv_len, kg.counts, kg.nblocks,
                                 tile, ka, kg_lds);
      if (t2 >= hi) break;
      const uint32_t t3 = t2 + wgs;
      if (t3 < hi) keygen_load<I32, false>(p, indices, offsets, t3, ka);
      keygen_process<I32, false>(p, offsets, kg.keys, kg.rows, kg.inv_len, kg.counts, kg.nblocks,
                                 t2, kb, kg_lds);
      tile = t3;
    }
  } else {
    const uint64_t t_lo = static_cast<uint64_t>(sm.x) * sm.K / sm.L;
    const uint64_t t_hi = (static_cast<uint64_t>(sm.x + 1) * sm.K - 1) / sm.L + 1;  // <= T
    const uint64_t g_lo = t_lo * p.B, g_hi = t_hi * p.B;
    const uint64_t es = I32 ? 4 : 8;
    auto touch = [&](const void* base, uint64_t n_entries) {
      const uint64_t hi_e = g_hi < n_entries ? g_hi : n_entries;
      if (g_lo >= hi_e) return;
      const uint64_t a0 = reinterpret_cast<uint64_t>(base);
      const uint64_t c_lo = (a0 + g_lo * es + 15) / 16, c_end = (a0 + hi_e * es) / 16;
      // kPrefetchBatch 16-byte pieces per lane requested before any is used
      constexpr int kPrefetchBatch = 16;
      const uint64_t stride = static_cast<uint64_t>(sm.nw) * kWave;
      for (uint64_t c0 = c_lo + static_cast<uint64_t>(sm.w) * kWave + lane; c0 < c_end;
           c0 += kPrefetchBatch * stride) {
        uint4 v4[kPrefetchBatch];
#pragma unroll
        for (int k = 0; k < kPrefetchBatch; ++k) {
          const uint64_t c = c0 + k * stride;
          v4[k] = c < c_end ? *reinterpret_cast<const uint4*>(c * 16) : uint4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int k = 0; k < kPrefetchBatch; ++k) pf ^= v4[k].x ^ v4[k].y ^ v4[k].z ^ v4[k].w;
      }
    };
    touch(indices, static_cast<uint64_t>(p.N));
    touch(offsets, p.num_bags + 1);
  }

  // lane's 4 elements: row piece pcl of the unit, dims c .. c+3 of it
  constexpr uint32_t kLanesPerPiece = kWave / PPU;
  const uint32_t pcl = static_cast<uint32_t>(lane) / kLanesPerPiece;
  const uint32_t c = (static_cast<uint32_t>(lane) % kLanesPerPiece) * 4;
  const uint32_t j = c / p.Z, kk = c - j * p.Z;
  const uint32_t stepj = chunk_step(p.a, j);
  const uint32_t step2j = SIGN ? chunk_step(p.a2, j) : 0u;

  auto hash_of = [&](const StreamItems& it) -> uint32_t {
    return item_hash(it.idx, it.t * p.C, p.TC, p.a, p.b);
  };
  // bags of a group that are not one item at position g
  auto slow_of = [&](const StreamItems& it) -> uint64_t {
    const bool fast = it.o0 == static_cast<int64_t>(it.g) &&
                      it.o1 == static_cast<int64_t>(it.g) + 1 && static_cast<int64_t>(it.g) < p.N;
    return __ballot(it.valid && !fast);
  };
  f32x4 v[D];
  // Pools each listed bag of a group over its items (all lanes of its row
  // piece), in place of the speculative gather.
  auto fixup = [&](uint64_t slow, const StreamItems& it) {
    while (slow) {
      const int i = __builtin_ctzll(slow);
      slow &= slow - 1;
      const int64_t o0 = readlane_i64(it.o0, i), o1 = readlane_i64(it.o1, i);
      const uint32_t tC = readlane_u32(it.t, i) * p.C;
      const int64_t e0 = o0 < 0 ? 0 : (o0 > p.N ? p.N : o0);
      int64_t e1 = o1 < 0 ? 0 : (o1 > p.N ? p.N : o1);
      if (e1 < e0) e1 = e0;
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      for (int64_t e = e0; e < e1; ++e) {
        const uint32_t h =
            item_hash(load_index_cached<I32>(indices, static_cast<uint64_t>(e)), tC, p.TC, p.a, p.b);
        acc += gather4<WT, SIGN>(w, stream_entry<SIGN>(h, stepj, step2j, p), kk, p.M);
      }
      if (p.mean && e1 > e0) acc /= static_cast<float>(e1 - e0);
      const int si = i / PPU;
      const uint32_t pi = static_cast<uint32_t>(i % PPU);
#pragma unroll
      for (int d = 0; d < D; ++d)
        if (d == si && pcl == pi) v[d] = acc;
    }
  };
  // Stores group n (in v; piece offsets o4n, valid pieces vm) and gathers
  // group n + 1 (item hashes hn) into v.
  auto store_gather = [&](uint32_t hn, uint32_t o4n, uint64_t vm) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const uint64_t e = static_cast<uint64_t>(pick_hash<PPU>(o4n, d, pcl)) * 4 + c;
      if ((vm >> (d * PPU + pcl)) & 1u) {
        if (p.rows_bf16) {
          const u32x2 x = {static_cast<uint32_t>(f32_to_bf16_rne(v[d].x)) |
                               (static_cast<uint32_t>(f32_to_bf16_rne(v[d].y)) << 16),
                           static_cast<uint32_t>(f32_to_bf16_rne(v[d].z)) |
                               (static_cast<uint32_t>(f32_to_bf16_rne(v[d].w)) << 16)};
          __builtin_nontemporal_store(x, reinterpret_cast<u32x2*>(static_cast<uint16_t*>(out) + e));
        } else {
          __builtin_nontemporal_store(v[d], reinterpret_cast<f32x4*>(static_cast<float*>(out) + e));
        }
      }
      v[d] = gather4<WT, SIGN>(w, stream_entry<SIGN>(pick_hash<PPU>(hn, d, pcl), stepj, step2j, p),
                               kk, p.M);
    }
  };

  // Three item sets take turns (no register copies of values still loading):
  // while group n is stored, one set holds group n's items (for the slow path
  // and the store addresses), the next group n + 1's, which are hashed, and
  // the third group n + 2's, still loading; then the first is refilled with
  // group n + 3.
  StreamItems A, B, C;
  stream_items<PPU, I32>(A, p, indices, offsets, 0, sm, lane);
  uint64_t slow = slow_of(A);
  {
    const uint32_t h = hash_of(A);
#pragma unroll
    for (int d = 0; d < D; ++d)
      v[d] = gather4<WT, SIGN>(w, stream_entry<SIGN>(pick_hash<PPU>(h, d, pcl), stepj, step2j, p),
                               kk, p.M);
  }
  stream_items<PPU, I32>(B, p, indices, offsets, 1, sm, lane);
  stream_items<PPU, I32>(C, p, indices, offsets, 2, sm, lane);
  for (uint64_t n = 0; n < groups; n += 3) {
    fixup(slow, A);
    slow = slow_of(B);
    uint32_t h = hash_of(B);
    const uint32_t o4A = A.o4;
    const uint64_t vmA = __ballot(A.valid);
    stream_items<PPU, I32>(A, p, indices, offsets, n + 3, sm, lane);
    store_gather(h, o4A, vmA);
    if (n + 1 >= groups) break;
    fixup(slow, B);
    slow = slow_of(C);
    h = hash_of(C);
    const uint32_t o4B = B.o4;
    const uint64_t vmB = __ballot(B.valid);
    stream_items<PPU, I32>(B, p, indices, offsets, n + 4, sm, lane);
    store_gather(h, o4B, vmB);
    if (n + 2 >= groups) break;
    fixup(slow, C);
    slow = slow_of(A);
    h = hash_of(A);
    const uint32_t o4C = C.o4;
    const uint64_t vmC = __ballot(C.valid);
    stream_items<PPU, I32>(C, p, indices, offsets, n + 5, sm, lane);
    store_gather(h, o4C, vmC);
  }
  // never true (N >= 0): keeps the prefetch loads
  if (pf == 0x9e3779b9u && p.N < 0) static_cast<uint32_t*>(out)[lane] = pf;
}

// The streamed forward applies when the batch has as many items as bags
// (every bag may then be one item; others take the slow path), a lane's 4
// elements lie in one chunk (Z % 4 == 0) and a 256-element unit holds whole
// row pieces (d in {64, 128, 256}).  It is used for shared arrays that fit
// the chip's aggregate L2; larger arrays keep the tiled kernel, whose tiles
// partition the tables over the XCDs.  Measured on the 26-table one-hot batch
// (65 536 samples, d = 128, 10 MB array), per launch: 172 us after another
// forward and 187 us in a training step, against 200 us for the tiled kernel
// (which gathers each distinct token of a tile once, but writes at about
// 5.1 TB/s in its pattern).
template <typename WT>
static bool stream_applies(const KParams& p) {
  return static_cast<uint64_t>(p.N) == p.num_bags && p.Z % 4 == 0 &&
         (p.d == 64 || p.d == 128 || p.d == 256) &&
         static_cast<uint64_t>(p.M) * sizeof(WT) <= kXcdSplitBytes &&
         p.num_bags * p.d < (1ull << 34);
}

// Compute units of each device, looked up once per device (callers may run
// on several threads and devices).
constexpr int kMaxDevices = 64;
static std::atomic<int> g_cus[kMaxDevices];

static int device_cus() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return 256;
  }
  int n = g_cus[dev].load(std::memory_order_relaxed);
  if (n <= 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n <= 0) {
      (void)hipGetLastError();
      n = 256;
    }
    g_cus[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

// Wavefronts of the streamed forward: one per SIMD (4 per compute unit).
static uint32_t stream_blocks(uint64_t units) {
  const uint64_t cus = static_cast<uint64_t>(device_cus());
  const uint64_t want = (units + kWavesPerBlock - 1) / kWavesPerBlock;
  uint64_t blocks = want < cus ? want : cus;
  if (blocks >= kXcds) blocks = blocks / kXcds * kXcds;
  return static_cast<uint32_t>(blocks < 1 ? 1 : blocks);
}

template <typename WT, int PPU, bool SIGN>
static hipError_t launch_stream_t(const WT* w, const KParams& p, const void* indices,
                                  const void* offsets, void* out, hipStream_t stream,
                                  const KeygenOut& kg) {
  const uint64_t units = (p.num_bags * p.d + kWave * 4 - 1) / (kWave * 4);
  const uint32_t blocks = stream_blocks(units);
  const uint32_t nx = blocks % kXcds == 0 ? kXcds : 1u;
  if (p.idx32)
    hipLaunchKernelGGL((forward_stream_kernel<WT, PPU, SIGN, true>), dim3(blocks),
                       dim3(kBlockThreads), 0, stream, w, p, indices, offsets, out, nx, kg);
  else
    hipLaunchKernelGGL((forward_stream_kernel<WT, PPU, SIGN, false>), dim3(blocks),
                       dim3(kBlockThreads), 0, stream, w, p, indices, offsets, out, nx, kg);
  return hipGetLastError();
}

template <typename WT, bool SIGN>
static hipError_t launch_stream_s(const WT* w, const KParams& p, const void* indices,
                                  const void* offsets, void* out, hipStream_t stream,
                                  const KeygenOut& kg) {
  if (p.d == 64) return launch_stream_t<WT, 4, SIGN>(w, p, indices, offsets, out, stream, kg);
  if (p.d == 128) return launch_stream_t<WT, 2, SIGN>(w, p, indices, offsets, out, stream, kg);
  return launch_stream_t<WT, 1, SIGN>(w, p, indices, offsets, out, stream, kg);
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
                               const void* offsets, void* out, hipStream_t stream,
                               const KeygenOut* kg) {
  if (stream_applies<WT>(p)) {
    const KeygenOut none{};
    const KeygenOut& k = kg != nullptr ? *kg : none;
    if (p.sign_mode) return launch_stream_s<WT, true>(w, p, indices, offsets, out, stream, k);
    return launch_stream_s<WT, false>(w, p, indices, offsets, out, stream, k);
  }
  if (kg != nullptr) return hipErrorInvalidValue;  // only the streamed kernel writes a keygen
  if (p.sign_mode) return launch_fwd_s<WT, true>(w, p, indices, offsets, out, stream);
  return launch_fwd_s<WT, false>(w, p, indices, offsets, out, stream);
}

bool forward_streams(const KParams& p, bool bf16) {
  return bf16 ? stream_applies<uint16_t>(p) : stream_applies<float>(p);
}

hipError_t launch_forward(const void* w, bool bf16, const KParams& p, const void* indices,
                          const void* offsets, void* out, hipStream_t stream,
                          const KeygenOut* kg) {
  if (bf16)
    return launch_fwd_w(static_cast<const uint16_t*>(w), p, indices, offsets, out, stream, kg);
  return launch_fwd_w(static_cast<const float*>(w), p, indices, offsets, out, stream, kg);
}

}  // namespace pss
