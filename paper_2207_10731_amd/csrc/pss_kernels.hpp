// Shared pieces of the PSS kernels: launch parameters, the per-wavefront bag
// tile, storage-type loads/stores.
//
// Work decomposition (forward and backward alike).  Bags are cut into tiles
// of kTileBags consecutive bags (g = t*B + b, table-major); one wavefront owns
// a tile.  Lane l holds the start offset of bag l of the tile; the tile's
// items form one contiguous range of `indices`, which the wave walks in
// blocks of 64 (one index per lane, one coalesced load).  For every item the
// wave evaluates the hash (the item part is wave-uniform, the chunk part is a
// per-lane constant) and touches the d embedding elements of the item with
// lanes spread over the dims: lane l owns dims c = c0 + l + 64 r.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pss_hash.hpp"

namespace pss {

constexpr int kWave = 64;
constexpr int kTileBags = 64;     // bags per wavefront tile
constexpr int kBlockThreads = 256;  // 4 wavefronts per workgroup
constexpr int kWavesPerBlock = kBlockThreads / kWave;
constexpr uint64_t kXcds = 8;  // XCDs of an MI355X, each with an L2 of its own

struct KParams {
  uint64_t fm_c;      // fast-mod constant of M
  uint64_t num_bags;  // T*B
  int64_t N;          // number of items
  uint32_t M;
  uint32_t a, b;
  uint32_t T, B;
  uint32_t C, Z, d;
  uint32_t TC;        // T*C (< 2^32)
  uint32_t row_stride;  // T*d: elements per pooled row
  // Options (pss_hash_params.flags).  sign_mode 0 = no sign; otherwise the
  // chunk sign comes from h2_0 = (s_alpha * h_0 + s_beta) mod p plus
  // a2 * j (mod p) for chunk j.
  uint32_t sign_mode, s_alpha, s_beta, a2;
  uint32_t mean;       // 1: mean pooling (each item weighs 1/|bag|)
  uint32_t idx32;      // 1: indices and offsets are int32
  uint32_t rows_bf16;  // 1: out / grad_out rows are bfloat16
};

// indices[e] / offsets[g] in either integer width (wave-uniform choice).
__device__ __forceinline__ uint32_t load_index(const void* idx, int64_t e, uint32_t i32) {
  return i32 ? static_cast<uint32_t>(
                   __builtin_nontemporal_load(static_cast<const int32_t*>(idx) + e))
             : static_cast<uint32_t>(
                   __builtin_nontemporal_load(static_cast<const int64_t*>(idx) + e));
}
__device__ __forceinline__ int64_t load_offset(const void* off, uint64_t g, uint32_t i32) {
  return i32 ? static_cast<int64_t>(
                   __builtin_nontemporal_load(static_cast<const int32_t*>(off) + g))
             : __builtin_nontemporal_load(static_cast<const int64_t*>(off) + g);
}

// bfloat16 bits <-> float
__device__ __forceinline__ float bf16_to_f32(uint16_t v) {
  return __uint_as_float(static_cast<uint32_t>(v) << 16);
}

// Round to nearest, ties to even; NaN stays a (quiet) NaN.
PSS_HD uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  __builtin_memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// Gradient rows: float32 or bfloat16 bits, widened exactly.
template <typename GT>
__device__ __forceinline__ float load_row(const GT* g, uint64_t k);
template <>
__device__ __forceinline__ float load_row<float>(const float* g, uint64_t k) {
  return __builtin_nontemporal_load(g + k);
}
template <>
__device__ __forceinline__ float load_row<uint16_t>(const uint16_t* g, uint64_t k) {
  return __uint_as_float(static_cast<uint32_t>(__builtin_nontemporal_load(g + k)) << 16);
}

template <typename WT>
__device__ __forceinline__ float load_weight(const WT* w, uint32_t m);

template <>
__device__ __forceinline__ float load_weight<float>(const float* w, uint32_t m) {
  return w[m];
}

template <>
__device__ __forceinline__ float load_weight<uint16_t>(const uint16_t* w, uint32_t m) {
  return bf16_to_f32(w[m]);
}

template <typename WT>
__device__ __forceinline__ void store_weight(WT* w, int64_t m, float v);
template <>
__device__ __forceinline__ void store_weight<float>(float* w, int64_t m, float v) {
  w[m] = v;
}
template <>
__device__ __forceinline__ void store_weight<uint16_t>(uint16_t* w, int64_t m, float v) {
  w[m] = f32_to_bf16_rne(v);
}
template <typename WT>
__device__ __forceinline__ float load_weight64(const WT* w, int64_t m);
template <>
__device__ __forceinline__ float load_weight64<float>(const float* w, int64_t m) {
  return w[m];
}
template <>
__device__ __forceinline__ float load_weight64<uint16_t>(const uint16_t* w, int64_t m) {
  return bf16_to_f32(w[m]);
}

// One element's update from its gradient sum g (g != 0): SGD w -= lr * g, or
// Adagrad s += g^2, w -= lr * g / (sqrt(s) + eps); float32 arithmetic,
// bfloat16 storage widened exactly and rounded once.
// The same with the element's weight (widened) and state already loaded;
// with NT_STATE the new state is stored non-temporally.
template <typename WT, bool ADAGRAD, bool NT_STATE = false>
__device__ __forceinline__ void update_loaded(WT* w, float* s, int64_t m, float g, float w_old,
                                              float s_old, float lr, float eps) {
  float upd;
  if (ADAGRAD) {
    const float sn = s_old + g * g;
    if (NT_STATE)
      __builtin_nontemporal_store(sn, s + m);
    else
      s[m] = sn;
    upd = lr * g / (sqrtf(sn) + eps);
  } else {
    upd = lr * g;
  }
  store_weight(w, m, w_old - upd);
}
template <typename WT, bool ADAGRAD>
__device__ __forceinline__ void apply_update(WT* w, float* s, int64_t m, float g, float lr,
                                             float eps) {
  update_loaded<WT, ADAGRAD>(w, s, m, g, load_weight64(w, m), ADAGRAD ? s[m] : 0.f, lr, eps);
}

__device__ __forceinline__ uint32_t readlane_u32(uint32_t v, int lane) {
  return static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(v), lane));
}

// Per-wavefront view of one tile of bags.
struct Tile {
  uint64_t g0;        // first bag
  int nb;             // bags in the tile (1..kTileBags)
  int64_t E0, E1;     // item range [E0, E1) of the tile (clamped to [0, N])
  int64_t start;      // lane l: first item of bag g0 + l (clamped, monotone)
  uint32_t tC;        // lane l: t * C of bag g0 + l
  uint64_t row_off;   // lane l: b * T*d + t*d of bag g0 + l
  uint32_t len;       // lane l: number of items of bag g0 + l
};

// Loads the tile's offsets (one coalesced load) and per-bag constants.
// Offsets are clamped to [0, N] and made monotone within the tile, so item
// ranges never leave `indices` whatever the offsets array holds.
__device__ __forceinline__ Tile load_tile(const KParams& p, const void* __restrict__ offsets,
                                          uint64_t g0, int lane) {
  Tile tl;
  tl.g0 = g0;
  const uint64_t left = p.num_bags - g0;
  tl.nb = left < static_cast<uint64_t>(kTileBags) ? static_cast<int>(left) : kTileBags;
  int64_t s = 0;
  if (lane < tl.nb) s = load_offset(offsets, g0 + lane, p.idx32);
  int64_t e_last = load_offset(offsets, g0 + tl.nb, p.idx32);
  s = s < 0 ? 0 : (s > p.N ? p.N : s);
  e_last = e_last < 0 ? 0 : (e_last > p.N ? p.N : e_last);
  // running max over lanes keeps starts monotone (inclusive scan of max)
  for (int sh = 1; sh < kWave; sh <<= 1) {
    const int64_t o = __shfl_up(s, sh);
    if (lane >= sh && o > s) s = o;
  }
  if (lane >= tl.nb) s = INT64_MAX;  // sentinel: no bag
  tl.start = s;
  const int64_t first = __shfl(s, 0);
  // largest start among real bags = start of bag nb-1
  const int64_t last_start = __shfl(s, tl.nb - 1);
  tl.E0 = first;
  tl.E1 = e_last < last_start ? last_start : e_last;
  // items of bag g0 + lane: [start, next start) (the last bag ends at E1)
  const int64_t nxt = __shfl_down(s, 1);
  tl.len = lane < tl.nb ? static_cast<uint32_t>((lane == tl.nb - 1 ? tl.E1 : nxt) - s) : 0u;
  const uint64_t g = g0 + static_cast<uint64_t>(lane < tl.nb ? lane : 0);
  const uint32_t t = static_cast<uint32_t>(g / p.B);
  const uint32_t b = static_cast<uint32_t>(g - static_cast<uint64_t>(t) * p.B);
  tl.tC = t * p.C;
  tl.row_off = static_cast<uint64_t>(b) * p.row_stride + static_cast<uint64_t>(t) * p.d;
  return tl;
}

// Chunk-base table.  For C = d/Z <= kTabChunks, lane l of a wavefront
// evaluates the C chunk bases of item l of the current 64-item block once
// (the modular reduction by M costs quarter-rate 64-bit multiplies) and keeps
// them in a wave-private LDS table; every lane then reads the base of the
// chunk it needs with a broadcast LDS read.  Wider C (small Z) hashes per lane.
constexpr int kTabChunks = 16;
constexpr int kTabStride = kTabChunks + 1;  // padding against bank conflicts

//
// With a chunk sign the entry also carries it: base | 2^31 for -1, and
// kSkip for a chunk that is not read (bases are below M <= 2^31 - 1, so
// neither collides with a plain base).
constexpr uint32_t kSkip = 0xffffffffu;

template <bool SIGN>
__device__ __forceinline__ uint32_t chunk_entry(uint32_t base, uint32_t h2, const KParams& p) {
  if (!SIGN) return base;
  const uint32_t code = sign_code(h2, p.sign_mode);
  return code == 2u ? kSkip : base | (code << 31);
}

template <bool SIGN>
__device__ __forceinline__ void fill_base_table(uint32_t* tab, uint32_t h0, const KParams& p,
                                                int lane) {
  uint32_t step = 0;  // a * j mod p, j = 0 .. C-1
  uint32_t h2 = SIGN ? sign_hash0(h0, p.s_alpha, p.s_beta) : 0u;
  for (uint32_t j = 0; j < p.C; ++j) {
    tab[lane * kTabStride + j] =
        chunk_entry<SIGN>(fast_mod(add_mod_p(h0, step), p.fm_c, p.M), h2, p);
    step = add_mod_p(step, p.a);
    if (SIGN) h2 = add_mod_p(h2, p.a2);
  }
}

// Element k of the chunk of table entry `ent`: its address (0 for a chunk
// that is not read, so the load stays in bounds) and the float sign mask.
struct Elem {
  uint32_t m, neg;
  bool read;
};
template <bool SIGN>
__device__ __forceinline__ Elem elem_of(uint32_t ent, uint32_t k, uint32_t M) {
  Elem e;
  if (!SIGN) {
    e.m = wrap_add(ent, k, M);
    e.neg = 0;
    e.read = true;
    return e;
  }
  e.read = ent != kSkip;
  e.neg = ent & 0x80000000u;
  e.m = e.read ? wrap_add(ent & 0x7fffffffu, k, M) : 0u;
  return e;
}

// x * (+1 or -1) by flipping the sign bit; a chunk that is not read gives 0.
__device__ __forceinline__ float apply_sign(float x, const Elem& e) {
  return e.read ? __uint_as_float(__float_as_uint(x) ^ e.neg) : 0.f;
}

// Bitonic sort of one (key, payload) pair per lane across the 64 lanes of a
// wavefront, ascending by key (ties keep no particular order).
__device__ __forceinline__ void wave_sort_pairs(uint32_t& key, uint32_t& val, int lane) {
#pragma unroll
  for (int k = 2; k <= kWave; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      const uint32_t ok = __shfl_xor(key, j);
      const uint32_t ov = __shfl_xor(val, j);
      const bool up = (lane & k) == 0;
      const bool lower = (lane & j) == 0;
      // the lower lane of an ascending pair keeps the smaller key
      const bool take = lower == up ? ok < key : ok > key;
      if (take) {
        key = ok;
        val = ov;
      }
    }
  }
}

// Exclusive scan over the 256 threads of a block (wave scans + LDS carry).
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* wsum,
                                                         uint32_t* total) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & (kWave - 1);
  uint32_t x = v;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const uint32_t y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  if (lane == kWave - 1) wsum[w] = x;
  __syncthreads();
  uint32_t before = 0, all = 0;
#pragma unroll
  for (int ww = 0; ww < kWavesPerBlock; ++ww) {
    before += ww < w ? wsum[ww] : 0u;
    all += wsum[ww];
  }
  __syncthreads();
  *total = all;
  return before + x - v;
}

// Local bag (0..nb-1) of item e of the tile: the largest l with start[l] <= e.
// Binary search over the starts held in the lanes (6 cross-lane reads).
__device__ __forceinline__ int bag_of_item(const Tile& tl, int64_t e) {
  int lo = 0;
  for (int step = kWave / 2; step >= 1; step >>= 1) {
    const int probe = lo + step;
    const int64_t sp = __shfl(tl.start, probe < kWave ? probe : kWave - 1);
    if (probe < tl.nb && sp <= e) lo = probe;
  }
  return lo;
}

}  // namespace pss
