// Backward of the PSS layer (paper Sec. 2.4 backward(i, Delta) = (S e_i) Delta;
// Alg. 1 dense branch: the gradient of the flat array is the scatter-add of
// the output gradient onto the addresses that were read) and the optimizer
// step.
//
// deposit_kernel walks the same bag tiles as the forward.  For each item it
// reads the bag's gradient row (non-temporal: read once) and adds
// scale * grad into dst at the item's hashed addresses with hardware float
// atomics (global_atomic_add_f32, no return value).  With mean pooling the
// row is divided by the bag's item count; with a chunk sign the value is
// negated for -1 chunks and chunks of factor 0 receive nothing.  With SGD on float32
// storage dst is the shared array itself and scale = -lr (the update is
// linear in G, so it fuses into the deposit).  Otherwise dst is a float32
// gradient buffer and optimizer_kernel applies SGD or Adagrad per element.
#include "pss_launch.hpp"

namespace pss {

__device__ __forceinline__ float readlane_f32(float v, int lane) {
  return __uint_as_float(readlane_u32(__float_as_uint(v), lane));
}

__device__ __forceinline__ uint64_t readlane_u64b(uint64_t v, int lane) {
  const uint32_t lo = readlane_u32(static_cast<uint32_t>(v), lane);
  const uint32_t hi = readlane_u32(static_cast<uint32_t>(v >> 32), lane);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

template <int EPL, int U, bool TAB, bool SIGN, typename GT>
__global__ __launch_bounds__(kBlockThreads) void deposit_kernel(
    float* __restrict__ dst, const float scale, const KParams p,
    const void* __restrict__ indices, const void* __restrict__ offsets,
    const GT* __restrict__ grad) {
  const int lane = threadIdx.x & (kWave - 1);
  const uint64_t wave = static_cast<uint64_t>(blockIdx.x) * kWavesPerBlock + (threadIdx.x >> 6);
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

  const Tile tl = load_tile(p, offsets, g0, lane);
  // per-bag factor of the deposit: scale, or scale / |bag| for mean pooling
  const float bag_scale = p.mean && tl.len ? scale / static_cast<float>(tl.len) : scale;

  for (int64_t blk = tl.E0; blk < tl.E1; blk += kWave) {
    const int64_t rem = tl.E1 - blk;
    const int n = rem < kWave ? static_cast<int>(rem) : kWave;
    const int64_t e = blk + lane;
    uint32_t idx = 0;
    if (lane < n) idx = load_index(indices, e, p.idx32);
    const int bag = bag_of_item(tl, e);
    const uint32_t tC = __shfl(tl.tC, bag);
    const uint64_t ro = __shfl(tl.row_off, bag);
    const float isc = __shfl(bag_scale, bag);
    if (TAB) fill_base_table<SIGN>(tab, item_hash(idx, tC, p.TC, p.a, p.b), p, lane);

    for (int q = 0; q < n; q += U) {
      float gv[U][EPL];
      Elem el[U][EPL];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (q + u < n) {
          const uint64_t grow = readlane_u64b(ro, q + u) + c0 + lane;
          uint32_t h0 = 0, h20 = 0;
          if (!TAB) {
            h0 = item_hash(readlane_u32(idx, q + u), readlane_u32(tC, q + u), p.TC, p.a, p.b);
            if (SIGN) h20 = sign_hash0(h0, p.s_alpha, p.s_beta);
          }
#pragma unroll
          for (int r = 0; r < EPL; ++r) {
            gv[u][r] = 0.f;
            el[u][r] = Elem{0u, 0u, false};
            if (act[r]) {
              gv[u][r] = load_row(grad, grow + kWave * r);
              const uint32_t ent =
                  TAB ? tab[(q + u) * kTabStride + jj[r]]
                      : chunk_entry<SIGN>(fast_mod(add_mod_p(h0, step[r]), p.fm_c, p.M),
                                          add_mod_p(h20, step2[r]), p);
              el[u][r] = elem_of<SIGN>(ent, kk[r], p.M);
            }
          }
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (q + u < n) {
          const float sc = readlane_f32(isc, q + u);
#pragma unroll
          for (int r = 0; r < EPL; ++r)
            if (act[r] && (!SIGN || el[u][r].read))
              unsafeAtomicAdd(dst + el[u][r].m,
                              SIGN ? apply_sign(sc * gv[u][r], el[u][r]) : sc * gv[u][r]);
        }
      }
    }
  }
}

template <int EPL, int U, bool TAB, bool SIGN, typename GT>
static hipError_t launch_dep_t(float* dst, float scale, const KParams& p, const void* indices,
                               const void* offsets, const GT* grad, hipStream_t stream) {
  const uint64_t tiles = (p.num_bags + kTileBags - 1) / kTileBags;
  const uint64_t blocks = (tiles + kWavesPerBlock - 1) / kWavesPerBlock;
  const uint32_t slabs = (p.d + kWave * EPL - 1) / (kWave * EPL);
  if (blocks > 0x7fffffffull) return hipErrorInvalidConfiguration;
  dim3 grid(static_cast<uint32_t>(blocks), slabs);
  hipLaunchKernelGGL((deposit_kernel<EPL, U, TAB, SIGN, GT>), grid, dim3(kBlockThreads), 0, stream,
                     dst, scale, p, indices, offsets, grad);
  return hipGetLastError();
}

template <bool TAB, bool SIGN, typename GT>
static hipError_t launch_dep_c(float* dst, float scale, const KParams& p, const void* indices,
                               const void* offsets, const GT* grad, hipStream_t stream) {
  if (p.d <= 64) return launch_dep_t<1, 16, TAB, SIGN>(dst, scale, p, indices, offsets, grad, stream);
  if (p.d <= 128) return launch_dep_t<2, 8, TAB, SIGN>(dst, scale, p, indices, offsets, grad, stream);
  if (p.d <= 256) return launch_dep_t<4, 4, TAB, SIGN>(dst, scale, p, indices, offsets, grad, stream);
  return launch_dep_t<8, 2, TAB, SIGN>(dst, scale, p, indices, offsets, grad, stream);
}

template <bool SIGN, typename GT>
static hipError_t launch_dep_s(float* dst, float scale, const KParams& p, const void* indices,
                               const void* offsets, const GT* grad, hipStream_t stream) {
  if (p.C <= static_cast<uint32_t>(kTabChunks))
    return launch_dep_c<true, SIGN>(dst, scale, p, indices, offsets, grad, stream);
  return launch_dep_c<false, SIGN>(dst, scale, p, indices, offsets, grad, stream);
}

template <typename GT>
static hipError_t launch_dep_g(float* dst, float scale, const KParams& p, const void* indices,
                               const void* offsets, const GT* grad, hipStream_t stream) {
  if (p.sign_mode) return launch_dep_s<true>(dst, scale, p, indices, offsets, grad, stream);
  return launch_dep_s<false>(dst, scale, p, indices, offsets, grad, stream);
}

hipError_t launch_deposit_atomic(float* dst, float scale, const KParams& p, const void* indices,
                                 const void* offsets, const void* grad, hipStream_t stream) {
  if (p.rows_bf16)
    return launch_dep_g(dst, scale, p, indices, offsets, static_cast<const uint16_t*>(grad), stream);
  return launch_dep_g(dst, scale, p, indices, offsets, static_cast<const float*>(grad), stream);
}

// ---------------------------------------------------------------------------
// Optimizer over a dense gradient buffer.
//   SGD:      w -= lr * g
//   Adagrad:  s += g^2;  w -= lr * g / (sqrt(s) + eps)
// Elements with g == 0 are skipped (bit-identical, no store).  float32
// arithmetic; bfloat16 storage is widened exactly and rounded once (RNE).
// ---------------------------------------------------------------------------

// G and the Adagrad state are read (and the state written) non-temporally,
// the weights through the caches: the memory-side cache then keeps the
// weights this pass has just written, which the next forward gathers,
// rather than the state streamed beside them (bfloat16 row-hash workload,
// 128 MB array and 256 MB state: that forward 876 -> 754 us).
template <typename WT, bool ADAGRAD>
__global__ __launch_bounds__(kBlockThreads) void optimizer_kernel(
    WT* __restrict__ w, float* __restrict__ s, const float* __restrict__ G, const int64_t M,
    const float lr, const float eps) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlockThreads;
  for (int64_t m = static_cast<int64_t>(blockIdx.x) * kBlockThreads + threadIdx.x; m < M;
       m += stride) {
    const float g = __builtin_nontemporal_load(G + m);
    if (g != 0.f)
      update_loaded<WT, ADAGRAD, true>(w, s, m, g, load_weight64(w, m),
                                       ADAGRAD ? __builtin_nontemporal_load(s + m) : 0.f, lr, eps);
  }
}

static uint32_t grid_for(int64_t n, int per_thread) {
  const int64_t want = (n + static_cast<int64_t>(kBlockThreads) * per_thread - 1) /
                       (static_cast<int64_t>(kBlockThreads) * per_thread);
  const int64_t cap = 256 * 32;  // 256 CUs x 32 blocks: enough to fill the chip
  return static_cast<uint32_t>(want < 1 ? 1 : (want > cap ? cap : want));
}

hipError_t launch_optimizer(void* w, bool bf16, float* state, const float* G, int64_t M, float lr,
                            float eps, hipStream_t stream) {
  const dim3 grid(grid_for(M, 4)), block(kBlockThreads);
  if (bf16) {
    uint16_t* wb = static_cast<uint16_t*>(w);
    if (state)
      hipLaunchKernelGGL((optimizer_kernel<uint16_t, true>), grid, block, 0, stream, wb, state, G,
                         M, lr, eps);
    else
      hipLaunchKernelGGL((optimizer_kernel<uint16_t, false>), grid, block, 0, stream, wb, state,
                         G, M, lr, eps);
  } else {
    float* wf = static_cast<float*>(w);
    if (state)
      hipLaunchKernelGGL((optimizer_kernel<float, true>), grid, block, 0, stream, wf, state, G, M,
                         lr, eps);
    else
      hipLaunchKernelGGL((optimizer_kernel<float, false>), grid, block, 0, stream, wf, state, G,
                         M, lr, eps);
  }
  return hipGetLastError();
}

__global__ __launch_bounds__(kBlockThreads) void zero_kernel(float* __restrict__ dst,
                                                             const int64_t n) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlockThreads;
  for (int64_t m = static_cast<int64_t>(blockIdx.x) * kBlockThreads + threadIdx.x; m < n;
       m += stride)
    dst[m] = 0.f;
}

hipError_t launch_zero(float* dst, int64_t n, hipStream_t stream) {
  hipLaunchKernelGGL(zero_kernel, dim3(grid_for(n, 4)), dim3(kBlockThreads), 0, stream, dst, n);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Debug export of the chunk bases (and sign factors): one thread per item.
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kBlockThreads) void debug_addresses_kernel(
    const KParams p, const void* __restrict__ indices, const void* __restrict__ offsets,
    uint32_t* __restrict__ base_out, int8_t* __restrict__ sign_out) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * kBlockThreads + threadIdx.x;
  if (e >= p.N) return;
  // largest bag g with offsets[g] <= e (offsets assumed monotone)
  uint64_t lo = 0, hi = p.num_bags - 1;
  while (lo < hi) {
    const uint64_t mid = lo + (hi - lo + 1) / 2;
    if (load_offset(offsets, mid, p.idx32) <= e) lo = mid; else hi = mid - 1;
  }
  const uint32_t t = static_cast<uint32_t>(lo / p.B);
  const uint32_t i = load_index(indices, e, p.idx32);
  const uint32_t h0 = item_hash(i, t * p.C, p.TC, p.a, p.b);
  const uint32_t h20 = p.sign_mode ? sign_hash0(h0, p.s_alpha, p.s_beta) : 0u;
  for (uint32_t j = 0; j < p.C; ++j) {
    if (base_out) base_out[e * p.C + j] = fast_mod(add_mod_p(h0, chunk_step(p.a, j)), p.fm_c, p.M);
    if (sign_out) {
      int8_t f = 1;
      if (p.sign_mode) {
        const uint32_t code = sign_code(add_mod_p(h20, chunk_step(p.a2, j)), p.sign_mode);
        f = code == 0 ? 1 : (code == 1 ? -1 : 0);
      }
      sign_out[e * p.C + j] = f;
    }
  }
}

hipError_t launch_debug_addresses(const KParams& p, const void* indices, const void* offsets,
                                  uint32_t* base_out, int8_t* sign_out, hipStream_t stream) {
  if (p.N == 0) return hipSuccess;
  const int64_t blocks = (p.N + kBlockThreads - 1) / kBlockThreads;
  hipLaunchKernelGGL(debug_addresses_kernel, dim3(static_cast<uint32_t>(blocks)),
                     dim3(kBlockThreads), 0, stream, p, indices, offsets, base_out, sign_out);
  return hipGetLastError();
}

}  // namespace pss
