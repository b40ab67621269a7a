// Exact integer hashing of the ROBE-Z mapping for gfx950 (and the host).
//
// The universal hash of the paper's Sec. 2.5 mapping is
//     h(key) = ((a * key + b) mod p) mod M,   p = 2^31 - 1,
//     key    = (i * T + t) * C + j.
// All arithmetic here is exact; nothing is rounded.
//
//  * mod p uses 2^31 = 1 (mod p): x = hi * 2^31 + lo  =>  x = hi + lo (mod p).
//  * Consecutive chunks of one token differ by one in the key, so
//    h_j = (h_0 + (a * j mod p)) mod p: the per-item part (h_0) is uniform
//    across a wavefront, the per-lane part (a * j mod p) is a constant.
//  * mod M uses Lemire, Kaser & Kurz, "Faster remainder by direct computation"
//    (Softw. Pract. Exp. 2019): with c = floor((2^64 - 1) / M) + 1,
//    x mod M = floor(((c * x) mod 2^64) * M / 2^64), exact for all 32-bit x
//    and 1 <= M < 2^32.
#pragma once

#include <stdint.h>

#if defined(__HIPCC__)
#define PSS_HD __host__ __device__ __forceinline__
#else
#define PSS_HD inline
#endif

namespace pss {

constexpr uint32_t kP = 2147483647u;  // 2^31 - 1

// x mod p for any 64-bit x.
PSS_HD uint32_t mod_p(uint64_t x) {
  uint64_t s = (x & kP) + (x >> 31);  // < 2^31 + 2^33
  s = (s & kP) + (s >> 31);           // < 2^31 + 5
  uint32_t r = static_cast<uint32_t>(s);
  return r >= kP ? r - kP : r;
}

// High 64 bits of the 96-bit product x * m (m < 2^32).
PSS_HD uint64_t mulhi_64x32(uint64_t x, uint32_t m) {
  const uint64_t lo = static_cast<uint64_t>(static_cast<uint32_t>(x)) * m;
  const uint64_t hi = static_cast<uint64_t>(static_cast<uint32_t>(x >> 32)) * m + (lo >> 32);
  return hi >> 32;
}

struct FastMod {
  uint64_t c;  // floor((2^64 - 1) / M) + 1  (0 when M == 1)
  uint32_t M;
};

inline FastMod make_fastmod(uint32_t M) {
  FastMod f;
  f.c = UINT64_MAX / M + 1;
  f.M = M;
  return f;
}

PSS_HD uint32_t fast_mod(uint32_t x, uint64_t c, uint32_t M) {
  const uint64_t low = c * x;  // mod 2^64
  return static_cast<uint32_t>(mulhi_64x32(low, M));
}

// (a * j) mod p, the per-chunk increment of the hash.
PSS_HD uint32_t chunk_step(uint32_t a, uint32_t j) {
  return mod_p(static_cast<uint64_t>(a) * j);
}

// h_0 = (a * ((i*T + t)*C mod p) + b) mod p for token i of table t.
// TC = T*C < 2^32 and i < 2^32, so (i*T + t)*C = i*TC + t*C < 2^64.
PSS_HD uint32_t item_hash(uint32_t i, uint32_t tC, uint32_t TC, uint32_t a, uint32_t b) {
  const uint64_t key0 = static_cast<uint64_t>(i) * TC + tC;
  return mod_p(static_cast<uint64_t>(a) * mod_p(key0) + b);
}

// (h_0 + step) mod p, both already reduced.
PSS_HD uint32_t add_mod_p(uint32_t h0, uint32_t step) {
  const uint32_t s = h0 + step;  // < 2^32
  return s >= kP ? s - kP : s;
}

// Address of element k (0 <= k < Z <= M) of the chunk starting at base < M.
PSS_HD uint32_t wrap_add(uint32_t base, uint32_t k, uint32_t M) {
  const uint32_t s = base + k;  // < 2^32 since base, k < M <= p
  return s >= M ? s - M : s;
}

// ---------------------------------------------------------------------------
// Optional chunk sign (Sec. 2.5: entries of S that are +1, -1 or 0, drawn by
// a universal hash).  A second hash of the same key, h2 = (a2 * key + b2)
// mod p, gives the factor of chunk (i, j):
//   mode 1 (+-1):   -1 if h2 >= 2^30, else +1
//   mode 2 (+-1/0): +1 if h2 < q, -1 if q <= h2 < 2q, else 0, q = floor(p/6)
// Kernels that only hold the item hash h_0 = (a * key_0 + b) mod p recover
// the second hash from it: key_0 = (h_0 - b) * a^-1 (mod p), hence
// h2_0 = alpha * h_0 + beta (mod p) with alpha = a2 * a^-1 and
// beta = b2 - alpha * b; chunk j adds a2 * j (mod p) as for the location.
// ---------------------------------------------------------------------------
constexpr uint32_t kQ6 = kP / 6;  // 357913941

// Sign code of a chunk: 0 = +1, 1 = -1, 2 = not read (factor 0).
PSS_HD uint32_t sign_code(uint32_t h2, uint32_t mode) {
  if (mode == 1) return h2 >= (1u << 30) ? 1u : 0u;
  return h2 < kQ6 ? 0u : (h2 < 2 * kQ6 ? 1u : 2u);
}

// h2_0 from the item hash h_0 (alpha, beta < p).
PSS_HD uint32_t sign_hash0(uint32_t h0, uint32_t alpha, uint32_t beta) {
  return mod_p(static_cast<uint64_t>(alpha) * h0 + beta);
}

// x^e mod p (host set-up of a^-1 = a^(p-2)).
PSS_HD uint32_t pow_mod_p(uint32_t x, uint32_t e) {
  uint32_t r = 1, b = x;
  while (e) {
    if (e & 1u) r = mod_p(static_cast<uint64_t>(r) * b);
    b = mod_p(static_cast<uint64_t>(b) * b);
    e >>= 1;
  }
  return r;
}

// Full chunk base h(i, j) = (((i*T + t)*C + j) * a + b mod p) mod M.
PSS_HD uint32_t chunk_base(uint32_t i, uint32_t t, uint32_t j, uint32_t C, uint32_t TC,
                           uint32_t a, uint32_t b, uint64_t c, uint32_t M) {
  const uint32_t h = add_mod_p(item_hash(i, t * C, TC, a, b), chunk_step(a, j));
  return fast_mod(h, c, M);
}

}  // namespace pss
