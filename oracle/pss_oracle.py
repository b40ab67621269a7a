"""Plain float64 oracle of the PSS hashed-embedding hot path.

TEST INFRASTRUCTURE ONLY (see the package docstring): never imported by the
product path.

What is computed, and where the paper defines it
------------------------------------------------
* Mapping (Sec. 2.5, "HashedNet and ROBE-Z"): chunk j of the embedding of
  token i is read from the flat learnable array at h(i, j) .. h(i, j) + Z - 1.
  h is a universal hash (Sec. 2.5, "Sparse JL with independence relaxation":
  the mapping is generated on the fly by universal hashing, O(1) memory).
  Readings used here (each listed in the design notes):
    - key   = (i * T + t) * C + j for token i of table t, chunk j, C = d / Z
              (one array shared by all T tables, t folded into the key);
    - h     = ((a * key + b) mod p) mod M with p = 2^31 - 1, range [0, M-1];
    - element k of the chunk lives at (h + k) mod M (circular wrap);
    - chunk j covers output dims [j Z, (j + 1) Z); Z must divide d.
* Forward (Sec. 2.4, forward(i) = (S e_i)^T M): sum-pool of the mapped rows
  over each bag.
* Backward (Sec. 2.4, backward(i, Delta) = (S e_i) Delta; Alg. 1): the
  gradient of the flat array is the scatter-add of the output gradient onto
  the addresses that were read.  Alg. 1 dense branch = ``gradient_dense``,
  sparse branch (findUnique + scatter_add) = ``gradient_sparse``.
* Update: plain SGD (Sec. 4, training-time experiment uses SGD) and Adagrad
  with the usual accumulator semantics (s += g^2; w -= lr g / (sqrt(s) + eps)).
  Both evaluated in float64 and rounded once to the storage type.

Everything here is exact integer arithmetic for the addresses (NumPy uint64,
no overflow for index < 2^31 and T*C <= 2^32) and float64 for the values.
"""
from __future__ import annotations

import numpy as np

P = 2**31 - 1  # Mersenne prime modulus of the universal hash
MASK64 = (1 << 64) - 1

F32 = "f32"
BF16 = "bf16"

# ---------------------------------------------------------------------------
# Hash parameters from a seed.  The paper draws the universal hash at random
# without fixing a generator; the reading taken here is SplitMix64 (Steele,
# Lea & Flood, "Fast splittable pseudorandom number generators", OOPSLA 2014):
# a = 1 + (x1 mod (p - 1)), b = x2 mod p from its first two outputs.
# ---------------------------------------------------------------------------


def splitmix64(seed: int, count: int) -> list[int]:
    """First ``count`` outputs of SplitMix64 started from state ``seed``."""
    state = seed & MASK64
    outs = []
    for _ in range(count):
        state = (state + 0x9E3779B97F4A7C15) & MASK64
        z = state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
        outs.append(z ^ (z >> 31))
    return outs


def hash_params_from_seed(seed: int) -> tuple[int, int]:
    x1, x2 = splitmix64(seed, 2)
    a = 1 + (x1 % (P - 1))
    b = x2 % P
    return a, b


def sign_params_from_seed(seed: int) -> tuple[int, int]:
    """(a2, b2) of the second (sign) hash: outputs 3 and 4 of the same stream."""
    x = splitmix64(seed, 4)
    return 1 + (x[2] % (P - 1)), x[3] % P


# ---------------------------------------------------------------------------
# Validation (same categories as the C ABI; raises ValueError)
# ---------------------------------------------------------------------------


def validate(M, Z, d, T, B, a, b, indices, offsets, weight_dtype=F32):
    if weight_dtype not in (F32, BF16):
        raise ValueError("unsupported weight dtype")
    if not (1 <= M <= P):
        raise ValueError("M out of range")
    if Z < 1 or Z > M:
        raise ValueError("Z out of range")
    if d < 1 or d > 4096 or d % Z != 0:
        raise ValueError("d must be a multiple of Z, 1 <= d <= 4096")
    if not (1 <= a <= P - 1):
        raise ValueError("a out of range")
    if not (0 <= b <= P - 1):
        raise ValueError("b out of range")
    if T < 1 or B < 1:
        raise ValueError("need at least one bag")
    if T * (d // Z) > 2**32:
        raise ValueError("T*C too large")
    offsets = np.asarray(offsets)
    indices = np.asarray(indices)
    if offsets.shape != (T * B + 1,):
        raise ValueError("offsets must have T*B+1 entries")
    if offsets[0] != 0 or offsets[-1] != indices.shape[0]:
        raise ValueError("offsets must start at 0 and end at N")
    if np.any(np.diff(offsets) < 0):
        raise ValueError("offsets must be non-decreasing")
    if indices.size and (indices.min() < 0 or indices.max() >= 2**31):
        raise ValueError("indices must lie in [0, 2^31)")


# ---------------------------------------------------------------------------
# Addresses
# ---------------------------------------------------------------------------


def item_bags(T, B, offsets):
    """For every bag item e: its bag g, table t = g div B and sample b = g mod B."""
    offsets = np.asarray(offsets, dtype=np.int64)
    lengths = np.diff(offsets)
    g = np.repeat(np.arange(T * B, dtype=np.int64), lengths)
    return g, g // B, g % B


def bases_for(M, Z, d, T, a, b, idx, t):
    """h(i, j) for items with token ``idx`` in table ``t``: uint64 [n, C].

    key = (i*T + t)*C + j and h = ((a*key + b) mod p) mod M.  Computed as
    ((a * (key mod p) + b) mod p) mod M, which is the same residue; every
    intermediate stays below 2^63.
    """
    C = d // Z
    i = np.asarray(idx, dtype=np.int64).astype(np.uint64)
    tt = np.asarray(t, dtype=np.int64).astype(np.uint64)
    j = np.arange(C, dtype=np.uint64)
    key = (i * np.uint64(T) + tt)[:, None] * np.uint64(C) + j[None, :]
    h = (np.uint64(a) * (key % np.uint64(P)) + np.uint64(b)) % np.uint64(P)
    return h % np.uint64(M)


def chunk_bases(M, Z, d, T, B, a, b, indices, offsets):
    """h(i, j) for every bag item and chunk: uint64 array [N, C]."""
    _, t, _ = item_bags(T, B, offsets)
    return bases_for(M, Z, d, T, a, b, indices, t)


def addresses_from_bases(M, Z, base):
    """Output dim c = j*Z + k of an item reads (h(i, j) + k) mod M: int64 [n, C*Z]."""
    base = np.asarray(base).astype(np.int64)
    k = np.arange(Z, dtype=np.int64)
    addr = (base[:, :, None] + k[None, None, :]) % M
    return addr.reshape(base.shape[0], base.shape[1] * Z)


def element_addresses(M, Z, d, T, B, a, b, indices, offsets):
    """Address in the flat array of every output element: int64 [N, d]."""
    return addresses_from_bases(M, Z, chunk_bases(M, Z, d, T, B, a, b, indices, offsets))


# ---------------------------------------------------------------------------
# Optional sign of each chunk (Sec. 2.5, sparse JL with independence
# relaxation: the entries of S are 0 with probability 2/3 and +1 / -1 with
# probability 1/6 each, generated on the fly by universal hashing).  Reading
# used here: a second universal hash of the same key,
#     h2 = (a2 * key + b2) mod p,
# decides the factor of the whole chunk (i, j):
#   "pm1"    : -1 if h2 >= 2^30 else +1            (random signs only)
#   "sparse" : +1 if h2 < q, -1 if q <= h2 < 2q, else 0,   q = floor(p / 6)
# A factor of 0 means the chunk is not read at all: it contributes nothing to
# the forward and receives no gradient.  ``sign`` arguments below are None
# (no sign, the ROBE-Z mapping as printed) or a tuple (mode, a2, b2).
# ---------------------------------------------------------------------------

SIGN_PM1 = "pm1"
SIGN_SPARSE = "sparse"
Q6 = P // 6  # 357913941


def signs_for(Z, d, T, a2, b2, idx, t, mode):
    """Factor (+1, -1 or 0) of chunk j of items with token ``idx`` in table ``t``: int64 [n, C]."""
    C = d // Z
    i = np.asarray(idx, dtype=np.int64).astype(np.uint64)
    tt = np.asarray(t, dtype=np.int64).astype(np.uint64)
    j = np.arange(C, dtype=np.uint64)
    key = (i * np.uint64(T) + tt)[:, None] * np.uint64(C) + j[None, :]
    h2 = ((np.uint64(a2) * (key % np.uint64(P)) + np.uint64(b2)) % np.uint64(P)).astype(np.int64)
    if mode == SIGN_PM1:
        return np.where(h2 >= 2**30, -1, 1).astype(np.int64)
    if mode == SIGN_SPARSE:
        return np.where(h2 < Q6, 1, np.where(h2 < 2 * Q6, -1, 0)).astype(np.int64)
    raise ValueError("unknown sign mode")


def element_factors(Z, d, T, B, offsets, indices, sign):
    """Factor of every read element, float64 [N, d] (chunk factor repeated Z times)."""
    mode, a2, b2 = sign
    _, t, _ = item_bags(T, B, offsets)
    return np.repeat(signs_for(Z, d, T, a2, b2, indices, t, mode), Z, axis=1).astype(np.float64)


def item_scale(T, B, offsets, mean):
    """Per-item weight of its bag's pooled row: 1, or 1/|bag| for mean pooling."""
    offsets = np.asarray(offsets, dtype=np.int64)
    g, _, _ = item_bags(T, B, offsets)
    if not mean:
        return np.ones(g.shape[0])
    return 1.0 / np.diff(offsets)[g].astype(np.float64)


# ---------------------------------------------------------------------------
# Storage types
# ---------------------------------------------------------------------------


def widen(w, weight_dtype=F32):
    """Stored weights as exact float64 (bf16 given as uint16 bit patterns)."""
    if weight_dtype == F32:
        return np.asarray(w, dtype=np.float32).astype(np.float64)
    bits = np.asarray(w, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return bits.view(np.float32).astype(np.float64)


def round_to_bf16_bits(x):
    """Round float64 values to bfloat16 (nearest, ties to even), once.

    bfloat16 has the float32 exponent range and 8 significant bits.  For a
    finite x the spacing of representable values around x is
    2^(e - 8) with x = f * 2^e, 0.5 <= |f| < 1, but never finer than the
    subnormal step 2^-133.  Values that round beyond the largest finite
    bfloat16 become infinity; NaN becomes the canonical quiet NaN.
    Returns uint16 bit patterns.
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.empty(x.shape, dtype=np.uint16)
    nan = np.isnan(x)
    fin = np.isfinite(x)
    _, e = np.frexp(np.where(fin, x, 1.0))
    step = np.ldexp(1.0, np.maximum(e - 8, -133))
    r = np.rint(np.where(fin, x, 0.0) / step) * step  # np.rint: ties to even
    r = np.where(fin, r, x)
    max_bf16 = float(np.uint32(0x7F7F0000).view(np.float32))
    overflow = np.abs(r) > max_bf16
    r32 = np.where(overflow, np.copysign(np.inf, r), r).astype(np.float32)
    out[...] = (r32.view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    out[nan] = 0x7FC0
    return out


def round_storage(x64, weight_dtype=F32):
    if weight_dtype == F32:
        return np.asarray(x64, dtype=np.float64).astype(np.float32)
    return round_to_bf16_bits(x64)


# ---------------------------------------------------------------------------
# Forward (Sec. 2.4 forward(i) = (S e_i)^T M, ROBE-Z mapping, sum pooling)
# ---------------------------------------------------------------------------


def _signed(rows, fac):
    """fac * rows with a factor of 0 giving exactly 0 (the element is not read)."""
    return rows if fac is None else np.where(fac == 0, 0.0, fac * rows)


def forward64(w, M, Z, d, T, B, a, b, indices, offsets, weight_dtype=F32, sign=None,
              mean=False):
    """Pooled embeddings in float64, [B, T*d], plus sum of |terms| per output.

    out[b, t*d + c] = sum over items e of bag (t, b) of w[addr(e, c)]
    (times the chunk's factor when ``sign`` is given; divided by |bag| when
    ``mean``).  An empty bag gives 0.
    """
    offsets = np.asarray(offsets, dtype=np.int64)
    addr = element_addresses(M, Z, d, T, B, a, b, indices, offsets)
    rows = widen(np.asarray(w)[addr], weight_dtype)  # [N, d]
    if sign is not None:
        rows = _signed(rows, element_factors(Z, d, T, B, offsets, indices, sign))
    out = np.zeros((T * B, d))
    s_abs = np.zeros((T * B, d))
    lengths = np.diff(offsets)
    nonempty = np.nonzero(lengths > 0)[0]
    if nonempty.size:
        starts = offsets[:-1][nonempty]
        out[nonempty] = np.add.reduceat(rows, starts, axis=0)
        s_abs[nonempty] = np.add.reduceat(np.abs(rows), starts, axis=0)
        if mean:
            out[nonempty] /= lengths[nonempty, None]
            s_abs[nonempty] /= lengths[nonempty, None]
    # bag g = t*B + b  ->  out[b, t*d : (t+1)*d]
    out = out.reshape(T, B, d).transpose(1, 0, 2).reshape(B, T * d)
    s_abs = s_abs.reshape(T, B, d).transpose(1, 0, 2).reshape(B, T * d)
    return out, s_abs


def forward_at(w, M, Z, d, T, B, a, b, indices, offsets, bags, weight_dtype=F32, sign=None,
               mean=False):
    """Pooled float64 rows of the listed bags g = t*B + b only: ([nb, d], s_abs).

    Same sums as ``forward64``; used to check sampled bags of large batches.
    """
    w = np.asarray(w)
    offsets = np.asarray(offsets, dtype=np.int64)
    indices = np.asarray(indices, dtype=np.int64)
    bags = np.asarray(bags, dtype=np.int64)
    out = np.zeros((bags.shape[0], d))
    s_abs = np.zeros((bags.shape[0], d))
    for r, g in enumerate(bags):
        lo, hi = offsets[g], offsets[g + 1]
        if hi == lo:
            continue
        t = np.full(hi - lo, g // B, dtype=np.int64)
        addr = addresses_from_bases(M, Z, bases_for(M, Z, d, T, a, b, indices[lo:hi], t))
        rows = widen(w[addr], weight_dtype)
        if sign is not None:
            mode, a2, b2 = sign
            fac = np.repeat(signs_for(Z, d, T, a2, b2, indices[lo:hi], t, mode), Z, axis=1)
            rows = _signed(rows, fac.astype(np.float64))
        div = float(hi - lo) if mean else 1.0
        out[r] = rows.sum(axis=0) / div
        s_abs[r] = np.abs(rows).sum(axis=0) / div
    return out, s_abs


def forward(w, M, Z, d, T, B, a, b, indices, offsets, weight_dtype=F32, sign=None, mean=False):
    """Pooled embeddings rounded once to float32, [B, T*d]."""
    out64, _ = forward64(w, M, Z, d, T, B, a, b, indices, offsets, weight_dtype, sign, mean)
    return out64.astype(np.float32)


# ---------------------------------------------------------------------------
# Gradient of the flat array (Alg. 1)
# ---------------------------------------------------------------------------


def _contributions(M, Z, d, T, B, a, b, indices, offsets, grad_out, sign=None, mean=False):
    """Flattened (address, upstream gradient) pairs of every read element.

    With mean pooling an item's share of its bag's gradient row is the row
    divided by |bag|; with a sign the chunk's factor multiplies it and
    chunks of factor 0 contribute nothing."""
    addr = element_addresses(M, Z, d, T, B, a, b, indices, offsets)
    _, t, bb = item_bags(T, B, offsets)
    g = np.asarray(grad_out, dtype=np.float64).reshape(B, T, d)[bb, t, :]
    if mean:
        g = g * item_scale(T, B, offsets, True)[:, None]
    if sign is None:
        return addr.ravel(), g.ravel()
    fac = element_factors(Z, d, T, B, offsets, indices, sign).ravel()
    keep = fac != 0
    return addr.ravel()[keep], (g.ravel() * fac)[keep]


def gradient_dense(M, Z, d, T, B, a, b, indices, offsets, grad_out, sign=None, mean=False):
    """Alg. 1, dense branch: G = zeros(M).scatter_add(addresses, grad values).

    Returns (G, A, cnt): the float64 gradient, the sum of |contributions| per
    element and the number of contributions per element.
    """
    addr, g = _contributions(M, Z, d, T, B, a, b, indices, offsets, grad_out, sign, mean)
    G = np.bincount(addr, weights=g, minlength=M)
    A = np.bincount(addr, weights=np.abs(g), minlength=M)
    cnt = np.bincount(addr, minlength=M)
    return G, A, cnt


def gradient_sparse(M, Z, d, T, B, a, b, indices, offsets, grad_out, sign=None, mean=False):
    """Alg. 1, sparse branch: unique addresses and the summed values there."""
    addr, g = _contributions(M, Z, d, T, B, a, b, indices, offsets, grad_out, sign, mean)
    unique, inverse = np.unique(addr, return_inverse=True)
    vals = np.zeros(unique.shape[0])
    np.add.at(vals, inverse, g)
    return unique, vals


def gradient_at(M, Z, d, T, B, a, b, indices, offsets, grad_out, where, sign=None, mean=False):
    """G, A and cnt restricted to the flat-array elements listed in ``where``.

    Same sums as ``gradient_dense`` without an M-sized result; used to check
    sampled elements of very large arrays.  Items are processed in blocks.
    """
    where = np.asarray(where, dtype=np.int64)
    if np.unique(where).shape[0] != where.shape[0]:
        raise ValueError("sampled elements must be distinct")
    order = np.argsort(where)
    sw = where[order]
    G = np.zeros(where.shape[0])
    A = np.zeros(where.shape[0])
    cnt = np.zeros(where.shape[0], dtype=np.int64)
    offsets = np.asarray(offsets, dtype=np.int64)
    indices = np.asarray(indices, dtype=np.int64)
    grad3 = np.asarray(grad_out).reshape(B, T, d)
    gbag, t_all, b_all = item_bags(T, B, offsets)
    scale = item_scale(T, B, offsets, mean)
    N = indices.shape[0]
    # one flat-array element per output dim: split the items into blocks
    block = max(1, 4_000_000 // max(d, 1))
    for s in range(0, N, block):
        e = min(N, s + block)
        idx = indices[s:e]
        tt = t_all[s:e]
        addr = addresses_from_bases(M, Z, bases_for(M, Z, d, T, a, b, idx, tt))
        pos = np.searchsorted(sw, addr)
        pos_c = np.minimum(pos, sw.shape[0] - 1)
        hit = sw[pos_c] == addr
        if not hit.any():
            continue
        if sign is not None:
            mode, a2, b2 = sign
            fac = np.repeat(signs_for(Z, d, T, a2, b2, idx, tt, mode), Z, axis=1)
            hit &= fac != 0
        ei, ci = np.nonzero(hit)
        vals = grad3[b_all[s:e][ei], tt[ei], ci].astype(np.float64) * scale[s:e][ei]
        if sign is not None:
            vals = vals * fac[ei, ci]
        slot = pos_c[ei, ci]
        np.add.at(G, order[slot], vals)
        np.add.at(A, order[slot], np.abs(vals))
        np.add.at(cnt, order[slot], 1)
    return G, A, cnt


# ---------------------------------------------------------------------------
# Updates (rounded once to storage)
# ---------------------------------------------------------------------------


def sgd_update(w, G, lr, weight_dtype=F32):
    """w <- w - lr * G, in float64, rounded once to the storage type."""
    w64 = widen(w, weight_dtype)
    return round_storage(w64 - lr * G, weight_dtype)


def adagrad_update(w, s, G, lr, eps, weight_dtype=F32):
    """s <- s + G^2 ; w <- w - lr * G / (sqrt(s) + eps), float64, rounded once.

    Returns (w_new, s_new) with w_new in the storage type and s_new float32.
    """
    w64 = widen(w, weight_dtype)
    s64 = np.asarray(s, dtype=np.float32).astype(np.float64)
    s_new = s64 + G * G
    w_new = w64 - lr * G / (np.sqrt(s_new) + eps)
    return round_storage(w_new, weight_dtype), s_new.astype(np.float32)


def backward_update(w, s, M, Z, d, T, B, a, b, indices, offsets, grad_out, lr,
                    eps=1e-10, weight_dtype=F32, sign=None, mean=False):
    """Full backward + fused update.  ``s is None`` selects SGD, else Adagrad.

    Returns (w_new, s_new or None, G, A, cnt).
    """
    G, A, cnt = gradient_dense(M, Z, d, T, B, a, b, indices, offsets, grad_out, sign, mean)
    if s is None:
        return sgd_update(w, G, lr, weight_dtype), None, G, A, cnt
    w_new, s_new = adagrad_update(w, s, G, lr, eps, weight_dtype)
    return w_new, s_new, G, A, cnt


# ---------------------------------------------------------------------------
# Post-hoc compression of a given table (Sec. 2.4 with Thm. 2: the flat
# array is M = S E and token i is retrieved as (S e_i)^T M) and the
# (1 +- eps) property of Def. 2.
# ---------------------------------------------------------------------------


def table_addresses(M, Z, d, T, n, a, b):
    """Address of element (t, i, c) of T tables with n rows each: int64 [T, n, d]."""
    t = np.repeat(np.arange(T, dtype=np.int64), n)
    i = np.tile(np.arange(n, dtype=np.int64), T)
    return addresses_from_bases(M, Z, bases_for(M, Z, d, T, a, b, i, t)).reshape(T, n, d)


def compress(E, M, Z, a, b):
    """M = S E for tables E [T, n, d]: element m of the flat array is the sum
    of the table entries the mapping sends to m.  Returns (Mv, Mabs) in
    float64, Mabs being the sum of the absolute values of those entries."""
    E64 = np.asarray(E, dtype=np.float64)
    T, n, d = E64.shape
    addr = table_addresses(M, Z, d, T, n, a, b).ravel()
    Mv = np.bincount(addr, weights=E64.ravel(), minlength=M)
    Mabs = np.bincount(addr, weights=np.abs(E64).ravel(), minlength=M)
    return Mv, Mabs


def recover(w, M, Z, d, T, n, a, b, weight_dtype=F32):
    """Retrieved rows (S e_(t,i))^T M of every token of every table: float64 [T, n, d]."""
    return widen(w, weight_dtype)[table_addresses(M, Z, d, T, n, a, b)]


def pss_row_error(E, R):
    """Per-row eps of Def. 2: sup over x != 0 of |<R_i, x> - <E_i, x>| / ||x||_2.

    By Cauchy-Schwarz the supremum is attained at x = R_i - E_i and equals
    ||R_i - E_i||_2.  E, R: [..., d]; returns float64 [...]."""
    D = np.asarray(R, dtype=np.float64) - np.asarray(E, dtype=np.float64)
    return np.sqrt(np.sum(D * D, axis=-1))
