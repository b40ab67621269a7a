"""Pure-Python brute force of the PSS layer on tiny inputs.

TEST INFRASTRUCTURE ONLY.  Independent of ``pss_oracle``: Python integers
for the hash (no key mod p pre-reduction, no NumPy), explicit loops, and the
linear-sketch form of Thm. 2 / Sec. 2.4:

    virtual table row of (t, i):  V[(t, i)] = (S e_(t,i))^T w
    forward:   out[b, t*d + c] = sum over items i of bag (t, b) of V[(t, i)][c]
    backward:  G = S^T (dL/dV)                       (Alg. 1, dense branch)

S has one row per (table, token, output dim) and one column per element of
the flat array; its entry is 1 where the ROBE-Z mapping (Sec. 2.5) reads that
element, so every row holds exactly one 1.
"""
from __future__ import annotations

P = 2**31 - 1


def base(a, b, M, T, C, t, i, j):
    """h(i, j) = ((a * key + b) mod p) mod M with key = (i*T + t)*C + j."""
    key = (i * T + t) * C + j
    return ((a * key + b) % P) % M


def sign_factor(a2, b2, T, C, t, i, j, mode):
    """Factor of chunk j of token i of table t from the second hash
    h2 = (a2 * key + b2) mod p (None mode: always 1)."""
    if mode is None:
        return 1
    h2 = (a2 * ((i * T + t) * C + j) + b2) % P
    if mode == "pm1":
        return -1 if h2 >= 2**30 else 1
    q = P // 6
    return 1 if h2 < q else (-1 if h2 < 2 * q else 0)


def sketch_rows(M, Z, d, T, rows_per_table, a, b):
    """Explicit S as a dict {(t, i, c): column of the single 1}.

    Column = (h(i, c // Z) + c % Z) mod M.  Also returned as a dense list of
    lists (rows ordered by (t, i, c)) to make S e_i a literal matrix product.
    """
    C = d // Z
    col = {}
    for t in range(T):
        for i in range(rows_per_table[t]):
            for c in range(d):
                col[(t, i, c)] = (base(a, b, M, T, C, t, i, c // Z) + c % Z) % M
    return col


def dense_S(M, Z, d, T, rows_per_table, a, b, sign=None):
    """S as a list of rows, row index r(t, i, c) in lexicographic order.

    Without ``sign`` the single nonzero of a row is 1; with sign = (mode,
    a2, b2) it is the chunk's factor (+1, -1, or 0: an all-zero row)."""
    col = sketch_rows(M, Z, d, T, rows_per_table, a, b)
    mode, a2, b2 = sign if sign is not None else (None, 0, 0)
    C = d // Z
    keys = sorted(col)
    S = []
    for k in keys:
        t, i, c = k
        row = [0] * M
        row[col[k]] = sign_factor(a2, b2, T, C, t, i, c // Z, mode)
        S.append(row)
    return keys, S


def virtual_table(w, M, Z, d, T, rows_per_table, a, b, sign=None):
    """V[(t, i)] = (S e_(t,i))^T w as lists of floats, via the dense S."""
    keys, S = dense_S(M, Z, d, T, rows_per_table, a, b, sign)
    V = {}
    for r, (t, i, c) in enumerate(keys):
        V.setdefault((t, i), [0.0] * d)
        V[(t, i)][c] = sum(S[r][m] * float(w[m]) for m in range(M))
    return V


def forward(w, M, Z, d, T, B, rows_per_table, a, b, indices, offsets, sign=None, mean=False):
    """Pooled embeddings [B][T*d] as Python floats (sums of doubles; with
    ``mean`` each nonempty bag's sum is divided by its length)."""
    V = virtual_table(w, M, Z, d, T, rows_per_table, a, b, sign)
    out = [[0.0] * (T * d) for _ in range(B)]
    for t in range(T):
        for bb in range(B):
            g = t * B + bb
            n = int(offsets[g + 1]) - int(offsets[g])
            for e in range(int(offsets[g]), int(offsets[g + 1])):
                i = int(indices[e])
                for c in range(d):
                    out[bb][t * d + c] += V[(t, i)][c]
            if mean and n:
                for c in range(d):
                    out[bb][t * d + c] /= n
    return out


def gradient(M, Z, d, T, B, rows_per_table, a, b, indices, offsets, grad_out, sign=None,
             mean=False):
    """G = S^T (dL/dV) with dL/dV[(t, i)][c] = sum of grad_out over the bags
    that contain token i of table t (with multiplicity; divided by the bag's
    length with ``mean``).  Returns (G, cnt), cnt counting the reads of each
    element (a zero entry of S is no read)."""
    keys, S = dense_S(M, Z, d, T, rows_per_table, a, b, sign)
    dV = {k: 0.0 for k in keys}
    reads = {k: 0 for k in keys}
    for t in range(T):
        for bb in range(B):
            g = t * B + bb
            n = int(offsets[g + 1]) - int(offsets[g])
            for e in range(int(offsets[g]), int(offsets[g + 1])):
                i = int(indices[e])
                for c in range(d):
                    dV[(t, i, c)] += float(grad_out[bb][t * d + c]) / (n if mean else 1)
                    reads[(t, i, c)] += 1
    G = [0.0] * M
    cnt = [0] * M
    for r, k in enumerate(keys):
        for m in range(M):
            if S[r][m]:
                G[m] += S[r][m] * dV[k]
                cnt[m] += reads[k]
    return G, cnt


def compress(E, M, Z, a, b):
    """M = S E with the explicit S (Thm. 2), E given as nested lists [T][n][d]."""
    T, n, d = len(E), len(E[0]), len(E[0][0])
    keys, S = dense_S(M, Z, d, T, [n] * T, a, b)
    Mv = [0.0] * M
    for r, (t, i, c) in enumerate(keys):
        for m in range(M):
            if S[r][m]:
                Mv[m] += float(E[t][i][c])
    return Mv
