"""Pins of the CPU oracle: checks against what the paper and mathematics fix.

Every ``pin_*`` function raises AssertionError when the oracle module ``o``
(normally ``oracle.pss_oracle``) disagrees with an independent fact:

  pin_hash_vectors       published SplitMix64 output, hand-computed residues,
                         exact big-integer evaluation of the hash definition
  pin_forward_brute      explicit 0/1 sketch matrix S (Thm. 2), pure Python
  pin_gradient_brute     G = S^T dL/dV (Alg. 1 dense branch), pure Python
  pin_integer_forward    w[m] = m: pooled sums are integers, exact
  pin_embedding_bag      injective special case == torch embedding_bag(sum)
                         and torch.optim.SGD / Adagrad on the plain table
  pin_mass               total and per-chunk-offset gradient mass; the
                         "loss = sum of retrieved elements" case gives
                         w_new = -count exactly
  pin_finite_difference  L(w) = <grad_out, forward(w)> is linear in w, so
                         L(w + e_m) - L(w) = G[m]
  pin_sparse_dense       Alg. 1 sparse branch, densified, equals dense branch
  pin_untouched          elements no lookup reads stay bit-identical
  pin_bf16_rounding      nearest-even bfloat16 rounding == torch's
  pin_bf16_widening      bfloat16 -> float of every bit pattern == torch's
  pin_sign_and_mean      sign variants and mean pooling against the signed
                         sketch; torch's mean embedding_bag; SplitMix64
                         outputs 2-4; factor frequencies
  pin_compress           post-hoc M = S E and (S e_i)^T M (Sec. 2.4, Thm. 2)
                         against the explicit S; the injective case; eps of
                         Def. 2 as a supremum; the distance bound of Thm. 1

The mutation tests plant mistakes in the oracle and require that at least
one of these pins fails.
"""
from __future__ import annotations

import numpy as np

from oracle import brute

P = 2**31 - 1


def tiny_case(rng, T=None, d=None, Z=None, M=None, B=None, max_len=5):
    T = T or int(rng.integers(1, 4))
    if d is None:
        d = int(rng.choice([1, 2, 4, 6, 8]))
    if Z is None:
        Z = int(rng.choice([z for z in range(1, d + 1) if d % z == 0]))
    M = M or int(rng.integers(max(Z, 2), 65))
    B = B or int(rng.integers(1, 5))
    rows = [int(rng.integers(1, 9)) for _ in range(T)]
    lens = rng.integers(0, max_len + 1, T * B)
    offsets = np.zeros(T * B + 1, dtype=np.int64)
    np.cumsum(lens, out=offsets[1:])
    idx = np.concatenate([rng.integers(0, rows[g // B], lens[g]) for g in range(T * B)]
                         + [np.zeros(0, dtype=np.int64)]).astype(np.int64)
    a = int(rng.integers(1, P))
    b = int(rng.integers(0, P))
    return dict(T=T, d=d, Z=Z, M=M, B=B, rows=rows, offsets=offsets, indices=idx, a=a, b=b)


# ---------------------------------------------------------------------------


def pin_hash_vectors(o):
    # SplitMix64 (Steele, Lea & Flood 2014): its first output from state 0 is
    # 0xE220A8397B1DCDAF (also the first nextLong of java.util.SplittableRandom(0)).
    assert o.splitmix64(0, 1)[0] == 0xE220A8397B1DCDAF
    # (a, b) = (1 + x1 mod (p-1), x2 mod p), evaluated independently with
    # exact integers when the workloads were specified.
    assert o.hash_params_from_seed(0) == (60845732, 2125112010)
    assert o.hash_params_from_seed(1) == (1294668924, 1667631020)
    assert o.hash_params_from_seed(42) == (659044154, 71743339)

    def h(a, b, M, T, C, t, i, j):
        # Z = 1, d = C: one element per chunk, chunk j of token i in table t
        return int(o.bases_for(M, 1, C, T, a, b, np.array([i]), np.array([t]))[0, j])

    # hand case: a=3, b=5, key=10: 3*10+5 = 35; 35 mod p = 35; 35 mod 7 = 0
    assert h(3, 5, 7, 1, 1, 0, 10, 0) == 0
    # a = b = p-1, key = p-1: (p-1)^2 + (p-1) = (p-1) p  == 0 (mod p)
    assert h(P - 1, P - 1, P, 1, 1, 0, P - 1, 0) == 0
    # key = p: a*p + b == b = p-1 (mod p); M = p leaves it unchanged
    assert h(P - 1, P - 1, P, 1, 1, 0, P, 0) == P - 1
    # keys k and k + p collide (T = 1, C = 2, key = 2i + j)
    i2, j2 = divmod(2 * 5 + 1 + P, 2)
    assert h(12345, 678, 1000, 1, 2, 0, 5, 1) == h(12345, 678, 1000, 1, 2, 0, i2, j2)
    # ... and differ from a neighbouring key for this a, b
    assert h(12345, 678, P, 1, 2, 0, 5, 1) != h(12345, 678, P, 1, 2, 0, 5, 0)
    # tiny layout (T=4, C=4, M=4096, seed 0), evaluated independently:
    a, b = 60845732, 2125112010
    for (t, i, j), want in {(0, 0, 0): 714, (0, 0, 1): 367, (1, 7, 2): 614,
                            (2, 500, 0): 3533, (3, 999, 3): 4076}.items():
        assert h(a, b, 4096, 4, 4, t, i, j) == want
    # random keys against the literal big-integer formula (keys up to ~2^62)
    rng = np.random.default_rng(7)
    for _ in range(200):
        a = int(rng.integers(1, P))
        b = int(rng.integers(0, P))
        M = int(rng.choice([1, 2, 7, 4096, 2_500_000, 16_000_000, 10**9, P, int(rng.integers(1, P + 1))]))
        T = int(rng.choice([1, 26, 1000, 65536]))
        C = int(rng.choice([1, 4, 128, 4096]))
        t = int(rng.integers(0, T))
        i = int(rng.choice([0, 1, P - 1, P, 2**31 - 1, int(rng.integers(0, 2**31))]))
        j = int(rng.integers(0, C))
        got = int(o.bases_for(M, 1, C, T, a, b, np.array([i]), np.array([t]))[0, j])
        assert got == brute.base(a, b, M, T, C, t, i, j), (a, b, M, T, C, t, i, j)


def pin_forward_brute(o, seed=0, cases=40):
    rng = np.random.default_rng(seed)
    for _ in range(cases):
        c = tiny_case(rng)
        w = (rng.standard_normal(c["M"]) * 0.5).astype(np.float32)
        got, _ = o.forward64(w, c["M"], c["Z"], c["d"], c["T"], c["B"], c["a"], c["b"],
                             c["indices"], c["offsets"])
        want = np.array(brute.forward(w, c["M"], c["Z"], c["d"], c["T"], c["B"], c["rows"],
                                      c["a"], c["b"], c["indices"], c["offsets"]))
        np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


def pin_gradient_brute(o, seed=1, cases=40):
    rng = np.random.default_rng(seed)
    for _ in range(cases):
        c = tiny_case(rng)
        g = rng.standard_normal((c["B"], c["T"] * c["d"])).astype(np.float32)
        G, A, cnt = o.gradient_dense(c["M"], c["Z"], c["d"], c["T"], c["B"], c["a"], c["b"],
                                     c["indices"], c["offsets"], g)
        Gw, cw = brute.gradient(c["M"], c["Z"], c["d"], c["T"], c["B"], c["rows"], c["a"],
                                c["b"], c["indices"], c["offsets"], g)
        np.testing.assert_allclose(G, Gw, rtol=1e-12, atol=1e-12)
        assert np.array_equal(cnt, np.array(cw))
        assert np.all(A >= np.abs(G) - 1e-12)


def pin_integer_forward(o, seed=2):
    # w[m] = m is exact in float32 for M = 4096; all pooled sums are integers
    # below 2^24, so the rounded output must equal brute force exactly.
    rng = np.random.default_rng(seed)
    for _ in range(6):
        c = tiny_case(rng, M=4096, d=8, Z=4, max_len=6)
        w = np.arange(4096, dtype=np.float32)
        got = o.forward(w, 4096, c["Z"], c["d"], c["T"], c["B"], c["a"], c["b"],
                        c["indices"], c["offsets"])
        want = np.array(brute.forward(w, 4096, c["Z"], c["d"], c["T"], c["B"], c["rows"],
                                      c["a"], c["b"], c["indices"], c["offsets"]))
        assert np.array_equal(got, want.astype(np.float32))
        assert np.array_equal(want, np.rint(want))


def pin_embedding_bag(o, seed=3):
    """Z = d, a = d, b = 0, M >= n*T*d: base(t, i) = d*(i*T + t), so rows are
    disjoint and PSS is a plain embedding table E[i*T + t] = w[d(iT+t) : +d]."""
    import torch
    rng = np.random.default_rng(seed)
    T, d, B, n = 3, 8, 5, 7
    M = n * T * d + 5
    lens = rng.integers(0, 4, T * B)
    offsets = np.zeros(T * B + 1, dtype=np.int64)
    np.cumsum(lens, out=offsets[1:])
    idx = rng.integers(0, n, int(offsets[-1])).astype(np.int64)
    w = rng.uniform(-1, 1, M).astype(np.float32)
    grad = rng.standard_normal((B, T * d)).astype(np.float32)
    lr, eps = 0.05, 1e-10

    table = torch.tensor(w[: n * T * d].astype(np.float64).reshape(n * T, d), requires_grad=True)
    t_of_item = np.repeat(np.arange(T * B) // B, lens)
    rows = torch.tensor(idx * T + t_of_item)
    pooled = torch.nn.functional.embedding_bag(rows, table, torch.tensor(offsets[:-1]), mode="sum")
    want = pooled.detach().numpy().reshape(T, B, d).transpose(1, 0, 2).reshape(B, T * d)
    got, _ = o.forward64(w, M, d, d, T, B, d, 0, idx, offsets)
    np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-15)

    g_t = torch.tensor(grad.astype(np.float64).reshape(B, T, d).transpose(1, 0, 2).reshape(T * B, d))
    (pooled * g_t).sum().backward()
    for opt_name in ("sgd", "adagrad"):
        p = torch.tensor(w.astype(np.float64).copy(), requires_grad=True)
        p.grad = torch.zeros_like(p)
        p.grad[: n * T * d] = table.grad.reshape(-1)
        s0 = np.full(M, 0.25, dtype=np.float32)
        if opt_name == "sgd":
            torch.optim.SGD([p], lr=lr).step()
            w_new, _, _, _, _ = o.backward_update(w, None, M, d, d, T, B, d, 0, idx, offsets, grad, lr)
        else:
            opt = torch.optim.Adagrad([p], lr=lr, eps=eps, initial_accumulator_value=0.25)
            opt.step()
            w_new, s_new, _, _, _ = o.backward_update(w, s0, M, d, d, T, B, d, 0, idx, offsets,
                                                      grad, lr, eps)
            s_want = opt.state[p]["sum"].numpy()
            np.testing.assert_allclose(s_new, s_want, rtol=2e-7, atol=0)
        np.testing.assert_allclose(w_new, p.detach().numpy(), rtol=2e-7, atol=1e-30)


def pin_mass(o, seed=4):
    rng = np.random.default_rng(seed)
    for _ in range(20):
        c = tiny_case(rng)
        M, Z, d, T, B = c["M"], c["Z"], c["d"], c["T"], c["B"]
        g = rng.standard_normal((B, T * d)).astype(np.float32)
        lens = np.diff(c["offsets"]).reshape(T, B)
        G, A, cnt = o.gradient_dense(M, Z, d, T, B, c["a"], c["b"], c["indices"], c["offsets"], g)
        # (i) total mass: every element of grad_out is deposited |bag| times
        g3 = g.astype(np.float64).reshape(B, T, d)
        total = sum(lens[t, bb] * g3[bb, t].sum() for t in range(T) for bb in range(B))
        assert abs(G.sum() - total) <= 1e-9 * (1 + np.abs(g3).sum() * lens.max())
        assert cnt.sum() == lens.sum() * d
        # (ii) per chunk offset k: columns c with c mod Z = k deposit into
        # h + k, so a mask of those columns carries exactly that mass
        w = rng.uniform(-1, 1, M).astype(np.float32)
        lr = 0.5
        for k in range(Z):
            mask = (np.arange(T * d) % d) % Z == k
            gk = np.where(mask[None, :], g, 0).astype(np.float32)
            Gk, Ak, _ = o.gradient_dense(M, Z, d, T, B, c["a"], c["b"], c["indices"], c["offsets"], gk)
            gk3 = gk.astype(np.float64).reshape(B, T, d)
            want = sum(lens[t, bb] * gk3[bb, t].sum() for t in range(T) for bb in range(B))
            w_new = o.sgd_update(w, Gk, lr)
            moved = (w.astype(np.float64) - w_new.astype(np.float64)).sum()
            assert abs(moved - lr * want) <= 1e-6 * (np.abs(w).sum() + lr * Ak.sum()) + 1e-12
        # (iii) grad_out = 1, w = 0, lr = 1  =>  w_new = -count (exact)
        ones = np.ones((B, T * d), dtype=np.float32)
        G1, _, _ = o.gradient_dense(M, Z, d, T, B, c["a"], c["b"], c["indices"], c["offsets"], ones)
        w_new = o.sgd_update(np.zeros(M, dtype=np.float32), G1, 1.0)
        _, cw = brute.gradient(M, Z, d, T, B, c["rows"], c["a"], c["b"], c["indices"],
                               c["offsets"], ones)
        assert np.array_equal(w_new, -np.array(cw, dtype=np.float32))


def pin_finite_difference(o, seed=5):
    rng = np.random.default_rng(seed)
    for _ in range(10):
        c = tiny_case(rng)
        M, Z, d, T, B = c["M"], c["Z"], c["d"], c["T"], c["B"]
        # values on a coarse dyadic grid keep every float64 sum exact
        w = (rng.integers(-64, 65, M) / 64.0).astype(np.float32)
        g = (rng.integers(-64, 65, (B, T * d)) / 64.0).astype(np.float32)
        G, _, _ = o.gradient_dense(M, Z, d, T, B, c["a"], c["b"], c["indices"], c["offsets"], g)
        base_out, _ = o.forward64(w, M, Z, d, T, B, c["a"], c["b"], c["indices"], c["offsets"])
        L0 = float((base_out * g).sum())
        for m in rng.choice(M, size=min(M, 8), replace=False):
            w2 = w.copy()
            w2[m] += 1.0
            out2, _ = o.forward64(w2, M, Z, d, T, B, c["a"], c["b"], c["indices"], c["offsets"])
            assert float((out2 * g).sum()) - L0 == G[m]


def pin_sparse_dense(o, seed=6):
    rng = np.random.default_rng(seed)
    for _ in range(20):
        c = tiny_case(rng)
        M, Z, d, T, B = c["M"], c["Z"], c["d"], c["T"], c["B"]
        g = rng.standard_normal((B, T * d)).astype(np.float32)
        G, _, _ = o.gradient_dense(M, Z, d, T, B, c["a"], c["b"], c["indices"], c["offsets"], g)
        loc, val = o.gradient_sparse(M, Z, d, T, B, c["a"], c["b"], c["indices"], c["offsets"], g)
        dense = np.zeros(M)
        dense[loc] = val
        np.testing.assert_allclose(dense, G, rtol=1e-12, atol=1e-12)
        assert np.all(np.diff(loc) > 0)


def pin_untouched(o, seed=8):
    rng = np.random.default_rng(seed)
    for _ in range(10):
        c = tiny_case(rng, M=64)
        M, Z, d, T, B = c["M"], c["Z"], c["d"], c["T"], c["B"]
        g = rng.standard_normal((B, T * d)).astype(np.float32)
        w = rng.uniform(-1, 1, M).astype(np.float32)
        s = rng.uniform(0, 1, M).astype(np.float32)
        _, cw = brute.gradient(M, Z, d, T, B, c["rows"], c["a"], c["b"], c["indices"], c["offsets"], g)
        untouched = np.array(cw) == 0
        w1, _, _, _, _ = o.backward_update(w, None, M, Z, d, T, B, c["a"], c["b"], c["indices"],
                                           c["offsets"], g, 0.1)
        w2, s2, _, _, _ = o.backward_update(w, s, M, Z, d, T, B, c["a"], c["b"], c["indices"],
                                            c["offsets"], g, 0.1, 1e-10)
        assert np.array_equal(w1[untouched].view(np.uint32), w[untouched].view(np.uint32))
        assert np.array_equal(w2[untouched].view(np.uint32), w[untouched].view(np.uint32))
        assert np.array_equal(s2[untouched].view(np.uint32), s[untouched].view(np.uint32))
        assert not np.array_equal(w1[~untouched], w[~untouched]) or (~untouched).sum() == 0


def pin_bf16_rounding(o, seed=9):
    import torch
    rng = np.random.default_rng(seed)
    vals = [rng.standard_normal(20000).astype(np.float32),
            (rng.standard_normal(2000) * 1e-39).astype(np.float32),        # subnormals
            np.array([0.0, -0.0, np.inf, -np.inf, 3.3895314e38, -3.3895314e38,
                      3.4028235e38, 1e-45, -1e-45, 1.0 + 2**-8, 1.0 + 3 * 2**-8,
                      1.0 - 2**-9, 2**-126, 2**-133, 2**-134, 3 * 2**-135], dtype=np.float32)]
    # exact ties: bf16 values plus half an ulp
    base = (rng.integers(0, 2**15, 4000).astype(np.uint32) << 16)
    ties = (base | 0x8000).view(np.float32)
    vals.append(ties[np.isfinite(ties)])
    x = np.concatenate(vals)
    got = o.round_to_bf16_bits(x.astype(np.float64))
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, want)
    nan = o.round_to_bf16_bits(np.array([np.nan]))
    assert (int(nan[0]) & 0x7F80) == 0x7F80 and (int(nan[0]) & 0x7F) != 0


def pin_bf16_widening(o):
    """bfloat16 storage widened to a float (the weights every bf16 forward and
    update reads): all 65,536 bit patterns (+-0, subnormals, +-inf, NaN
    payloads, max-finite) against torch's own bfloat16 -> float32 conversion,
    bit for bit."""
    import torch
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    got = np.asarray(o.widen(bits, o.BF16), dtype=np.float64)
    ref32 = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).float().numpy()
    want = ref32.astype(np.float64)
    assert np.array_equal(got.view(np.uint64), want.view(np.uint64))
    # the sign bit alone distinguishes +-0 and the two halves of the table
    assert np.signbit(got[0x8000]) and not np.signbit(got[0]) and got[0x8000] == 0.0
    assert got[0x7F7F] == np.float64(np.float32(3.3895314e38)) and np.isinf(got[0x7F80])


def pin_compress(o, seed=10):
    """M = S E and (S e_i)^T M against the explicit S; the injective case;
    eps of Def. 2 as the supremum it is defined to be; Thm. 1."""
    rng = np.random.default_rng(seed)
    for _ in range(25):
        T = int(rng.integers(1, 4))
        n = int(rng.integers(1, 7))
        d = int(rng.choice([1, 2, 4, 6, 8]))
        Z = int(rng.choice([z for z in range(1, d + 1) if d % z == 0]))
        M = int(rng.integers(max(Z, 2), 48))
        a, b = int(rng.integers(1, P)), int(rng.integers(0, P))
        E = rng.standard_normal((T, n, d))
        Mv, Mabs = o.compress(E, M, Z, a, b)
        want = np.array(brute.compress(E.tolist(), M, Z, a, b))
        assert np.all(np.abs(Mv - want) <= 1e-12 * (1 + Mabs))
        w = rng.uniform(-1, 1, M).astype(np.float32)
        V = brute.virtual_table(w, M, Z, d, T, [n] * T, a, b)
        R = o.recover(w, M, Z, d, T, n, a, b)
        for t in range(T):
            for i in range(n):
                assert np.array_equal(R[t, i], np.array(V[(t, i)]))
        # Def. 2: |<R_i - E_i, x>| <= eps_i ||x|| for every x, equality at x = R_i - E_i
        eps = o.pss_row_error(E, R)
        for t in range(T):
            for i in range(n):
                D = R[t, i] - E[t, i]
                for x in list(rng.standard_normal((4, d))) + [D]:
                    nx = np.sqrt((x * x).sum())
                    if nx > 0:
                        assert abs(D @ x) <= eps[t, i] * nx * (1 + 1e-12) + 1e-300
                assert abs(D @ D - eps[t, i] ** 2) <= 1e-12 * (1 + D @ D)
        # Thm. 1: pairwise distances move by at most eps_i + eps_j
        R2, E2, e2 = R.reshape(T * n, d), E.reshape(T * n, d), eps.ravel()
        for p_ in range(T * n):
            for q in range(T * n):
                gap = abs(np.linalg.norm(R2[p_] - R2[q]) - np.linalg.norm(E2[p_] - E2[q]))
                assert gap <= e2[p_] + e2[q] + 1e-12
    # injective special case: Z = d, a = Z, b = 0, M = n T Z puts the row of
    # (t, i) at Z (i T + t): compression is a permutation and recovery exact
    T, n, d = 3, 5, 4
    E = rng.standard_normal((T, n, d)).astype(np.float32)
    M = n * T * d
    Mv, _ = o.compress(E, M, d, d, 0)
    for t in range(T):
        for i in range(n):
            assert np.array_equal(Mv[d * (i * T + t): d * (i * T + t) + d], E[t, i].astype(np.float64))
    R = o.recover(Mv.astype(np.float32), M, d, d, T, n, d, 0)
    assert np.array_equal(R, E.astype(np.float64))
    assert np.all(o.pss_row_error(E, R) == 0)


def pin_sign_and_mean(o, seed=11):
    """Sign variants (Sec. 2.5 Achlioptas-type entries from a second hash)
    and mean pooling against the pure-Python sketch with signed entries;
    torch's mean embedding_bag in the injective case; the published
    SplitMix64 stream behind (a2, b2); the frequencies of the factors."""
    import torch
    # SplitMix64 from state 0, outputs 2..4 (java.util.SplittableRandom(0))
    assert o.splitmix64(0, 4)[1:] == [0x6E789E6AA1B965F4, 0x06C45D188009454F, 0xF88BB8A8724C81EC]
    assert o.sign_params_from_seed(0) == (1 + 0x06C45D188009454F % (P - 1), 0xF88BB8A8724C81EC % P)
    rng = np.random.default_rng(seed)
    for k in range(36):
        c = tiny_case(rng)
        M, Z, d, T, B = c["M"], c["Z"], c["d"], c["T"], c["B"]
        mode = [None, o.SIGN_PM1, o.SIGN_SPARSE][k % 3]
        mean = bool((k // 3) % 2)
        a2, b2 = int(rng.integers(1, P)), int(rng.integers(0, P))
        sign = None if mode is None else (mode, a2, b2)
        bsign = None if mode is None else (mode, a2, b2)
        w = (rng.standard_normal(M) * 0.5).astype(np.float32)
        got, s_abs = o.forward64(w, M, Z, d, T, B, c["a"], c["b"], c["indices"], c["offsets"],
                                 sign=sign, mean=mean)
        want = np.array(brute.forward(w, M, Z, d, T, B, c["rows"], c["a"], c["b"], c["indices"],
                                      c["offsets"], sign=bsign, mean=mean))
        np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)
        assert np.all(s_abs >= np.abs(got) - 1e-12)
        g = rng.standard_normal((B, T * d)).astype(np.float32)
        G, A, cnt = o.gradient_dense(M, Z, d, T, B, c["a"], c["b"], c["indices"], c["offsets"], g,
                                     sign=sign, mean=mean)
        Gw, cw = brute.gradient(M, Z, d, T, B, c["rows"], c["a"], c["b"], c["indices"],
                                c["offsets"], g, sign=bsign, mean=mean)
        np.testing.assert_allclose(G, Gw, rtol=1e-12, atol=1e-12)
        loc, val = o.gradient_sparse(M, Z, d, T, B, c["a"], c["b"], c["indices"], c["offsets"], g,
                                     sign=sign, mean=mean)
        assert np.array_equal(loc, np.nonzero(cnt)[0])
        np.testing.assert_allclose(val, G[loc], rtol=1e-12, atol=1e-12)
        where = rng.choice(M, size=min(M, 9), replace=False)
        Ga, Aa, ca = o.gradient_at(M, Z, d, T, B, c["a"], c["b"], c["indices"], c["offsets"], g,
                                   where, sign=sign, mean=mean)
        np.testing.assert_allclose(Ga, G[where], rtol=1e-12, atol=1e-12)
        assert np.array_equal(ca, cnt[where])
        # brute's reads count the zero entries of S too; the oracle drops them
        if mode != o.SIGN_SPARSE:
            assert np.array_equal(cnt, np.array(cw))
        bags = rng.choice(T * B, size=min(T * B, 4), replace=False)
        fa, _ = o.forward_at(w, M, Z, d, T, B, c["a"], c["b"], c["indices"], c["offsets"], bags,
                             sign=sign, mean=mean)
        full = got.reshape(B, T, d).transpose(1, 0, 2).reshape(T * B, d)
        np.testing.assert_allclose(fa, full[bags], rtol=1e-12, atol=1e-12)
    # factor frequencies over many keys: 1/2 each for pm1; 1/6, 1/6, 2/3 for sparse
    n = 300_000
    idx = rng.integers(0, 2**31, n)
    t = rng.integers(0, 26, n)
    for mode, want in ((o.SIGN_PM1, {1: 0.5, -1: 0.5, 0: 0.0}),
                       (o.SIGN_SPARSE, {1: 1 / 6, -1: 1 / 6, 0: 2 / 3})):
        f = o.signs_for(1, 4, 26, 987654321, 123456789, idx, t, mode)
        for v, frac in want.items():
            assert abs((f == v).mean() - frac) < 0.004, (mode, v, (f == v).mean())
        # independent of the location hash: factor vs low bit of the base
        base = o.bases_for(4096, 1, 4, 26, 55555, 777, idx, t)
        for v, frac in want.items():
            if frac:
                both = ((f == v) & (base % np.uint64(2) == 0)).mean()
                assert abs(both - frac / 2) < 0.004
    # injective layout: mean pooling == torch embedding_bag(mode="mean"),
    # and its weight gradient
    T, d, B, nr = 3, 8, 5, 7
    M = nr * T * d + 5
    lens = rng.integers(0, 4, T * B)
    offsets = np.zeros(T * B + 1, dtype=np.int64)
    np.cumsum(lens, out=offsets[1:])
    idx = rng.integers(0, nr, int(offsets[-1])).astype(np.int64)
    w = rng.uniform(-1, 1, M).astype(np.float32)
    grad = rng.standard_normal((B, T * d)).astype(np.float32)
    table = torch.tensor(w[: nr * T * d].astype(np.float64).reshape(nr * T, d), requires_grad=True)
    t_of_item = np.repeat(np.arange(T * B) // B, lens)
    rows = torch.tensor(idx * T + t_of_item)
    pooled = torch.nn.functional.embedding_bag(rows, table, torch.tensor(offsets[:-1]), mode="mean")
    want = pooled.detach().numpy().reshape(T, B, d).transpose(1, 0, 2).reshape(B, T * d)
    got, _ = o.forward64(w, M, d, d, T, B, d, 0, idx, offsets, mean=True)
    np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-15)
    g_t = torch.tensor(grad.astype(np.float64).reshape(B, T, d).transpose(1, 0, 2).reshape(T * B, d))
    (pooled * g_t).sum().backward()
    G, _, _ = o.gradient_dense(M, d, d, T, B, d, 0, idx, offsets, grad, mean=True)
    np.testing.assert_allclose(G[: nr * T * d], table.grad.numpy().reshape(-1), rtol=1e-12,
                               atol=1e-15)
    assert np.all(G[nr * T * d:] == 0)


ALL_PINS = [pin_hash_vectors, pin_forward_brute, pin_gradient_brute, pin_integer_forward,
            pin_embedding_bag, pin_mass, pin_finite_difference, pin_sparse_dense,
            pin_untouched, pin_bf16_rounding, pin_bf16_widening, pin_compress,
            pin_sign_and_mean]
