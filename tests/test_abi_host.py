"""The C-ABI library on the host: loads, exports what include/pss.h declares,
rejects bad arguments before touching a GPU, and its hash code (compiled for
the host from the same source the kernels use) agrees with the oracle."""
import ctypes

import numpy as np
import pytest

import synth
from oracle import pss_oracle as o
from paper_2207_10731_amd import pss

P = 2**31 - 1


@pytest.fixture(scope="module")
def lib():
    return pss.load_library()


def test_exports_every_declared_function(lib):
    names = pss.header_functions([pss.HEADER])
    assert {"pss_forward", "pss_backward_update", "pss_debug_addresses",
            "pss_hash_params_from_seed", "pss_status_string"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n


def test_measurement_library_is_separate(lib):
    """include/pss_bench.h is served by libpss_bench.so; the layer's library
    exports none of it."""
    import os
    bench = pss.load_bench_library()
    names = pss.header_functions([os.path.join(pss.INCLUDE, "pss_bench.h")])
    assert {"pss_bench_copy", "pss_bench_read", "pss_bench_gather"} <= set(names)
    for n in names:
        assert hasattr(bench, n), n
        assert not hasattr(lib, n), n
    assert set(pss.header_functions()) == set(names) | set(pss.header_functions([pss.HEADER]))


def test_flag_layout(lib):
    """Backward variant in bits 0-1, options in bits 2-8; the sign field value
    3 << 2 and any bit from 9 up are rejected before anything is enqueued."""
    assert pss.PSS_BWD_MASK == 3
    opts = [pss.PSS_SIGN_PM1, pss.PSS_SIGN_SPARSE, pss.PSS_POOL_MEAN, pss.PSS_INDEX_I32,
            pss.PSS_ROWS_BF16, pss.PSS_PREPARE_BACKWARD, pss.PSS_DEPOSIT_BY_ADDRESS]
    for f in opts:
        assert f & 3 == 0 and f < (1 << 9)
    assert pss.PSS_SIGN_MASK == 3 << 2
    hp = pss.make_hash_params(1, num_tables=1, batch=1, num_indices=1)
    for bad in [pss.PSS_SIGN_MASK, 1 << 9, 1 << 31]:
        hp.flags = bad
        st = lib.pss_forward(ctypes.c_void_p(8), 4096, 4, 16, ctypes.byref(hp), ctypes.c_void_p(8),
                             ctypes.c_void_p(8), ctypes.c_void_p(8), None)
        assert st == pss.PSS_ERR_INVALID_ARG, bad


def test_status_strings(lib):
    for s in range(6):
        assert pss.status_string(s) and pss.status_string(s) != "unknown status"
    assert pss.status_string(99) == "unknown status"


@pytest.mark.parametrize("seed", [0, 1, 2, 3, 4, 5, 42, 2**64 - 1, 123456789])
def test_hash_params_from_seed_matches_oracle(seed):
    hp = pss.make_hash_params(seed, num_tables=1, batch=1, num_indices=0)
    assert (hp.a, hp.b) == o.hash_params_from_seed(seed)
    assert (hp.sign_a, hp.sign_b) == o.sign_params_from_seed(seed)


@pytest.mark.parametrize("mode", ["pm1", "sparse"])
def test_host_signs_match_oracle(mode):
    """The kernels' route to the sign (second hash recovered from the item
    hash by an affine map mod p) against the oracle's direct evaluation."""
    flag = pss.PSS_SIGN_PM1 if mode == "pm1" else pss.PSS_SIGN_SPARSE
    rng = np.random.default_rng(11)
    for k in range(40):
        M = int(rng.choice([1, 7, 4096, 2_500_000, 10**9, P]))
        T = int(rng.choice([1, 3, 26]))
        Z = min(int(rng.choice([1, 2, 4])), M)
        d = Z * int(rng.choice([1, 2, 32]))
        B = int(rng.integers(1, 6))
        lens = rng.integers(0, 5, T * B)
        off = np.zeros(T * B + 1, dtype=np.int64)
        np.cumsum(lens, out=off[1:])
        n = int(off[-1])
        idx = rng.integers(0, 2**31, n).astype(np.int64)
        if k % 5 == 0:
            idx[: n // 2] = rng.choice([0, 1, P - 1, P, 2**31 - 1], n // 2)
        a = int(rng.choice([1, 2, P - 1, int(rng.integers(1, P))]))
        b = int(rng.choice([0, P - 1, int(rng.integers(0, P))]))
        a2 = int(rng.choice([1, P - 1, int(rng.integers(1, P))]))
        b2 = int(rng.choice([0, P - 1, int(rng.integers(0, P))]))
        hp = pss.make_hash_params(a=a, b=b, sign_a=a2, sign_b=b2, num_tables=T, batch=B,
                                  num_indices=n, flags=flag)
        got = pss.pss_hash_signs_host(M, Z, d, hp, idx, off)
        _, t, _ = o.item_bags(T, B, off)
        want = o.signs_for(Z, d, T, a2, b2, idx, t, mode)
        assert np.array_equal(got.astype(np.int64), want), (k, a, b, a2, b2)
    # without a sign option every factor is +1
    hp = pss.make_hash_params(3, num_tables=1, batch=2, num_indices=3)
    assert np.all(pss.pss_hash_signs_host(64, 4, 8, hp, np.array([1, 2, 3]),
                                          np.array([0, 1, 3])) == 1)


def _host_bases(M, Z, d, T, B, a, b, idx, off):
    hp = pss.make_hash_params(a=a, b=b, num_tables=T, batch=B, num_indices=len(idx))
    return pss.pss_hash_bases_host(M, Z, d, hp, idx, off)


@pytest.mark.parametrize("key", ["c1", "c2", "c3", "c4", "c5"])
def test_host_hash_matches_oracle_on_workloads(key):
    wl = synth.get(key)
    x = synth.make_inputs(wl, B=96)
    a, b = o.hash_params_from_seed(wl.hash_seed)
    got = _host_bases(wl.M, wl.Z, wl.d, wl.T, 96, a, b, x.indices, x.offsets)
    want = o.chunk_bases(wl.M, wl.Z, wl.d, wl.T, 96, a, b, x.indices, x.offsets)
    assert np.array_equal(got.astype(np.uint64), want)


def test_host_hash_random_parameters_and_extremes():
    rng = np.random.default_rng(3)
    for _ in range(60):
        M = int(rng.choice([1, 2, 3, 7, 4096, 2_500_000, 16_000_000, 64_000_000, 10**9, P,
                            int(rng.integers(1, P + 1))]))
        T = int(rng.choice([1, 3, 26, 1000]))
        Z = int(rng.choice([1, 2, 4]))
        Z = min(Z, M)
        d = Z * int(rng.choice([1, 2, 32]))
        B = int(rng.integers(1, 6))
        lens = rng.integers(0, 4, T * B)
        off = np.zeros(T * B + 1, dtype=np.int64)
        np.cumsum(lens, out=off[1:])
        n = int(off[-1])
        idx = rng.choice(np.array([0, 1, P - 1, P, 2**31 - 1, 2**30]), n) if rng.random() < 0.3 \
            else rng.integers(0, 2**31, n)
        idx = idx.astype(np.int64)
        a = int(rng.choice([1, 2, P - 1, int(rng.integers(1, P))]))
        b = int(rng.choice([0, P - 1, int(rng.integers(0, P))]))
        got = _host_bases(M, Z, d, T, B, a, b, idx, off)
        want = o.chunk_bases(M, Z, d, T, B, a, b, idx, off)
        assert np.array_equal(got.astype(np.uint64), want), (M, T, Z, d, a, b)


@pytest.mark.parametrize("M", [1, 2, 3, 4096, 65536, 2_500_000, 16_000_000, 64_000_000,
                               1_000_000_000, P - 1, P, 1 << 30, (1 << 30) + 1, 1_000_000_007])
def test_host_fast_mod(M):
    # a = 1, b = 0, T = C = 1: the base is (i mod p) mod M, so for i < p this
    # checks the library's remainder by M directly against NumPy's.
    rng = np.random.default_rng(M % 1000)
    vals = np.concatenate([rng.integers(0, P, 200_000),
                           np.array([0, 1, P - 1, P - 2, M - 1, M, M + 1, 2 * M - 1, 2 * M]),
                           (np.arange(1, 200) * M - 1), (np.arange(1, 200) * M)])
    vals = vals[(vals >= 0) & (vals < P)].astype(np.int64)
    off = np.array([0, vals.shape[0]], dtype=np.int64)
    got = _host_bases(M, 1, 1, 1, 1, 1, 0, vals, off)[:, 0]
    assert np.array_equal(got.astype(np.int64), vals % M)


def _bad_call(lib, **kw):
    args = dict(M=4096, Z=4, d=16, a=5, b=7, T=4, B=2, N=8, dtype=0, flags=0, eps=1e-10,
                sign_a=3, sign_b=11)
    args.update(kw)
    hp = pss.pss_hash_params(args["a"], args["b"], args["T"], args["B"], args["N"], args["dtype"],
                             args["eps"], args["flags"], args["sign_a"], args["sign_b"])
    dummy = ctypes.c_void_p(0x1000)  # never dereferenced: checks fail before any use
    return lib.pss_forward(kw.get("shared", dummy), args["M"], args["Z"], args["d"],
                           ctypes.byref(hp), dummy, dummy, dummy, None)


@pytest.mark.parametrize("kw", [dict(M=0), dict(M=2**31), dict(Z=0), dict(Z=5000, M=4096),
                                dict(Z=3), dict(d=4097 * 4), dict(a=0), dict(a=P),
                                dict(b=P), dict(T=0), dict(B=0), dict(N=-1), dict(flags=1 << 9),
                                dict(flags=3 << 2), dict(flags=pss.PSS_SIGN_PM1, sign_a=0),
                                dict(flags=pss.PSS_SIGN_SPARSE, sign_a=P),
                                dict(flags=pss.PSS_SIGN_PM1, sign_b=P),
                                dict(flags=pss.PSS_INDEX_I32, N=2**31),
                                dict(T=2**31, Z=1, d=2), dict(shared=None)])
def test_forward_rejects_bad_arguments(lib, kw):
    assert _bad_call(lib, **kw) == pss.PSS_ERR_INVALID_ARG


def test_forward_rejects_unknown_dtype(lib):
    assert _bad_call(lib, dtype=7) == pss.PSS_ERR_UNSUPPORTED


def test_backward_rejects_bad_arguments(lib):
    dummy = ctypes.c_void_p(0x1000)
    hp = pss.pss_hash_params(5, 7, 4, 2, 8, 0, 1e-10, 0)
    f = lib.pss_backward_update
    assert f(dummy, None, 4096, 4, 16, ctypes.byref(hp), dummy, dummy, dummy,
             ctypes.c_float(float("nan")), None) == pss.PSS_ERR_INVALID_ARG
    assert f(dummy, None, 4096, 4, 16, ctypes.byref(hp), dummy, dummy, None,
             ctypes.c_float(0.1), None) == pss.PSS_ERR_INVALID_ARG
    hp_neg = pss.pss_hash_params(5, 7, 4, 2, 8, 0, -1.0, 0)
    assert f(dummy, dummy, 4096, 4, 16, ctypes.byref(hp_neg), dummy, dummy, dummy,
             ctypes.c_float(0.1), None) == pss.PSS_ERR_INVALID_ARG
    hp4 = pss.pss_hash_params(5, 7, 4, 2, 8, 0, 1e-10, 1 << 9)
    assert f(dummy, None, 4096, 4, 16, ctypes.byref(hp4), dummy, dummy, dummy,
             ctypes.c_float(0.1), None) == pss.PSS_ERR_INVALID_ARG


def test_gradient_sparse_rejects_bad_arguments(lib):
    dummy = ctypes.c_void_p(0x1000)
    f = lib.pss_gradient_sparse
    hp = pss.pss_hash_params(5, 7, 4, 2, 8, 0, 1e-10, 0)
    # capacity below min(M, N*d) = min(4096, 128)
    assert f(4096, 4, 16, ctypes.byref(hp), dummy, dummy, dummy, dummy, dummy, 127, dummy,
             None) == pss.PSS_ERR_INVALID_ARG
    assert f(4096, 4, 16, ctypes.byref(hp), dummy, dummy, dummy, dummy, dummy, 128, None,
             None) == pss.PSS_ERR_INVALID_ARG
    big = pss.pss_hash_params(5, 7, 4, 2, 2**30, 0, 1e-10, 0)  # N*C = 2^32
    assert f(4096, 4, 16, ctypes.byref(big), dummy, dummy, dummy, dummy, dummy, 4096, dummy,
             None) == pss.PSS_ERR_UNSUPPORTED


def test_offsets_validator():
    assert pss.pss_validate_offsets_host(np.array([0, 1, 1, 3]), 3, 3) == pss.PSS_OK
    assert pss.pss_validate_offsets_host(np.array([0, 2, 1, 3]), 3, 3) == pss.PSS_ERR_INVALID_ARG
    assert pss.pss_validate_offsets_host(np.array([1, 2, 2, 3]), 3, 3) == pss.PSS_ERR_INVALID_ARG
    assert pss.pss_validate_offsets_host(np.array([0, 1, 2, 3]), 3, 4) == pss.PSS_ERR_INVALID_ARG
    # shorter than num_bags + 1 entries: rejected before the library reads it
    assert pss.pss_validate_offsets_host(np.array([0, 1, 3]), 3, 3) == pss.PSS_ERR_INVALID_ARG


def test_host_hash_rejects_short_arrays():
    """The host hash entry points read N indices and T*B + 1 offsets: the
    binding refuses arrays shorter than the sizes the parameters declare."""
    hp = pss.make_hash_params(7, num_tables=2, batch=3, num_indices=6)
    idx = np.arange(6)
    off = np.arange(7)
    for fn in (pss.pss_hash_bases_host, pss.pss_hash_signs_host):
        assert fn(64, 4, 8, hp, idx, off).shape == (6, 2)
        with pytest.raises(ValueError):
            fn(64, 4, 8, hp, idx[:5], off)
        with pytest.raises(ValueError):
            fn(64, 4, 8, hp, idx, off[:6])


def test_prepare_rejects_bad_arguments(lib):
    """pss_prepare_backward checks its arguments on the host before anything
    is enqueued (the dummy pointers are never dereferenced)."""
    dummy = ctypes.c_void_p(0x1000)

    def call(M=4096, Z=4, d=16, a=5, T=4, B=2, N=8, offsets=dummy):
        hp = pss.pss_hash_params(a, 7, T, B, N, 0, 1e-10, 0, 3, 11)
        return lib.pss_prepare_backward(M, Z, d, ctypes.byref(hp), dummy, offsets, None)

    assert call(M=0) == pss.PSS_ERR_INVALID_ARG
    assert call(Z=5) == pss.PSS_ERR_INVALID_ARG  # Z does not divide d
    assert call(a=0) == pss.PSS_ERR_INVALID_ARG
    assert call(T=0) == pss.PSS_ERR_INVALID_ARG
    assert call(offsets=None) == pss.PSS_ERR_INVALID_ARG


def test_noalloc_rejects_bad_arguments_and_oversized_calls(lib):
    """The allocation-free backward runs the same host checks, and refuses a
    call whose scratch exceeds its static array before anything is enqueued
    (no GPU is touched: the pointers are never dereferenced)."""
    dummy = ctypes.c_void_p(0x1000)
    f = lib.pss_backward_update_noalloc
    hp = pss.pss_hash_params(5, 7, 4, 2, 8, 0, 1e-10, 0)
    assert f(dummy, None, 4096, 4, 16, ctypes.byref(hp), dummy, dummy, dummy,
             ctypes.c_float(float("nan")), None) == pss.PSS_ERR_INVALID_ARG
    assert f(None, None, 4096, 4, 16, ctypes.byref(hp), dummy, dummy, dummy,
             ctypes.c_float(0.1), None) == pss.PSS_ERR_INVALID_ARG
    # SORTED grouping of 4.2M lookups: 16 B each, beyond 64 MiB
    big = pss.pss_hash_params(5, 7, 26, 262144, 26 * 262144, 0, 1e-10, pss.PSS_BWD_SORTED)
    assert f(dummy, None, 2_500_000, 32, 128, ctypes.byref(big), dummy, dummy, dummy,
             ctypes.c_float(0.1), None) == pss.PSS_ERR_SCRATCH_LIMIT
    # an unfused update needs a float32 gradient buffer of M: 64 MiB + 4 B is too much
    hp_m = pss.pss_hash_params(5, 7, 1, 1, 1, 0, 1e-10, pss.PSS_BWD_ATOMIC)
    M = (pss.PSS_NOALLOC_SCRATCH_BYTES // 4) + 1
    assert f(dummy, dummy, M, 4, 16, ctypes.byref(hp_m), dummy, dummy, dummy,
             ctypes.c_float(0.1), None) == pss.PSS_ERR_SCRATCH_LIMIT
    assert "allocation-free" in pss.status_string(pss.PSS_ERR_SCRATCH_LIMIT)
    # no lookups: nothing to do, whatever the size
    hp0 = pss.pss_hash_params(5, 7, 26, 262144, 0, 0, 1e-10, 0)
    assert f(dummy, None, 2_500_000, 32, 128, ctypes.byref(hp0), dummy, dummy, dummy,
             ctypes.c_float(0.1), None) == pss.PSS_OK


def test_by_address_flag_rules(lib):
    """PSS_DEPOSIT_BY_ADDRESS is refused with ATOMIC or SPARSE and beyond
    2^31 (lookup, dim) records, on the host before anything is enqueued; the
    run-sum form's scratch (N x d floats of run sums) counts against the
    allocation-free entry point's limit."""
    dummy = ctypes.c_void_p(0x1000)
    f = lib.pss_backward_update
    A = pss.PSS_DEPOSIT_BY_ADDRESS
    for variant in (pss.PSS_BWD_ATOMIC, pss.PSS_BWD_SPARSE):
        hp = pss.pss_hash_params(5, 7, 4, 2, 8, 0, 1e-10, variant | A)
        assert f(dummy, None, 4096, 4, 16, ctypes.byref(hp), dummy, dummy, dummy,
                 ctypes.c_float(0.1), None) == pss.PSS_ERR_UNSUPPORTED
    for Z in (1, 128):  # single contributions, run sums
        big = pss.pss_hash_params(5, 7, 1, 2**24, 2**24, 0, 1e-10, pss.PSS_BWD_SORTED | A)
        assert f(dummy, None, 2_500_000, Z, 128, ctypes.byref(big), dummy, dummy, dummy,
                 ctypes.c_float(0.1), None) == pss.PSS_ERR_UNSUPPORTED
    # run sums of 200 K whole-row lookups: 102 MB of run sums, beyond 64 MiB
    runs = pss.pss_hash_params(5, 7, 1, 200_000, 200_000, 0, 1e-10, pss.PSS_BWD_SORTED | A)
    assert lib.pss_backward_update_noalloc(dummy, dummy, 2_500_000, 128, 128, ctypes.byref(runs),
                                           dummy, dummy, dummy, ctypes.c_float(0.1),
                                           None) == pss.PSS_ERR_SCRATCH_LIMIT


def test_reduce_events_hook_rules(lib):
    """The timing hook takes both events or neither (no GPU work: it only
    stores the handles; they are cleared again before the test ends)."""
    fake = ctypes.c_void_p(0x1000)
    assert lib.pss_debug_reduce_events(fake, None) == pss.PSS_ERR_INVALID_ARG
    assert lib.pss_debug_reduce_events(None, fake) == pss.PSS_ERR_INVALID_ARG
    assert lib.pss_debug_reduce_events(None, None) == pss.PSS_OK
    with pytest.raises(ValueError):
        pss.pss_debug_reduce_events(0, 0)
    pss.pss_debug_reduce_events()
