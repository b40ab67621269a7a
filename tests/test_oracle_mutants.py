"""Plant plausible mistakes in the CPU oracle and require a pin to catch each.

Every mutant replaces one function of ``oracle.pss_oracle`` (on the CPU, for
the duration of one test) with a version carrying a single typical slip: a
dropped term, a wrong sign or index, a transposed layout, a missing wrap.
The pins must reject every one of them.
"""
import numpy as np
import pytest

from oracle import pss_oracle as o
import pins

P = o.P


def _bases_drop_b(M, Z, d, T, a, b, idx, t):
    C = d // Z
    i = np.asarray(idx, dtype=np.int64).astype(np.uint64)
    tt = np.asarray(t, dtype=np.int64).astype(np.uint64)
    key = (i * np.uint64(T) + tt)[:, None] * np.uint64(C) + np.arange(C, dtype=np.uint64)[None, :]
    h = (np.uint64(a) * (key % np.uint64(P))) % np.uint64(P)          # "+ b" dropped
    return h % np.uint64(M)


def _bases_swapped_key(M, Z, d, T, a, b, idx, t):
    C = d // Z
    i = np.asarray(idx, dtype=np.int64).astype(np.uint64)
    tt = np.asarray(t, dtype=np.int64).astype(np.uint64)
    key = (tt * np.uint64(T) + i)[:, None] * np.uint64(C) + np.arange(C, dtype=np.uint64)[None, :]
    h = (np.uint64(a) * (key % np.uint64(P)) + np.uint64(b)) % np.uint64(P)
    return h % np.uint64(M)


def _bases_no_mersenne(M, Z, d, T, a, b, idx, t):
    # forgets the mod p step: ((a*key + b) mod 2^64) mod M
    C = d // Z
    i = np.asarray(idx, dtype=np.int64).astype(np.uint64)
    tt = np.asarray(t, dtype=np.int64).astype(np.uint64)
    key = (i * np.uint64(T) + tt)[:, None] * np.uint64(C) + np.arange(C, dtype=np.uint64)[None, :]
    with np.errstate(over="ignore"):
        h = np.uint64(a) * key + np.uint64(b)
    return h % np.uint64(M)


def _addr_no_wrap(M, Z, base):
    base = np.asarray(base).astype(np.int64)
    addr = np.minimum(base[:, :, None] + np.arange(Z)[None, None, :], M - 1)
    return addr.reshape(base.shape[0], base.shape[1] * Z)


def _addr_reversed_offset(M, Z, base):
    base = np.asarray(base).astype(np.int64)
    addr = (base[:, :, None] + (Z - 1 - np.arange(Z))[None, None, :]) % M
    return addr.reshape(base.shape[0], base.shape[1] * Z)


def _item_bags_sample_major(T, B, offsets):
    offsets = np.asarray(offsets, dtype=np.int64)
    g = np.repeat(np.arange(T * B, dtype=np.int64), np.diff(offsets))
    return g, g % T, g // T                                              # bag = b*T + t misread


def _sgd_wrong_sign(w, G, lr, weight_dtype=o.F32):
    return o.round_storage(o.widen(w, weight_dtype) + lr * G, weight_dtype)


def _adagrad_old_state(w, s, G, lr, eps, weight_dtype=o.F32):
    w64 = o.widen(w, weight_dtype)
    s64 = np.asarray(s, dtype=np.float32).astype(np.float64)
    w_new = w64 - lr * G / (np.sqrt(s64) + eps)                          # uses s before the update
    return o.round_storage(w_new, weight_dtype), (s64 + G * G).astype(np.float32)


def _bf16_truncate(x):
    x32 = np.asarray(x, dtype=np.float64).astype(np.float32)
    return (x32.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


_orig_widen = o.widen


def _widen_bf16_drops_sign(w, weight_dtype=o.F32):
    if weight_dtype != o.BF16:
        return _orig_widen(w, weight_dtype)
    bits = (np.asarray(w, dtype=np.uint16).astype(np.uint32) & np.uint32(0x7FFF)) << np.uint32(16)
    return bits.view(np.float32).astype(np.float64)                     # sign bit dropped


def _widen_bf16_shift15(w, weight_dtype=o.F32):
    if weight_dtype != o.BF16:
        return _orig_widen(w, weight_dtype)
    bits = np.asarray(w, dtype=np.uint16).astype(np.uint32) << np.uint32(15)
    return bits.view(np.float32).astype(np.float64)                     # off by one bit


_orig_contrib = o._contributions


def _gradient_last_write_wins(M, Z, d, T, B, a, b, indices, offsets, grad_out, sign=None,
                              mean=False):
    addr, g = _orig_contrib(M, Z, d, T, B, a, b, indices, offsets, grad_out, sign, mean)
    G = np.zeros(M)
    G[addr] = g                                                          # no accumulation
    A = np.zeros(M)
    A[addr] = np.abs(g)
    return G, A, np.bincount(addr, minlength=M)


def _compress_overwrites(E, M, Z, a, b):
    E64 = np.asarray(E, dtype=np.float64)
    T, n, d = E64.shape
    addr = o.table_addresses(M, Z, d, T, n, a, b).ravel()
    Mv = np.zeros(M)
    Mv[addr] = E64.ravel()                                               # collisions overwrite
    Mabs = np.zeros(M)
    Mabs[addr] = np.abs(E64).ravel()
    return Mv, Mabs


def _recover_token_major(w, M, Z, d, T, n, a, b, weight_dtype=o.F32):
    addr = o.table_addresses(M, Z, d, T, n, a, b)
    # reads the (t, i) address block as if it were laid out [n, T, d]
    return o.widen(w, weight_dtype)[addr.reshape(n, T, d).transpose(1, 0, 2)]


def _row_error_squared(E, R):
    D = np.asarray(R, dtype=np.float64) - np.asarray(E, dtype=np.float64)
    return np.sum(D * D, axis=-1)                                        # sqrt dropped


def _signs_threshold_third(Z, d, T, a2, b2, idx, t, mode):
    f = _orig_signs(Z, d, T, a2, b2, idx, t, mode)
    if mode != o.SIGN_SPARSE:
        return f
    C = d // Z
    i = np.asarray(idx, dtype=np.int64).astype(np.uint64)
    tt = np.asarray(t, dtype=np.int64).astype(np.uint64)
    key = (i * np.uint64(T) + tt)[:, None] * np.uint64(C) + np.arange(C, dtype=np.uint64)[None, :]
    h2 = ((np.uint64(a2) * (key % np.uint64(P)) + np.uint64(b2)) % np.uint64(P)).astype(np.int64)
    q = P // 3                                                           # 1/3 instead of 1/6
    return np.where(h2 < q, 1, np.where(h2 < 2 * q, -1, 0)).astype(np.int64)


def _signs_per_item(Z, d, T, a2, b2, idx, t, mode):
    f = _orig_signs(Z, d, T, a2, b2, idx, t, mode)
    return np.repeat(f[:, :1], f.shape[1], axis=1)                       # chunk 0's sign for all


def _item_scale_ignores_mean(T, B, offsets, mean):
    return _orig_scale(T, B, offsets, False)


_orig_signs = o.signs_for
_orig_scale = o.item_scale


MUTANTS = {
    "hash_drops_b": ("bases_for", _bases_drop_b),
    "key_swaps_table_and_token": ("bases_for", _bases_swapped_key),
    "hash_skips_mod_p": ("bases_for", _bases_no_mersenne),
    "chunk_without_wrap": ("addresses_from_bases", _addr_no_wrap),
    "chunk_offset_reversed": ("addresses_from_bases", _addr_reversed_offset),
    "bags_read_sample_major": ("item_bags", _item_bags_sample_major),
    "sgd_wrong_sign": ("sgd_update", _sgd_wrong_sign),
    "adagrad_stale_accumulator": ("adagrad_update", _adagrad_old_state),
    "bf16_truncates": ("round_to_bf16_bits", _bf16_truncate),
    "scatter_without_accumulation": ("gradient_dense", _gradient_last_write_wins),
    "compress_overwrites": ("compress", _compress_overwrites),
    "recover_token_major": ("recover", _recover_token_major),
    "row_error_squared": ("pss_row_error", _row_error_squared),
    "sparse_signs_at_one_third": ("signs_for", _signs_threshold_third),
    "one_sign_per_item": ("signs_for", _signs_per_item),
    "gradient_ignores_mean": ("item_scale", _item_scale_ignores_mean),
    "bf16_widen_drops_sign": ("widen", _widen_bf16_drops_sign),
    "bf16_widen_shift_15": ("widen", _widen_bf16_shift15),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_mutant(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(o, attr, fn)
    failed = []
    for pin in pins.ALL_PINS:
        try:
            pin(o)
        except (AssertionError, IndexError, ValueError):
            failed.append(pin.__name__)
    assert failed, f"mutant {name} passed every pin"
