"""Post-hoc compression M = S E and retrieval (S e_i)^T M (Sec. 2.4, Thm. 2)
on the GPU against the oracle."""
import numpy as np
import pytest
import torch

from oracle import pss_oracle as o
from paper_2207_10731_amd import pss

pytestmark = pytest.mark.gpu

CASES = [(3, 500, 16, 4, 997), (2, 2000, 128, 32, 40_000), (1, 300, 64, 64, 64),
         (4, 100, 8, 1, 333), (26, 50, 128, 128, 1_000_003), (1, 1, 4, 2, 2)]
VARIANTS = [pss.PSS_BWD_SPARSE, pss.PSS_BWD_SORTED, pss.PSS_BWD_ATOMIC]


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("T,n,d,Z,M", CASES)
def test_compress_and_recover_match_oracle(T, n, d, Z, M, variant):
    print(f"compress T={T} n={n} d={d} Z={Z} M={M} variant={variant}", flush=True)
    rng = np.random.default_rng(T * 1000 + n)
    E = rng.standard_normal((T, n, d)).astype(np.float32)
    hp = pss.make_hash_params(17, num_tables=T, batch=n, num_indices=T * n)
    shared = pss.compress_table(torch.from_numpy(E).cuda(), M, Z, hp, variant=variant)
    torch.cuda.synchronize()
    got = shared.cpu().numpy()
    want, wabs = o.compress(E, M, Z, hp.a, hp.b)
    assert np.all(np.abs(got.astype(np.float64) - want) <= 1e-5 * wabs + 1e-30)
    R = pss.lookup_rows(shared, M, Z, d, T, n, hp).cpu().numpy()
    Rw = o.recover(got, M, Z, d, T, n, hp.a, hp.b)
    assert np.array_equal(R.astype(np.float64), Rw)  # one element per output: a plain copy
    # eps of Def. 2 per row, from the GPU retrieval vs the oracle's chain
    eps_gpu = o.pss_row_error(E, R)
    eps_ref = o.pss_row_error(E, o.recover(want.astype(np.float32), M, Z, d, T, n, hp.a, hp.b))
    np.testing.assert_allclose(eps_gpu, eps_ref, rtol=1e-4, atol=1e-5)


def test_compress_sparse_is_reproducible():
    T, n, d, Z, M = 2, 3000, 64, 16, 5000
    E = torch.from_numpy(np.random.default_rng(9).standard_normal((T, n, d)).astype(np.float32)).cuda()
    hp = pss.make_hash_params(3, num_tables=T, batch=n, num_indices=T * n)
    x = pss.compress_table(E, M, Z, hp)
    y = pss.compress_table(E, M, Z, hp, out=torch.full((M,), 7.0, device="cuda"))
    assert torch.equal(x.view(torch.int32), y.view(torch.int32))


def test_compress_injective_is_exact():
    """Z = d, a = d, b = 0 and M = n T d place row (t, i) at d (i T + t):
    compression is a permutation and retrieval returns the table exactly."""
    T, n, d = 3, 64, 16
    E = np.random.default_rng(0).standard_normal((T, n, d)).astype(np.float32)
    hp = pss.make_hash_params(a=d, b=0, num_tables=T, batch=n, num_indices=T * n)
    M = n * T * d
    shared = pss.compress_table(torch.from_numpy(E).cuda(), M, d, hp)
    flat = shared.cpu().numpy().reshape(n, T, d)
    assert np.array_equal(flat.transpose(1, 0, 2), E)
    R = pss.lookup_rows(shared, M, d, d, T, n, hp).cpu().numpy()
    assert np.array_equal(R, E)


def test_compress_bf16_lookup():
    """Retrieval from a bf16 copy of the compressed array reads the rounded values."""
    T, n, d, Z, M = 2, 400, 32, 8, 3001
    E = np.random.default_rng(4).standard_normal((T, n, d)).astype(np.float32)
    hp = pss.make_hash_params(8, num_tables=T, batch=n, num_indices=T * n)
    shared = pss.compress_table(torch.from_numpy(E).cuda(), M, Z, hp)
    sb = shared.to(torch.bfloat16)
    R = pss.lookup_rows(sb, M, Z, d, T, n, hp).cpu().numpy()
    bits = sb.cpu().view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(R.astype(np.float64), o.recover(bits, M, Z, d, T, n, hp.a, hp.b, o.BF16))
