"""Statistical behaviour of post-hoc compression (Def. 2, Thm. 2) in the oracle.

For a table E with i.i.d. zero-mean entries of variance s^2 and a fixed
mapping, the retrieved row differs from E_i by the sum of the other entries
sharing each of its locations, so over the draw of E

    E[eps_i^2] summed over all rows = s^2 * sum_m load(m) (load(m) - 1),

load(m) being the number of table entries mapped to m (obtained by
compressing a table of ones).  The check is empirical: the sample mean over
many rows must sit near that expectation.
"""
import numpy as np
import pytest

from oracle import pss_oracle as o


@pytest.mark.parametrize("T,n,d,Z,r", [(1, 20000, 16, 4, 10), (2, 10000, 32, 8, 4),
                                       (1, 50000, 8, 1, 2), (3, 4000, 16, 16, 1)])
def test_mean_squared_row_error_matches_collision_count(T, n, d, Z, r):
    rng = np.random.default_rng(n + d)
    M = n * T * d // r
    s = 0.5
    E = rng.standard_normal((T, n, d)) * s
    a, b = o.hash_params_from_seed(5)
    Mv, _ = o.compress(E, M, Z, a, b)
    eps = o.pss_row_error(E, o.recover(Mv, M, Z, d, T, n, a, b, weight_dtype=o.F32))
    load, _ = o.compress(np.ones((T, n, d)), M, Z, a, b)
    expect = s * s * (load * (load - 1)).sum() / (T * n)
    assert abs((eps ** 2).mean() / expect - 1) < 0.05


def test_error_grows_with_compression():
    T, n, d, Z = 1, 20000, 16, 4
    E = np.random.default_rng(0).standard_normal((T, n, d))
    a, b = o.hash_params_from_seed(1)
    means = []
    for r in (1, 4, 16, 64):
        M = n * T * d // r
        Mv, _ = o.compress(E, M, Z, a, b)
        means.append(o.pss_row_error(E, o.recover(Mv, M, Z, d, T, n, a, b)).mean())
    assert all(x < y for x, y in zip(means, means[1:]))
