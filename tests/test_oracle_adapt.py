"""Pins of the oracle's resource-adaptive rank choice (Section 3 Step 2,
Eq. 7): a lower rank taken from a larger eigensystem equals a fresh setup at
that rank, and the chosen rank is the largest one whose critical batch fits
m_G, checked by brute force over fresh setups."""

import numpy as np
import pytest

import oracle


def _data(n=240, d=10, seed=0):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((n, d)) / np.sqrt(d)


@pytest.mark.parametrize("kernel", [oracle.GAUSSIAN, oracle.LAPLACIAN])
def test_with_rank_equals_fresh_setup(kernel):
    X = _data()
    r = np.arange(0, 240, 2)
    big = oracle.setup(X, kernel, 0.8, 120, 30, r)
    for k in (0, 1, 7, 29, 30):
        a = oracle.with_rank(big, k)
        b = oracle.setup(X, kernel, 0.8, 120, k, r)
        assert a.m_star == pytest.approx(b.m_star, rel=1e-10)
        assert a.beta == pytest.approx(b.beta, rel=1e-12)
        P_a = a.V @ np.diag(a.D) @ a.V.T
        P_b = b.V @ np.diag(b.D) @ b.V.T
        np.testing.assert_allclose(P_a, P_b, atol=1e-10)


def test_choose_rank_brute_force():
    X = _data(300, 12, 1)
    r = np.arange(300)[::2]
    big = oracle.setup(X, oracle.GAUSSIAN, 1.0, 150, 40, r)
    fresh = [oracle.setup(X, oracle.GAUSSIAN, 1.0, 150, k, r).m_star for k in range(41)]
    assert fresh[-1] > fresh[0]           # flattening raises the critical batch
    for m_G in [1, fresh[0] * 0.5, fresh[0], fresh[5] + 1e-9, fresh[20] * 1.001, 1e9]:
        k = oracle.choose_rank(big, m_G)
        ok = [kk for kk in range(41) if fresh[kk] <= m_G]
        assert k == (max(ok) if ok else 0)


def test_acceleration_of_the_original_kernel_is_one():
    X = _data(200, 8, 2)
    st = oracle.setup(X, oracle.GAUSSIAN, 1.0, 100, 10, np.arange(100))
    k0 = oracle.with_rank(st, 0)
    # with k = 0 and m_G = m*(k) the claim's factor is exactly 1
    assert oracle.acceleration(k0, k0.m_star) == pytest.approx(1.0)
    assert oracle.acceleration(oracle.with_rank(st, 10), 500) > oracle.acceleration(k0, 500) * 0.99
