"""Pins of the oracle's kernel evaluation (Appendix B) against values fixed
by the mathematics: hand-computed entries, a brute-force double loop over
coordinates, and the structural properties of a positive definite kernel."""

import math

import numpy as np
import pytest

import oracle
from direct_kernel import kmat


def _brute(A, B, kernel, bw):
    out = np.empty((A.shape[0], B.shape[0]))
    for i in range(A.shape[0]):
        for j in range(B.shape[0]):
            d2 = 0.0
            for a, b in zip(A[i], B[j]):
                d2 += (float(a) - float(b)) ** 2
            if kernel == oracle.GAUSSIAN:
                out[i, j] = math.exp(-d2 / (2.0 * bw * bw))
            else:
                out[i, j] = math.exp(-math.sqrt(d2) / bw)
    return out


def test_hand_values():
    # |(0,0) - (3,4)| = 5
    A = np.array([[0.0, 0.0]])
    B = np.array([[3.0, 4.0], [0.0, 0.0]])
    g = oracle.kernel_matrix(A, B, oracle.GAUSSIAN, 5.0)
    lap = oracle.kernel_matrix(A, B, oracle.LAPLACIAN, 5.0)
    assert g[0, 0] == pytest.approx(math.exp(-0.5), rel=1e-15)
    assert lap[0, 0] == pytest.approx(math.exp(-1.0), rel=1e-14)
    assert g[0, 1] == 1.0 and lap[0, 1] == 1.0


@pytest.mark.parametrize("kernel", [oracle.GAUSSIAN, oracle.LAPLACIAN])
def test_matches_brute_force(kernel):
    rng = np.random.default_rng(1)
    A = rng.standard_normal((7, 5)).astype(np.float32)
    B = rng.standard_normal((9, 5)).astype(np.float32) * 1.5
    K = oracle.kernel_matrix(A, B, kernel, 1.3)
    np.testing.assert_allclose(K, _brute(A, B, kernel, 1.3), rtol=1e-12, atol=0)


@pytest.mark.parametrize("kernel", [oracle.GAUSSIAN, oracle.LAPLACIAN])
def test_symmetric_unit_diagonal_psd(kernel):
    rng = np.random.default_rng(2)
    X = rng.random((120, 16))
    ids = np.arange(120)
    K = oracle.kernel_matrix(X, X, kernel, 0.8, ids, ids)
    np.testing.assert_allclose(K, K.T, rtol=0, atol=1e-15)
    # the same training row on both sides: distance exactly 0, k(x, x) = 1
    assert np.all(np.diag(K) == 1.0)
    w = np.linalg.eigvalsh(K)
    assert w.min() > -1e-12 * K.shape[0]


@pytest.mark.parametrize("kernel", [oracle.GAUSSIAN, oracle.LAPLACIAN])
def test_matches_direct_differences_with_row_ids(kernel):
    """Against scipy's cdist (direct differences): a batch of training rows
    against a block of centres that shares some of them, as in step 2 and
    steps 4-5. Without ids the Laplacian diagonal carries the square root of
    the expansion's rounding (~1e-8); with them it is exact."""
    rng = np.random.default_rng(12)
    X = rng.random((300, 40)) * 3.0
    t = rng.choice(300, 50, replace=False)
    blk = np.arange(100, 260)
    K = oracle.kernel_matrix(X[t], X[blk], kernel, 2.0, t, blk)
    ref = kmat(X[t], X[blk], kernel, 2.0)
    np.testing.assert_allclose(K, ref, rtol=1e-12, atol=0)
    hit = np.isin(t, blk)
    assert hit.sum() > 5
    assert np.all(K[np.nonzero(hit)[0], t[hit] - 100] == 1.0)


def test_sq_dist_clamped_and_translation_invariant():
    rng = np.random.default_rng(3)
    X = rng.random((30, 8)) * 10
    d2 = oracle.sq_dist(X, X)
    assert (d2 >= 0).all()
    d2s = oracle.sq_dist(X + 3.25, X + 3.25)
    np.testing.assert_allclose(d2, d2s, rtol=1e-9, atol=1e-9)
