"""Pins of the oracle's iteration (Algorithm 1 steps 1-5, Eq. 8) against
results fixed by the mathematics:

* k = 0 removes the correction, leaving the coordinate form of mini-batch
  SGD (Eq. 3), computed here from an explicit kernel matrix;
* one point with k = 0 at the optimal step interpolates that point exactly;
* with s = n, a full batch and the exact eigensystem, the error in the
  eigenbasis of K is multiplied by 1 - c min(sigma_j, sigma_{k+1})
  (Appendix C's flattened spectrum);
* a literal point-by-point loop of the algorithm agrees with the matrix form;
* the step is invariant to the order within a batch and to eigenvector signs;
* the iteration converges to the interpolant K^{-1} y (Section 2), faster
  with preconditioning;
* prediction equals a brute-force sum and is linear in alpha.
"""

import math

import numpy as np
import pytest

import oracle
from direct_kernel import kmat


def _problem(n=60, d=6, l=3, seed=0):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((n, d)) / np.sqrt(d)
    Y = np.eye(l)[rng.integers(0, l, n)]
    a0 = rng.standard_normal((n, l)) / np.sqrt(n)
    return X, Y, a0


@pytest.mark.parametrize("kernel", [oracle.GAUSSIAN, oracle.LAPLACIAN])
def test_k0_is_plain_sgd(kernel):
    X, Y, a0 = _problem()
    st = oracle.setup(X, kernel, 0.9, 30, 0, np.arange(0, 60, 2))
    t = np.array([3, 17, 40, 41, 59, 8])
    a1, F = oracle.step(st, a0, t, Y[t])
    K = kmat(X, X, kernel, 0.9)
    c = 1.0 / (1.0 + (len(t) - 1) * st.sigma[0] / 30)
    expect = a0.copy()
    expect[t] -= c * ((K @ a0)[t] - Y[t])
    np.testing.assert_allclose(F, (K @ a0)[t], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(a1, expect, rtol=1e-12, atol=1e-14)


def test_single_point_interpolates():
    X, Y, a0 = _problem(40, 5, 2, 1)
    st = oracle.setup(X, oracle.GAUSSIAN, 1.0, 20, 0, np.arange(20))
    for j in (0, 7, 39):
        a1, _ = oracle.step(st, a0, np.array([j]), Y[j:j + 1])
        f = oracle.predict(X, a1, X[j:j + 1], oracle.GAUSSIAN, 1.0)
        np.testing.assert_allclose(f, Y[j:j + 1], atol=1e-12)


@pytest.mark.parametrize("kernel", [oracle.GAUSSIAN, oracle.LAPLACIAN])
@pytest.mark.parametrize("k", [0, 5, 12])
def test_full_batch_flattened_spectrum(kernel, k):
    n = 50
    X, Y, a0 = _problem(n, 5, 2, 2)
    rng = np.random.default_rng(9)
    r = rng.permutation(n)                  # s = n, in a shuffled order
    st = oracle.setup(X, kernel, 0.8, n, k, r)
    t = rng.permutation(n)                  # full batch, another order
    a1, _ = oracle.step(st, a0, t, Y[t])
    K = kmat(X, X, kernel, 0.8)
    sig, U = np.linalg.eigh(K)
    a_star = np.linalg.solve(K, Y)
    c = oracle.step_coefficient(st.beta, st.lam, n)
    floor = st.sigma[k]
    mult = 1.0 - c * np.minimum(sig, floor)
    e0 = U.T @ (a0 - a_star)
    e1 = U.T @ (a1 - a_star)
    np.testing.assert_allclose(e1, mult[:, None] * e0, rtol=1e-9, atol=1e-9 * np.abs(e0).max())


@pytest.mark.parametrize("kernel", [oracle.GAUSSIAN, oracle.LAPLACIAN])
def test_pointwise_loop_matches_matrix_form(kernel):
    X, Y, a0 = _problem(24, 4, 2, 3)
    r = np.array([5, 1, 20, 13, 9, 2, 17, 11, 3, 22])
    st = oracle.setup(X, kernel, 0.7, 10, 4, r)
    t = np.array([2, 19, 5, 7, 23])        # overlaps r in rows 2 and 5
    a_mat, F_mat = oracle.step(st, a0, t, Y[t])
    a_pt, F_pt = oracle.step_pointwise(st, a0, t, Y[t])
    np.testing.assert_allclose(F_mat, F_pt, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(a_mat, a_pt, rtol=1e-11, atol=1e-13)


def test_batch_order_and_sign_invariance():
    X, Y, a0 = _problem(80, 6, 3, 4)
    st = oracle.setup(X, oracle.GAUSSIAN, 1.0, 40, 8, np.arange(40, 80))
    t = np.array([1, 50, 3, 44, 79, 20, 61])
    a1, _ = oracle.step(st, a0, t, Y[t])
    p = np.array([6, 2, 0, 5, 1, 4, 3])
    a2, _ = oracle.step(st, a0, t[p], Y[t[p]])
    np.testing.assert_allclose(a1, a2, rtol=1e-12, atol=1e-14)
    st.V = st.V * np.where(np.arange(8) % 3 == 0, -1.0, 1.0)
    a3, _ = oracle.step(st, a0, t, Y[t])
    np.testing.assert_allclose(a1, a3, rtol=1e-12, atol=1e-14)


def _train_error(X, Y, kernel, bw, s, k, epochs, m=None, seed=0):
    n = X.shape[0]
    rng = np.random.default_rng(seed)
    st = oracle.setup(X, kernel, bw, s, k, rng.choice(n, s, replace=False))
    m = st.m if m is None else m
    a = np.zeros_like(Y)
    a_star = oracle.interpolant(X, Y, kernel, bw)
    errs = []
    for e in range(epochs):
        p = rng.permutation(n)
        a = oracle.run_epoch(st, a, [p[i:i + m] for i in range(0, n, m)], lambda t: Y[t])
        errs.append(np.linalg.norm(a - a_star) / np.linalg.norm(a_star))
    return np.array(errs), st


def test_converges_to_interpolant():
    rng = np.random.default_rng(10)
    n, d = 400, 64
    X = rng.standard_normal((n, d)) / math.sqrt(d)
    Y = np.eye(4)[np.argmax(X @ rng.standard_normal((d, 4)), axis=1)]
    errs_ep, st = _train_error(X, Y, oracle.GAUSSIAN, 1.0, 100, 10, 300, m=64)
    errs_sgd, _ = _train_error(X, Y, oracle.GAUSSIAN, 1.0, 100, 0, 300, m=64)
    assert errs_ep[-1] < 1e-6
    assert errs_sgd[-1] > 10 * errs_ep[-1]     # preconditioning accelerates
    assert errs_sgd[-1] < errs_sgd[0]          # plain SGD also converges, slowly


def test_predict_brute_force_and_linear():
    X, Y, a0 = _problem(30, 4, 2, 5)
    rng = np.random.default_rng(11)
    Z = rng.standard_normal((7, 4))
    P = oracle.predict(X, a0, Z, oracle.LAPLACIAN, 1.1)
    brute = np.zeros((7, 2))
    for i in range(7):
        for j in range(30):
            brute[i] += a0[j] * math.exp(-math.sqrt(((Z[i] - X[j]) ** 2).sum()) / 1.1)
    np.testing.assert_allclose(P, brute, rtol=1e-12)
    P2 = oracle.predict(X, 2.0 * a0 - Y, Z, oracle.LAPLACIAN, 1.1)
    np.testing.assert_allclose(P2, 2.0 * P - oracle.predict(X, Y, Z, oracle.LAPLACIAN, 1.1), rtol=1e-12, atol=1e-13)


def test_blocking_does_not_change_the_sum():
    X, Y, a0 = _problem(70, 5, 3, 6)
    Z = X[:9] + 0.01
    np.testing.assert_allclose(
        oracle.predict(X, a0, Z, oracle.GAUSSIAN, 1.0, block=7),
        oracle.predict(X, a0, Z, oracle.GAUSSIAN, 1.0, block=1000), rtol=1e-13)
