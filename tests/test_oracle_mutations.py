"""The oracle's pins must catch plausible mistakes. Each case below plants one
mistake in a copy of the oracle's step (on the CPU, never in the product) and
checks that at least one pin rejects it."""

import numpy as np
import pytest

import oracle
from direct_kernel import kmat
from oracle import eigenpro as ep


def _mutant(kind):
    def step(state, alpha, t, y_b, block=16384):
        t = np.asarray(t, dtype=np.int64)
        alpha = np.asarray(alpha, dtype=np.float64)
        Xb = np.asarray(state.X[t], dtype=np.float64)
        F = ep._kernel_times(Xb, state.X, alpha, state.kernel, state.bandwidth, block, q_ids=t)
        R = F - y_b
        m = t.shape[0]
        c = ep.step_coefficient(state.beta, state.lam, m)
        if kind == "no_batch_term":
            c = 1.0 / state.beta
        Ksb = ep.kernel_matrix(state.Xs, Xb, state.kernel, state.bandwidth, state.r, t)
        if kind == "wrong_row_of_R":
            R_g = R[::-1]
        else:
            R_g = R
        G = Ksb @ R_g
        D = state.D
        if kind == "D_without_floor":
            D = 1.0 / state.sigma[:state.k]
        if kind == "D_not_inverted":
            D = 1.0 - state.sigma[state.k] / state.sigma[:state.k]
        H = state.V @ (D[:, None] * (state.V.T @ G))
        out = alpha.copy()
        out[t] -= c * R
        if kind == "correction_sign":
            out[state.r] -= c * H
        elif kind == "correction_on_batch_rows":
            out[t[: state.s]] += c * H[: len(t)]
        else:
            out[state.r] += c * H
        return out, F
    return step


def _full_batch_pin(step_fn, k=6):
    n = 40
    rng = np.random.default_rng(2)
    X = rng.standard_normal((n, 5)) / np.sqrt(5)
    Y = np.eye(2)[rng.integers(0, 2, n)]
    a0 = rng.standard_normal((n, 2)) / np.sqrt(n)
    r = rng.permutation(n)
    st = oracle.setup(X, oracle.GAUSSIAN, 0.8, n, k, r)
    t = rng.permutation(n)
    a1, _ = step_fn(st, a0, t, Y[t])
    K = kmat(X, X, oracle.GAUSSIAN, 0.8)
    sig, U = np.linalg.eigh(K)
    a_star = np.linalg.solve(K, Y)
    c = 1.0 / (st.beta + (n - 1) * st.sigma[k] / n)
    mult = 1.0 - c * np.minimum(sig, st.sigma[k])
    e0 = U.T @ (a0 - a_star)
    e1 = U.T @ (a1 - a_star)
    np.testing.assert_allclose(e1, mult[:, None] * e0, rtol=1e-9, atol=1e-9 * np.abs(e0).max())


def test_pin_accepts_the_oracle():
    _full_batch_pin(oracle.step)


@pytest.mark.parametrize("kind", ["no_batch_term", "wrong_row_of_R", "D_without_floor",
                                  "D_not_inverted", "correction_sign",
                                  "correction_on_batch_rows"])
def test_pin_rejects_planted_mistake(kind):
    with pytest.raises(AssertionError):
        _full_batch_pin(_mutant(kind))
