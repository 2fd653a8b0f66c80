"""Pins of the oracle's setup (Algorithm 1 initialisation, Section 4 Nystrom
extension, Section 3 Steps 2-3) against a different eigen routine, the
eigen-equation residual, brute-force evaluation of k_P(x, x), the s = n
Nystrom identities and the closed forms of the step coefficient."""

import numpy as np
import pytest

import oracle
from direct_kernel import kmat


def _data(n=300, d=12, seed=0):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((n, d)) / np.sqrt(d)


@pytest.mark.parametrize("kernel", [oracle.GAUSSIAN, oracle.LAPLACIAN])
def test_eigensystem(kernel):
    X = _data()
    rng = np.random.default_rng(5)
    r = rng.choice(X.shape[0], 120, replace=False)
    st = oracle.setup(X, kernel, 1.0, 120, 15, r)
    Ks = kmat(X[r], X[r], kernel, 1.0)
    # eigen-equation residual and orthonormality
    res = Ks @ st.V - st.V * st.sigma[:15]
    assert np.linalg.norm(res) <= 1e-10 * np.linalg.norm(Ks)
    np.testing.assert_allclose(st.V.T @ st.V, np.eye(15), atol=1e-12)
    # eigenvalues against numpy's divide-and-conquer routine on the full matrix
    w = np.linalg.eigvalsh(Ks)[::-1]
    np.testing.assert_allclose(st.sigma, w[:16], rtol=1e-11)
    assert np.all(np.diff(st.sigma) <= 0)


def _kp_diag_brute(st):
    """k(x,x) - phi(x)^T V D V^T phi(x) at every subsample point, with phi
    evaluated from the kernel itself."""
    P = st.V @ np.diag(st.D) @ st.V.T
    out = []
    for i in range(st.s):
        x = st.Xs[i:i + 1]
        phi = kmat(st.Xs, x, st.kernel, st.bandwidth)[:, 0]
        kxx = kmat(x, x, st.kernel, st.bandwidth)[0, 0]
        out.append(kxx - phi @ P @ phi)
    return np.array(out)


@pytest.mark.parametrize("kernel", [oracle.GAUSSIAN, oracle.LAPLACIAN])
def test_beta_closed_form_equals_brute_force(kernel):
    X = _data(200, 10, 1)
    r = np.arange(0, 200, 2)
    st = oracle.setup(X, kernel, 0.7, 100, 12, r)
    brute = _kp_diag_brute(st)
    assert st.beta == pytest.approx(brute.max(), abs=1e-12)
    assert 0.0 < st.beta <= 1.0


def test_beta_is_one_without_preconditioning():
    X = _data(100, 6, 2)
    st = oracle.setup(X, oracle.GAUSSIAN, 1.0, 50, 0, np.arange(50))
    assert st.beta == 1.0 and st.V.shape == (50, 0)
    assert st.lam == pytest.approx(st.sigma[0] / 50)
    assert st.m_star == pytest.approx(50 / st.sigma[0])


def test_nystrom_identities_full_subsample():
    # s = n: lambda_i = sigma_i / n and e_i = sigma_i^{-1/2} v_i^T phi has
    # unit RKHS norm: (1/sigma_i) v_i^T K v_i = 1
    X = _data(80, 5, 3)
    st = oracle.setup(X, oracle.GAUSSIAN, 1.0, 80, 10, np.arange(80))
    K = kmat(X, X, oracle.GAUSSIAN, 1.0)
    for i in range(10):
        v = st.V[:, i]
        assert (v @ K @ v) / st.sigma[i] == pytest.approx(1.0, rel=1e-12)
    assert st.lam == pytest.approx(st.sigma[10] / 80)


def test_flattened_spectrum_gives_critical_batch():
    # lambda_1(K_P) = sigma_{k+1}/s and m* = beta / lambda_1(K_P)
    X = _data(150, 8, 4)
    st = oracle.setup(X, oracle.GAUSSIAN, 1.0, 150, 7, np.arange(150))
    assert st.m_star == pytest.approx(st.beta * 150 / st.sigma[7])
    assert st.m == int(np.floor(st.m_star))
    st0 = oracle.setup(X, oracle.GAUSSIAN, 1.0, 150, 0, np.arange(150))
    assert st.m_star > st0.m_star  # flattening raises the critical batch


def test_q_equals_k_plus_one_form():
    # the paper's D with q = k+1 columns has D_qq = 0, so V D V^T is the same
    X = _data(120, 6, 5)
    st = oracle.setup(X, oracle.GAUSSIAN, 1.0, 60, 9, np.arange(60))
    Ks = kmat(X[:60], X[:60], oracle.GAUSSIAN, 1.0)
    w, U = np.linalg.eigh(Ks)
    w, U = w[::-1][:10], U[:, ::-1][:, :10]
    Dq = (1.0 - w[9] / w) / w          # Sigma^-1 (1 - sigma_q Sigma^-1), q = 10
    assert Dq[9] == 0.0
    P_q = U @ np.diag(Dq) @ U.T
    P_k = st.V @ np.diag(st.D) @ st.V.T
    np.testing.assert_allclose(P_k, P_q, atol=1e-12)


def test_step_coefficient_closed_forms():
    X = _data(100, 6, 6)
    st = oracle.setup(X, oracle.GAUSSIAN, 1.0, 100, 0, np.arange(100))
    # k = 0, beta = 1: plain SGD optimum 1/(1 + (m-1) sigma_1/s)
    for m in (1, 7, 64):
        c = oracle.step_coefficient(st.beta, st.lam, m)
        assert c == pytest.approx(1.0 / (1.0 + (m - 1) * st.sigma[0] / 100))
    st2 = oracle.setup(X, oracle.GAUSSIAN, 1.0, 100, 5, np.arange(100))
    assert oracle.step_coefficient(st2.beta, st2.lam, 1) == pytest.approx(1.0 / st2.beta)


def test_eigenvector_sign_invariance():
    X = _data(90, 6, 7)
    st = oracle.setup(X, oracle.LAPLACIAN, 1.0, 45, 6, np.arange(45))
    flipped = st.V * np.where(np.arange(6) % 2 == 0, -1.0, 1.0)
    assert oracle.beta_closed_form(st.sigma, flipped) == pytest.approx(st.beta, abs=1e-15)


@pytest.mark.parametrize("kernel,bw", [(oracle.GAUSSIAN, 15.0), (oracle.LAPLACIAN, 10.0)])
def test_lanczos_route_equals_dense_eigh(kernel, bw):
    """The two library routes of top_eigenpairs give the same eigensystem on a
    K_s with the flat bulk of the workloads (rows from the TIMIT-shaped law:
    one large eigenvalue, then near-equal ones around sigma_{k+1})."""
    rng = np.random.default_rng(21)
    X = rng.standard_normal((1500, 440))
    Ks = kmat(X, X, kernel, bw)
    q = 121
    wd, Ud = oracle.top_eigenpairs(Ks, q, "dense")
    wl, Ul = oracle.top_eigenpairs(Ks, q, "lanczos")
    np.testing.assert_allclose(wl, wd, rtol=1e-12)
    assert np.all(np.diff(wl) <= 0)
    # the bulk really is flat: sigma_q and sigma_{q-1} within 1 %
    assert wd[q - 2] / wd[q - 1] < 1.01
    # same spectral projector onto the top q - 1 (eigenvector signs and
    # rotations inside near-degenerate pairs do not matter there)
    D = 1.0 / wd[:q - 1]
    Pd = (Ud[:, :q - 1] * D) @ Ud[:, :q - 1].T
    Pl = (Ul[:, :q - 1] * D) @ Ul[:, :q - 1].T
    assert np.linalg.norm(Pl - Pd) / np.linalg.norm(Pd) < 1e-9
    res = Ks @ Ul - Ul * wl
    assert np.linalg.norm(res) <= 1e-10 * np.linalg.norm(Ks)
    # and the setup built on either route agrees
    r = np.arange(1500)
    st_d = oracle.setup(X, kernel, bw, 1500, q - 1, r, eig="dense")
    st_l = oracle.setup(X, kernel, bw, 1500, q - 1, r, eig="lanczos")
    assert st_l.beta == pytest.approx(st_d.beta, rel=1e-11)
    assert st_l.m_star == pytest.approx(st_d.m_star, rel=1e-11)
