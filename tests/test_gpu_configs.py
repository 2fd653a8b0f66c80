"""GPU vs fp64 oracle on the five synthetic workloads, driven through the
C ABI exactly as bench.py drives it.

* tiny (n=2000): setup, one step from a seeded alpha0, three epochs from
  zero, predictions: all compared in full.
* MNIST- and CIFAR-shaped (n=60000 / 50000): setup, one step from alpha0
  and predictions in full; one epoch from zero in full.
* TIMIT- and ImageNet-shaped (n=1.1M / 1.28M) at full size: one step from
  alpha0, checked on a sample of batch rows the oracle computes one by one,
  plus properties that hold at any size (eigenpairs of the oracle's K_s,
  the batch-block update equals -c R, the fixed-block update equals
  c V D V^T K(X_r, X_t) R). One epoch on a row prefix of the same law, with
  the same d and l, a smaller s (stated in the test), compared in full.
"""

import numpy as np
import pytest

import oracle
import synth
from gpu_common import Gpu, TOL_EPOCH, TOL_STEP, kernel_id, lowrank, rel

_CACHE = {}


def _workload(name, **over):
    key = (name, tuple(sorted(over.items())))
    if key not in _CACHE:
        _CACHE.clear()
        cfg = synth.get_config(name, **over)
        _CACHE[key] = synth.make_workload(cfg, 0)
    return _CACHE[key]


def _setup_pair(w):
    cfg = w.cfg
    st = oracle.setup(w.X, kernel_id(cfg.kernel), cfg.bandwidth, cfg.s, cfg.k, w.r)
    g = Gpu(w.X, cfg.l, cfg.kernel, cfg.bandwidth, cfg.s, cfg.k, w.r)
    return st, g


def _check_setup(st, g):
    info = g.info
    assert abs(info.m - st.m) <= 1
    assert info.m_star == pytest.approx(st.m_star, rel=1e-6)
    assert info.beta == pytest.approx(st.beta, rel=1e-6)
    assert info.sigma_k1 == pytest.approx(st.sigma[-1], rel=1e-6)
    sigma, D, V, _ = g.preconditioner()
    np.testing.assert_allclose(sigma, st.sigma, rtol=1e-6)
    if st.k:
        assert rel(lowrank(V, D), lowrank(st.V, st.D)) < 1e-5


def _one_step_full(w, st, g, m):
    t = synth.epoch_batches(w.n, m, 0)[0]
    a0 = synth.initial_alpha(w.n, w.cfg.l, 0)
    a1_o, F_o = oracle.step(st, a0, t, w.y(t))
    g.set_alpha(a0)
    F = g.step(t, w.y(t))
    a1 = g.alpha()
    assert rel(F, F_o) < TOL_STEP
    assert rel(a1 - a0, a1_o - a0) < TOL_STEP
    return a1_o


def _epoch(w, st, g, m, epochs=1):
    a = np.zeros((w.n, w.cfg.l))
    g.set_alpha(np.zeros((w.n, w.cfg.l), dtype=np.float32))
    for e in range(epochs):
        for t in synth.epoch_batches(w.n, m, e):
            a, _ = oracle.step(st, a, t, w.y(t))
            g.step(t, w.y(t), want_f=False)
    a_gpu = g.alpha()
    assert rel(a_gpu, a) < TOL_EPOCH
    return a


@pytest.mark.gpu
def test_tiny_config():
    w = _workload("tiny")
    cfg = w.cfg
    st, g = _setup_pair(w)
    with g:
        _check_setup(st, g)
        _one_step_full(w, st, g, cfg.m)
        a = _epoch(w, st, g, cfg.m, epochs=cfg.epochs)
        Z = synth.heldout(cfg, 0)
        P_o = oracle.predict(w.X, a, Z, kernel_id(cfg.kernel), cfg.bandwidth)
        assert rel(g.predict(Z), P_o) < TOL_EPOCH
    # training residual |K alpha - y| falls over the epochs (it is |y| at 0)
    Y = w.y(np.arange(w.n))
    K = oracle.kernel_matrix(w.X, w.X, kernel_id(cfg.kernel), cfg.bandwidth)
    assert np.linalg.norm(K @ a - Y) < 0.6 * np.linalg.norm(Y)


@pytest.mark.gpu
@pytest.mark.timeout(600)
@pytest.mark.parametrize("name", ["mnist", "cifar"])
def test_medium_config(name):
    w = _workload(name)
    cfg = w.cfg
    st, g = _setup_pair(w)
    with g:
        _check_setup(st, g)
        m = st.m
        a1 = _one_step_full(w, st, g, m)
        Z = synth.heldout(cfg, 0, n_z=2000)
        P_o = oracle.predict(w.X, a1, Z, kernel_id(cfg.kernel), cfg.bandwidth)
        assert rel(g.predict(Z), P_o) < TOL_STEP
        a = _epoch(w, st, g, m)
        P_o = oracle.predict(w.X, a, Z, kernel_id(cfg.kernel), cfg.bandwidth)
        assert rel(g.predict(Z), P_o) < TOL_EPOCH


@pytest.mark.gpu
@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["timit", "imagenet"])
def test_large_config_one_step(name):
    """Full size; outputs the oracle computes one by one, and exact
    properties of the rest."""
    w = _workload(name)
    cfg = w.cfg
    kid = kernel_id(cfg.kernel)
    g = Gpu(w.X, cfg.l, cfg.kernel, cfg.bandwidth, cfg.s, cfg.k, w.r)
    with g:
        info = g.info
        m = int(info.m)
        sigma, D, V, r = g.preconditioner()
        # eigenpairs of the oracle's K_s (float64)
        Ks = oracle.kernel_matrix(w.X[r], w.X[r], kid, cfg.bandwidth)
        V64 = V.astype(np.float64)
        res = Ks @ V64 - V64 * sigma[:cfg.k]
        assert np.linalg.norm(res) / np.linalg.norm(Ks) < 1e-5
        np.testing.assert_allclose(V64.T @ V64, np.eye(cfg.k), atol=1e-5)
        assert np.all(np.diff(sigma) <= 0) and sigma[-1] > 0
        beta = oracle.beta_closed_form(sigma, V64)
        assert info.beta == pytest.approx(beta, rel=1e-5)
        assert info.m_star == pytest.approx(info.beta * cfg.s / sigma[-1], rel=1e-12)
        del Ks

        t = synth.epoch_batches(w.n, m, 0)[0]
        a0 = synth.initial_alpha(w.n, cfg.l, 0)
        g.set_alpha(a0)
        y = w.y(t)
        F = g.step(t, y)
        a1 = g.alpha()
        # predictions on sampled batch rows, by the oracle one row at a time
        rng = np.random.default_rng(7)
        sample = rng.choice(m, 24, replace=False)
        for j in sample[:2]:
            f_o = oracle.predict(w.X, a0, w.X[t[j]:t[j] + 1], kid, cfg.bandwidth)
            assert rel(F[j:j + 1], f_o) < TOL_STEP
        F_o = oracle.predict(w.X, a0, w.X[t[sample]], kid, cfg.bandwidth)
        assert rel(F[sample], F_o) < TOL_STEP

        c = 1.0 / (info.beta + (m - 1) * info.lambda_k1)
        R = F.astype(np.float64) - y
        dA = a1.astype(np.float64) - a0
        in_r = np.isin(t, r)
        # batch-block update (Algorithm 1 step 3) on rows not in the subsample
        assert rel(dA[t[~in_r]], -c * R[~in_r]) < TOL_STEP
        # fixed-block update (step 5): c V D V^T K(X_r, X_t) R, with the
        # kernel block formed by the oracle
        G = oracle.kernel_matrix(w.X[r], w.X[t], kid, cfg.bandwidth) @ R
        H = V64 @ (D[:, None] * (V64.T @ G))
        expect = c * H
        pos = {int(v): i for i, v in enumerate(t)}
        for i, row in enumerate(r):
            if row in pos:
                expect[i] -= c * R[pos[row]]
        assert rel(dA[r], expect) < TOL_STEP
        untouched = np.setdiff1d(np.arange(w.n), np.concatenate([t, r]))
        assert np.array_equal(a1[untouched[:100000]], a0[untouched[:100000]])


@pytest.mark.gpu
@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,n,s", [("timit", 60000, 4000), ("imagenet", 24000, 4000)])
def test_large_config_epoch_prefix(name, n, s):
    """One epoch on the first n rows of the workload's law, same d, l, k,
    kernel and bandwidth, subsample s (smaller than the full workload's so
    the float64 oracle finishes)."""
    w = _workload(name, n=n, s=s)
    st, g = _setup_pair(w)
    with g:
        _check_setup(st, g)
        _epoch(w, st, g, st.m)
