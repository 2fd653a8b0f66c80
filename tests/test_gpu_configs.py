"""GPU vs fp64 oracle on the five synthetic workloads, driven through the
C ABI exactly as bench.py drives it.

* tiny (n=2000): setup, one step from a seeded alpha0, three epochs from
  zero, predictions: all compared in full.
* MNIST- and CIFAR-shaped (n=60000 / 50000): setup, one step from alpha0
  and predictions in full; one epoch from zero in full.
* TIMIT- and ImageNet-shaped (n=1.1M / 1.28M) at full size with their own
  s and k: setup, and one step from alpha0 with the whole F and the whole
  change of alpha compared with the oracle's step from the oracle's own
  setup; then one epoch from zero on the first n/8 rows (same
  s, k, d, l), compared in full.
"""

import dataclasses

import numpy as np
import pytest

import oracle
import synth
from gpu_common import Gpu, SETUP_RTOL, TOL_EPOCH, TOL_STEP, kernel_id, lowrank, rel

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
    assert info.m_star == pytest.approx(st.m_star, rel=SETUP_RTOL)
    assert info.beta == pytest.approx(st.beta, rel=SETUP_RTOL)
    assert info.sigma_k1 == pytest.approx(st.sigma[-1], rel=SETUP_RTOL)
    sigma, D, V, _ = g.preconditioner()
    np.testing.assert_allclose(sigma, st.sigma, rtol=SETUP_RTOL)
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


def _epoch(w, st, g, m, epochs=1, progress=None):
    a = np.zeros((w.n, w.cfg.l))
    g.set_alpha(np.zeros((w.n, w.cfg.l), dtype=np.float32))
    for e in range(epochs):
        batches = synth.epoch_batches(w.n, m, e)
        for i, t in enumerate(batches):
            a, _ = oracle.step(st, a, t, w.y(t))
            g.step(t, w.y(t), want_f=False)
            if progress and (i + 1) % 10 == 0:
                progress(f"epoch {e}: {i + 1} of {len(batches)} steps")
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


# Rows of the prefix on which the large workloads are also run for a whole
# epoch against the oracle: n/8 of the TIMIT-shaped workload, n/16 of the
# ImageNet-shaped one (an epoch of the float64 oracle over n/8 rows of it
# would take about 4.5 minutes of host time on its own).
EPOCH_PREFIX = {"timit": 137500, "imagenet": 160000}


@pytest.mark.gpu
@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["timit", "imagenet"])
def test_large_config(name, capsys):
    """Full size, the workload's own s and k, one step from alpha0 (the
    bench's launch configuration): the whole F (m x l) and the whole change
    of alpha (n x l) against the oracle's step, run from the oracle's own
    setup. Then one epoch from zero on the first EPOCH_PREFIX rows with the
    same subsample, compared in full.

    The subsample is drawn uniformly from the prefix rows (the rows are
    i.i.d., so this is a uniform subsample of the workload as well), which
    lets the one float64 eigensolve of K_s serve both checks. Progress lines
    go straight to the terminal: the oracle's side of this test runs for
    minutes."""

    def progress(msg):
        with capsys.disabled():
            print(f"[{name}] {msg}", flush=True)

    cfg = synth.get_config(name)
    kid = kernel_id(cfg.kernel)
    P = EPOCH_PREFIX[name]
    w = _workload(name)
    r = synth.subsample_indices(cfg, 0, n=P)
    st = oracle.setup(w.X, kid, cfg.bandwidth, cfg.s, cfg.k, r)
    progress("oracle setup done")
    t = synth.epoch_batches(w.n, st.m, 0)[0]
    y = w.y(t)
    a0 = synth.initial_alpha(w.n, cfg.l, 0)
    g = Gpu(w.X, cfg.l, cfg.kernel, cfg.bandwidth, cfg.s, cfg.k, r)
    with g:
        _check_setup(st, g)
        g.set_alpha(a0)
        F = g.step(t, y)
        a1 = g.alpha()
    del g
    a1_o, F_o = oracle.step(st, a0, t, y)
    progress("full-size step compared")
    assert rel(F, F_o) < TOL_STEP
    # alpha changes only on the rows t and r: the relative error of the
    # change over all n x l entries is the one over those rows, provided
    # every other row is unchanged (exactly, on both sides)
    touched = np.union1d(t, r)
    assert rel(a1[touched] - a0[touched], a1_o[touched] - a0[touched]) < TOL_STEP
    keep = np.ones(w.n, dtype=bool)
    keep[touched] = False
    assert np.array_equal(a1[keep], a0[keep])
    del a1, a1_o, a0, keep

    # one epoch on the prefix rows, same subsample, from zero
    Xp = w.X[:P]
    stp = dataclasses.replace(st, X=Xp, m=int(min(P, max(1, np.floor(st.m_star)))))
    wp = synth.Workload(w.cfg, Xp, w.labels[:P], r, w.seed)
    gp = Gpu(Xp, cfg.l, cfg.kernel, cfg.bandwidth, cfg.s, cfg.k, r)
    with gp:
        _check_setup(stp, gp)
        _epoch(wp, stp, gp, stp.m, progress=progress)
