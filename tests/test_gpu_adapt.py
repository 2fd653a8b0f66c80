"""GPU vs oracle for the resource-adaptive parameters (Section 3 Steps 1-3):
lowering the rank from a held eigensystem, the Eq. 7 rank choice for a
resource batch m_G, and the batch-capacity measurement."""

import numpy as np
import pytest

import oracle
from gpu_common import Gpu, SETUP_RTOL, TOL_STEP, rel


def _problem(n=3000, d=24, l=5, seed=11):
    rng = np.random.default_rng(seed)
    X = (rng.standard_normal((n, d)) / np.sqrt(d)).astype(np.float32)
    Y = np.eye(l, dtype=np.float32)[rng.integers(0, l, n)]
    a0 = (rng.standard_normal((n, l)) / np.sqrt(n)).astype(np.float32)
    return X, Y, a0, rng


@pytest.mark.gpu
def test_set_rank_matches_fresh_oracle_setup():
    import paper_1806_06144_amd as ep
    X, Y, a0, rng = _problem()
    n, l, s, kmax = X.shape[0], Y.shape[1], 400, 40
    r = rng.choice(n, s, replace=False)
    big = oracle.setup(X, oracle.GAUSSIAN, 1.0, s, kmax, r)
    with Gpu(X, l, "gaussian", 1.0, s, kmax, r) as g:
        assert g.info.k_max == kmax
        for k in (0, 3, 17, 40):
            ep.ep_set_rank(g.ctx, k)
            info = ep.ep_get_info(g.ctx)
            st = oracle.with_rank(big, k)
            assert info.k == k and info.m == st.m
            assert info.beta == pytest.approx(st.beta, rel=SETUP_RTOL)
            assert info.m_star == pytest.approx(st.m_star, rel=SETUP_RTOL)
            t = rng.choice(n, 150, replace=False)
            a1_o, F_o = oracle.step(st, a0, t, Y[t])
            g.set_alpha(a0)
            F = g.step(t, Y[t])
            assert rel(F, F_o) < TOL_STEP
            assert rel(g.alpha() - a0, a1_o - a0) < TOL_STEP
        with pytest.raises(ep.EigenProError):
            ep.ep_set_rank(g.ctx, kmax + 1)


@pytest.mark.gpu
def test_adapt_picks_the_eq7_rank():
    import paper_1806_06144_amd as ep
    X, Y, a0, rng = _problem(seed=12)
    n, l, s, kmax = X.shape[0], Y.shape[1], 500, 60
    r = rng.choice(n, s, replace=False)
    big = oracle.setup(X, oracle.GAUSSIAN, 1.0, s, kmax, r)
    mstars = np.array([oracle.with_rank(big, k).m_star for k in range(kmax + 1)])
    # resource batches between consecutive critical batches (no ties)
    picks = [int(np.floor(0.5 * mstars[0])) or 1]
    for k in (2, 10, 30, 59):
        lo, hi = sorted((mstars[k], mstars[k + 1]))
        picks.append(int(np.floor(0.5 * (lo + hi))))
    picks.append(n + 50)
    with Gpu(X, l, "gaussian", 1.0, s, kmax, r) as g:
        for m_G in picks:
            info = ep.ep_adapt(g.ctx, m_G)
            k_o = oracle.choose_rank(big, m_G)
            assert info.k == k_o, (m_G, info.k, k_o)
            assert info.m == min(n, m_G)
            st = oracle.with_rank(big, k_o)
            assert info.accel == pytest.approx(oracle.acceleration(st, min(n, m_G)), rel=SETUP_RTOL)
            t = rng.choice(n, info.m, replace=False)
            a1_o, F_o = oracle.step(st, a0, t, Y[t])
            g.set_alpha(a0)
            F = g.step(t, Y[t])
            assert rel(g.alpha() - a0, a1_o - a0) < TOL_STEP


@pytest.mark.gpu
def test_batch_sweep_and_resource_batch():
    import paper_1806_06144_amd as ep
    X, Y, _, rng = _problem(n=40000, d=128, l=10, seed=13)
    with Gpu(X, 10, "gaussian", 2.0, 300, 20, rng.choice(40000, 300, replace=False)) as g:
        ms = [64, 256, 1024, 4096]
        t = ep.ep_batch_sweep(g.ctx, ms, reps=2)
        assert np.all(t > 0) and t[-1] > t[0]
        mc, msz, mg = ep.ep_resource_batch(g.ctx, 0.1)
        assert 16 <= mc <= 32768 and mg == min(mc, msz)
        # the knee of medians of repeated sweeps is reproducible
        assert ep.ep_resource_batch(g.ctx, 0.1) == (mc, msz, mg)
        # the paper's memory model on this device: (d + l + m) n floats
        assert msz > 10000
        with pytest.raises(ep.EigenProError):
            ep.ep_batch_sweep(g.ctx, [0], reps=1)
