"""GPU vs fp64 oracle on small seeded problems that exercise the edges of
the tiling: ragged query / centre / feature / label tails, label blocks
above 1024, label-tile counts that leave a wave's tiles partly empty, k = 0 (plain SGD), s = n, a single-point batch, a full batch,
batch rows that are also subsample rows, and both kernels."""

import numpy as np
import pytest

import oracle
from gpu_common import Gpu, SETUP_RTOL, TOL_STEP, TOL_EPOCH, bw32, kernel_id, lowrank, rel

CASES = [
    # kernel, n, d, l, s, k, m, bw
    ("gaussian", 300, 17, 3, 50, 5, 40, 1.0),
    ("laplacian", 1000, 64, 33, 200, 20, 130, 1.5),
    ("gaussian", 777, 36, 10, 777, 30, 777, 0.9),
    ("gaussian", 129, 8, 1, 20, 0, 1, 1.0),
    ("laplacian", 2000, 100, 160, 300, 40, 257, 2.0),
    ("gaussian", 600, 40, 1100, 64, 10, 70, 1.2),
    ("laplacian", 5000, 130, 7, 400, 60, 700, 3.0),
    # 3 and 7 label tiles (2 x 4 wave layout with two and four tiles per
    # wave, one of them partly empty)
    ("laplacian", 3000, 48, 70, 300, 30, 200, 2.0),
    ("gaussian", 2600, 96, 200, 256, 25, 300, 1.5),
    # 16-wide contraction (l <= 160): tiles of 16 labels exactly full (16,
    # 144 = 9 x 16) or one label past a tile (17), 7 and 10 tiles
    ("gaussian", 1500, 40, 16, 200, 20, 150, 1.2),
    ("laplacian", 1500, 40, 17, 200, 20, 150, 1.2),
    ("laplacian", 1800, 36, 100, 256, 30, 200, 1.5),
    ("gaussian", 2200, 44, 144, 300, 30, 260, 1.4),
    ("gaussian", 1300, 52, 150, 200, 25, 129, 1.1),
    # first label count past the 16-wide contraction (161: 32-wide again)
    ("laplacian", 1400, 36, 161, 200, 20, 150, 1.3),
    # batches of exactly one and two 512-row chunks for the product of
    # steps 4-5 (subsample of 192 = 3 x 64 rows for V^T G)
    ("laplacian", 1200, 32, 5, 192, 20, 512, 1.0),
    ("gaussian", 1500, 32, 5, 200, 20, 1024, 1.0),
]


def _problem(n, d, l, seed):
    rng = np.random.default_rng(seed)
    X = (rng.standard_normal((n, d)) / np.sqrt(d)).astype(np.float32)
    Y = np.eye(l, dtype=np.float32)[rng.integers(0, l, n)]
    a0 = (rng.standard_normal((n, l)) / np.sqrt(n)).astype(np.float32)
    return X, Y, a0, rng


def _batch(rng, n, r, m):
    """m distinct indices; about a quarter of them also subsample rows."""
    q = min(max(1, m // 4), len(r), m)
    head = r[:q]
    rest = rng.choice(np.setdiff1d(np.arange(n), head), m - q, replace=False)
    t = np.concatenate([head, rest]).astype(np.int64)
    rng.shuffle(t)
    return t


@pytest.mark.gpu
@pytest.mark.parametrize("case", CASES, ids=[f"{c[0][:3]}-n{c[1]}-d{c[2]}-l{c[3]}-s{c[4]}-k{c[5]}-m{c[6]}" for c in CASES])
def test_one_step_setup_predict(case):
    kernel, n, d, l, s, k, m, bw = case
    bw = bw32(bw)
    X, Y, a0, rng = _problem(n, d, l, 1)
    r = rng.choice(n, s, replace=False)
    t = _batch(rng, n, r, m)
    Z = (rng.standard_normal((77, d)) / np.sqrt(d)).astype(np.float32)
    st = oracle.setup(X, kernel_id(kernel), bw, s, k, r)
    a1_o, F_o = oracle.step(st, a0, t, Y[t])
    P_o = oracle.predict(X, a1_o, Z, kernel_id(kernel), bw)
    with Gpu(X, l, kernel, bw, s, k, r) as g:
        info = g.info
        assert info.m == st.m
        # setup is float64 on both sides (SETUP_RTOL)
        assert info.m_star == pytest.approx(st.m_star, rel=SETUP_RTOL)
        assert info.beta == pytest.approx(st.beta, rel=SETUP_RTOL)
        assert info.sigma_k1 == pytest.approx(st.sigma[k], rel=SETUP_RTOL)
        sigma, D, V, r_back = g.preconditioner()
        np.testing.assert_array_equal(r_back, r)
        np.testing.assert_allclose(sigma, st.sigma, rtol=SETUP_RTOL)
        if k:
            assert rel(lowrank(V, D), lowrank(st.V, st.D)) < 1e-5
        g.set_alpha(a0)
        F = g.step(t, Y[t])
        a1 = g.alpha()
        P = g.predict(Z)
    assert rel(F, F_o) < TOL_STEP
    assert rel(a1 - a0, a1_o - a0) < TOL_STEP
    assert rel(P, P_o) < TOL_STEP


EDGES = [
    # n, d, kernel: feature counts around the 16-feature chunk and the
    # 64-feature batch of the vector path (d % 4 == 0), one centre tile
    # exactly full (256) or one centre past it
    (700, 4, "gaussian"), (700, 12, "laplacian"), (700, 16, "gaussian"),
    (700, 20, "laplacian"), (700, 44, "gaussian"), (700, 60, "laplacian"),
    (700, 68, "gaussian"), (700, 128, "laplacian"), (700, 132, "gaussian"),
    (700, 196, "laplacian"), (256, 64, "gaussian"), (257, 64, "laplacian"),
    # long rows: 257 chunks (4-chunk batches) and 512 chunks (8-chunk)
    (300, 4112, "gaussian"), (300, 8192, "laplacian"),
]


@pytest.mark.gpu
@pytest.mark.parametrize("n,d,kernel", EDGES, ids=[f"n{c[0]}-d{c[1]}-{c[2][:3]}" for c in EDGES])
def test_feature_and_tile_edges(n, d, kernel):
    l, s, k, m, bw = 5, 60, 4, 70, bw32(1.3)
    X, Y, a0, rng = _problem(n, d, l, 5)
    r = rng.choice(n, s, replace=False)
    t = _batch(rng, n, r, m)
    Z = (rng.standard_normal((40, d)) / np.sqrt(d)).astype(np.float32)
    st = oracle.setup(X, kernel_id(kernel), bw, s, k, r)
    a1_o, F_o = oracle.step(st, a0, t, Y[t])
    with Gpu(X, l, kernel, bw, s, k, r) as g:
        g.set_alpha(a0)
        F = g.step(t, Y[t])
        a1 = g.alpha()
        P = g.predict(Z)
    assert rel(F, F_o) < TOL_STEP
    assert rel(a1 - a0, a1_o - a0) < TOL_STEP
    # predictions checked on the GPU's own alpha (near-flat kernels cancel)
    assert rel(P, oracle.predict(X, a1, Z, kernel_id(kernel), bw)) < TOL_STEP


@pytest.mark.gpu
@pytest.mark.parametrize("kernel,k", [("gaussian", 12), ("laplacian", 0)])
def test_epochs_from_zero(kernel, k):
    n, d, l, s = 1500, 32, 4, 250
    X, Y, _, rng = _problem(n, d, l, 2)
    r = rng.choice(n, s, replace=False)
    st = oracle.setup(X, kernel_id(kernel), 1.0, s, k, r)
    m = min(st.m, 300)
    a = np.zeros((n, l))
    with Gpu(X, l, kernel, 1.0, s, k, r) as g:
        for e in range(2):
            p = rng.permutation(n)
            batches = [p[i:i + m] for i in range(0, n, m)]
            for t in batches:
                a, _ = oracle.step(st, a, t, Y[t])
                g.step(t, Y[t], want_f=False)
        a_gpu = g.alpha()
    assert rel(a_gpu, a) < TOL_EPOCH


@pytest.mark.gpu
def test_error_paths_and_alpha_roundtrip():
    import torch
    import paper_1806_06144_amd as ep
    n, d, l = 200, 12, 3
    X, Y, a0, rng = _problem(n, d, l, 3)
    with pytest.raises(ep.EigenProError) as ei:
        Gpu(X, l, "gaussian", 1.0, 20, 4, np.array([1] * 20))
    assert ei.value.code == ep.EP_EINVAL
    with Gpu(X, l, "gaussian", 1.0, 20, 4, None, seed=7) as g:
        _, _, _, r = g.preconditioner()
        assert len(np.unique(r)) == 20 and r.min() >= 0 and r.max() < n
        g.set_alpha(a0)
        np.testing.assert_array_equal(g.alpha(), a0)
        # an index outside [0, n) is neither read nor written; ep_sync reports it
        bad = np.array([3, n + 5, 7], dtype=np.int64)
        g.step(bad, Y[:3], want_f=False)
        with pytest.raises(ep.EigenProError) as ei:
            ep.ep_sync(g.ctx)
        assert ei.value.code == ep.EP_EINDEX
        ep.ep_sync(g.ctx)              # flag is cleared once reported
        # repeated indices are rejected when checks are on
        ep.ep_set_checks(g.ctx, True)
        with pytest.raises(ep.EigenProError) as ei:
            g.step(np.array([4, 9, 4]), Y[:3], want_f=False)
        assert ei.value.code == ep.EP_EINDEX
        with pytest.raises(ep.EigenProError) as ei:
            ep.ep_step(g.ctx, g.t(np.array([1], dtype=np.int64)), 0, g.t(Y[:1]))
        assert ei.value.code == ep.EP_EINVAL
        # empty prediction is a no-op
        ep.ep_predict(g.ctx, g.t(X[:1]), 0, torch.empty((1, l), device="cuda:0"))


@pytest.mark.gpu
@pytest.mark.parametrize("kernel", ["gaussian", "laplacian"])
def test_predict_over_several_row_chunks(kernel):
    # 70000 query rows: two full 32768-row prediction chunks and a ragged one
    n, d, l = 400, 16, 3
    X, _, a, rng = _problem(n, d, l, 9)
    a = a * np.sqrt(n)                    # O(1) weights: no cancellation to hide errors in
    Z = (rng.standard_normal((70000, d)) / np.sqrt(d)).astype(np.float32)
    r = rng.choice(n, 50, replace=False)
    with Gpu(X, l, kernel, 1.1, 50, 5, r) as g:
        g.set_alpha(a)
        P = g.predict(Z)
    P_o = oracle.predict(X, a.astype(np.float64), Z, kernel_id(kernel), bw32(1.1))
    assert rel(P, P_o) < TOL_STEP
    for z0 in (0, 32767, 32768, 65535, 65536, 69999):   # rows at the chunk seams
        assert np.allclose(P[z0], P_o[z0], rtol=1e-4, atol=1e-4 * np.abs(P_o).max())


@pytest.mark.gpu
def test_restore_from_saved_setup():
    import paper_1806_06144_amd as ep
    n, d, l, s, k = 900, 20, 6, 150, 15
    X, Y, a0, rng = _problem(n, d, l, 4)
    r = rng.choice(n, s, replace=False)
    t = _batch(rng, n, r, 100)
    with Gpu(X, l, "laplacian", 1.3, s, k, r) as g:
        sigma, D, V, r_back = g.preconditioner()
        g.set_alpha(a0)
        F1 = g.step(t, Y[t])
        a1 = g.alpha()
        ctx2, info2 = ep.ep_restore(g.Xd, n, d, l, "laplacian", 1.3, s, k, r_back, sigma, V)
        try:
            assert info2.beta == pytest.approx(g.info.beta, rel=1e-6)
            assert info2.m == g.info.m
            sigma2, D2, V2, r2 = ep.ep_get_preconditioner(ctx2, info2)
            np.testing.assert_array_equal(V2, V)
            np.testing.assert_array_equal(D2, D)
            ep.ep_set_alpha(ctx2, g.t(a0))
            F2 = g.torch.empty((len(t), l), dtype=g.torch.float32, device=g.dev)
            ep.ep_step(ctx2, g.t(t), len(t), g.t(Y[t]), F2)
            a2 = g.torch.empty((n, l), dtype=g.torch.float32, device=g.dev)
            ep.ep_get_alpha(ctx2, a2)
            ep.ep_sync(ctx2)
        finally:
            ep.ep_destroy(ctx2)
    np.testing.assert_array_equal(F2.cpu().numpy(), F1)
    assert rel(a2.cpu().numpy() - a0, a1 - a0) < 1e-6
    with pytest.raises(ep.EigenProError):
        ep.ep_restore(g.Xd, n, d, l, "laplacian", 1.3, s, k, r_back, sigma[::-1].copy(), V)
