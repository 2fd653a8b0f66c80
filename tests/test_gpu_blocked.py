"""The blocked form of F = K(X_t, X) alpha (a kernel-block kernel per
centre chunk, then a float32 GEMM) against the fp64 oracle, and against the
fused form, through the C ABI. Chunks are forced small (block_bytes) so that
the accumulation over several chunks, ragged last chunks and ragged tiles
are exercised on small problems."""

import numpy as np
import pytest

import oracle
import synth
from gpu_common import Gpu, TOL_EPOCH, TOL_STEP, bw32, kernel_id, rel

CASES = [
    # kernel, n, d, l, s, k, m, bw          (d % 4 == 0: the blocked form applies)
    ("gaussian", 300, 16, 3, 50, 5, 40, 1.0),
    ("laplacian", 1000, 64, 33, 200, 20, 130, 1.5),
    ("gaussian", 777, 36, 10, 777, 30, 777, 0.9),
    ("gaussian", 129, 8, 1, 20, 0, 1, 1.0),
    ("laplacian", 2000, 100, 160, 300, 40, 257, 2.0),
    ("gaussian", 600, 40, 1100, 64, 10, 70, 1.2),
    ("gaussian", 3000, 132, 300, 400, 60, 600, 3.0),
]


def _problem(n, d, l, seed):
    rng = np.random.default_rng(seed)
    X = (rng.standard_normal((n, d)) / np.sqrt(d)).astype(np.float32)
    Y = np.eye(l, dtype=np.float32)[rng.integers(0, l, n)]
    a0 = (rng.standard_normal((n, l)) / np.sqrt(n)).astype(np.float32)
    return X, Y, a0, rng


def _kblock_launches(g, fn):
    g.ep.ep_timing_enable(g.ctx, True)
    out = fn()
    tim = g.ep.ep_timing_read(g.ctx)
    g.ep.ep_timing_enable(g.ctx, False)
    return out, tim.kblock_launches


@pytest.mark.gpu
@pytest.mark.parametrize("block_bytes", [0, 1], ids=["one-chunk", "256-centre-chunks"])
@pytest.mark.parametrize("case", CASES, ids=[f"{c[0][:3]}-n{c[1]}-d{c[2]}-l{c[3]}-m{c[6]}" for c in CASES])
def test_blocked_step_and_predict(case, block_bytes):
    kernel, n, d, l, s, k, m, bw = case
    bw = bw32(bw)
    X, Y, a0, rng = _problem(n, d, l, 3)
    r = rng.choice(n, s, replace=False)
    t = rng.choice(n, m, replace=False).astype(np.int64)
    Z = (rng.standard_normal((90, d)) / np.sqrt(d)).astype(np.float32)
    st = oracle.setup(X, kernel_id(kernel), bw, s, k, r)
    a1_o, F_o = oracle.step(st, a0, t, Y[t])
    # block_bytes = 1 rounds up to the smallest chunk: 256 centres
    with Gpu(X, l, kernel, bw, s, k, r, contraction="blocked", block_bytes=block_bytes) as g:
        g.set_alpha(a0)
        F, launches = _kblock_launches(g, lambda: g.step(t, Y[t]))
        expect = 1 if block_bytes == 0 else -(-n // 256)
        assert launches == expect
        a1 = g.alpha()
        P = g.predict(Z)
    assert rel(F, F_o) < TOL_STEP
    assert rel(a1 - a0, a1_o - a0) < TOL_STEP
    # prediction pass checked on the GPU's own alpha: predictions of these
    # near-flat kernels cancel (|K||a| / |K a| ~ 40), which would otherwise
    # amplify the step's own 1e-5-level error in alpha
    P_o = oracle.predict(X, a1, Z, kernel_id(kernel), bw)
    assert rel(P, P_o) < TOL_STEP


@pytest.mark.gpu
def test_blocked_epochs_from_zero():
    n, d, l, s, k, bw = 1500, 32, 4, 250, 12, 1.0
    X, Y, _, rng = _problem(n, d, l, 4)
    r = rng.choice(n, s, replace=False)
    st = oracle.setup(X, oracle.GAUSSIAN, bw, s, k, r)
    m = st.m
    a = np.zeros((n, l))
    with Gpu(X, l, "gaussian", bw, s, k, r, contraction="blocked", block_bytes=1) as g:
        for e in range(2):
            for tb in synth.epoch_batches(n, m, e):
                a, _ = oracle.step(st, a, tb, Y[tb])
                g.step(tb, Y[tb], want_f=False)
        assert rel(g.alpha(), a) < TOL_EPOCH


@pytest.mark.gpu
def test_blocked_falls_back_when_rows_are_not_vector_aligned():
    """d % 4 != 0: the blocked form does not apply and the fused one runs."""
    n, d, l, s, k, m, bw = 500, 17, 5, 60, 6, 50, 1.0
    X, Y, a0, rng = _problem(n, d, l, 5)
    r = rng.choice(n, s, replace=False)
    t = rng.choice(n, m, replace=False).astype(np.int64)
    st = oracle.setup(X, oracle.GAUSSIAN, bw, s, k, r)
    _, F_o = oracle.step(st, a0, t, Y[t])
    with Gpu(X, l, "gaussian", bw, s, k, r, contraction="blocked") as g:
        g.set_alpha(a0)
        F, launches = _kblock_launches(g, lambda: g.step(t, Y[t]))
    assert launches == 0
    assert rel(F, F_o) < TOL_STEP


@pytest.mark.gpu
def test_contraction_mode_errors():
    import paper_1806_06144_amd as ep
    X, _, _, rng = _problem(200, 8, 2, 6)
    with Gpu(X, 2, "gaussian", 1.0, 20, 2, rng.choice(200, 20, replace=False)) as g:
        for mode, nbytes in [(3, 0), (-1, 0), (1, -5)]:
            with pytest.raises(ep.EigenProError) as e:
                ep.ep_set_contraction(g.ctx, mode, nbytes)
            assert e.value.code == ep.EP_EINVAL
