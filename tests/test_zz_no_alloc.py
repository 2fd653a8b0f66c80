"""ep_predict_noalloc (the entry point for callers that cannot allocate)
against ep_predict, through the C ABI, on two calls in a row, the second
with a smaller input; and its size limit."""

import numpy as np
import pytest

from gpu_common import Gpu, bw32, rel

TOL = 1e-5   # same float32 terms, summed in another order (other splits)


def _problem(n, d, l, seed):
    rng = np.random.default_rng(seed)
    X = (rng.standard_normal((n, d)) / np.sqrt(d)).astype(np.float32)
    a = rng.standard_normal((n, l)).astype(np.float32)
    return X, a, rng


def _both(g, Z):
    import paper_1806_06144_amd as ep
    torch = g.torch
    out_a = torch.empty((Z.shape[0], g.l), dtype=torch.float32, device=g.dev)
    out_b = torch.full((Z.shape[0], g.l), float("nan"), dtype=torch.float32, device=g.dev)
    Zd = g.t(Z)
    ep.ep_predict(g.ctx, Zd, Z.shape[0], out_a)
    ep.ep_predict_noalloc(g.ctx, Zd, Z.shape[0], out_b)
    ep.ep_sync(g.ctx)
    return out_a.cpu().numpy(), out_b.cpu().numpy()


@pytest.mark.gpu
@pytest.mark.parametrize("kernel,n,d,l", [("gaussian", 5000, 64, 10),
                                          ("gaussian", 4100, 48, 144),
                                          ("laplacian", 3001, 37, 1100)])
def test_noalloc_predict_matches_predict(kernel, n, d, l):
    X, a, rng = _problem(n, d, l, 3)
    with Gpu(X, l, kernel, bw32(1.3), 200, 10, rng.choice(n, 200, replace=False)) as g:
        g.set_alpha(a)
        for n_z in (20000, 333):          # two calls in a row, the second smaller
            Z = (rng.standard_normal((n_z, d)) / np.sqrt(d)).astype(np.float32)
            p_a, p_b = _both(g, Z)
            assert np.all(np.isfinite(p_b))
            assert rel(p_b, p_a) < TOL


@pytest.mark.gpu
def test_noalloc_predict_rejects_too_many_labels():
    import paper_1806_06144_amd as ep
    n, d, l = 64, 4, 270000
    X, _, rng = _problem(n, d, 1, 4)
    with Gpu(X, l, "gaussian", 1.0, 8, 2, np.arange(8)) as g:
        Z = g.t(X[:5])
        out = g.torch.empty((5, l), dtype=g.torch.float32, device=g.dev)
        with pytest.raises(ep.EigenProError) as ei:
            ep.ep_predict_noalloc(g.ctx, Z, 5, out)
        assert ei.value.code == ep.EP_EINVAL
        assert "scratch" in str(ei.value)
