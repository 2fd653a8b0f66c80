"""Shared helpers of the GPU parity tests: drive the HIP library through its
binding and the fp64 oracle on the same seeded inputs."""

import numpy as np

import oracle

TOL_STEP = 1e-4      # relative Frobenius error after one step
TOL_EPOCH = 1e-3     # relative Frobenius error after one epoch
# Setup scalars (sigma, beta, m*): float64 on both sides. The device forms
# K_s from direct coordinate differences, the oracle from the expansion
# with exact same-point distances, so the two K_s agree to ~1e-15; the
# eigenpairs come from different float64 solvers (the device's subspace
# iteration stops at a residual of 1e-11 sigma_1), and beta is a max over
# the subsample of a sum formed from the float64 eigenvectors on both sides.
SETUP_RTOL = 1e-9


def bw32(bw):
    """The bandwidth as the library receives it: the C ABI takes it as a
    float32, and setup and step use exactly that value, so the oracle is
    handed the same number (0.9 in float32 is 0.9 - 2.4e-8, which moves K_s
    by ~5e-8)."""
    return float(np.float32(bw))


def rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    nb = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (nb if nb > 0 else 1.0))


def kernel_id(name):
    return {"gaussian": oracle.GAUSSIAN, "laplacian": oracle.LAPLACIAN}[name]


class Gpu:
    """One ep_ctx on cuda:0 over a host feature matrix."""

    def __init__(self, X, l, kernel, bw, s, k, r, seed=0, contraction=None, block_bytes=0):
        import torch
        import paper_1806_06144_amd as ep
        self.ep = ep
        self.torch = torch
        self.dev = torch.device("cuda:0")
        self.n, self.d = X.shape
        self.l = l
        self.Xd = torch.from_numpy(np.ascontiguousarray(X, dtype=np.float32)).to(self.dev)
        self.ctx, self.info = ep.ep_setup(self.Xd, self.n, self.d, l, kernel, bw, s, k,
                                          sub_idx=r, seed=seed)
        if contraction is not None:
            ep.ep_set_contraction(self.ctx, contraction, block_bytes)

    def t(self, a):
        return self.torch.from_numpy(np.ascontiguousarray(a)).to(self.dev)

    def set_alpha(self, a):
        self.ep.ep_set_alpha(self.ctx, self.t(a.astype(np.float32)))

    def alpha(self):
        out = self.torch.empty((self.n, self.l), dtype=self.torch.float32, device=self.dev)
        self.ep.ep_get_alpha(self.ctx, out)
        self.ep.ep_sync(self.ctx)
        return out.cpu().numpy()

    def step(self, idx, y, want_f=True):
        m = len(idx)
        f = self.torch.empty((m, self.l), dtype=self.torch.float32, device=self.dev) if want_f else None
        self.ep.ep_step(self.ctx, self.t(np.asarray(idx, dtype=np.int64)), m,
                        self.t(y.astype(np.float32)), f)
        if want_f:
            self.ep.ep_sync(self.ctx)
            return f.cpu().numpy()
        return None

    def predict(self, Z):
        out = self.torch.empty((Z.shape[0], self.l), dtype=self.torch.float32, device=self.dev)
        self.ep.ep_predict(self.ctx, self.t(Z.astype(np.float32)), Z.shape[0], out)
        self.ep.ep_sync(self.ctx)
        return out.cpu().numpy()

    def preconditioner(self):
        return self.ep.ep_get_preconditioner(self.ctx, self.info)

    def close(self):
        if self.ctx is not None:
            self.ep.ep_destroy(self.ctx)
            self.ctx = None

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()


def lowrank(V, D):
    return (V.astype(np.float64) * D) @ V.astype(np.float64).T
