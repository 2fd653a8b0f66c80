"""fp64 CPU oracle for one EigenPro 2.0 iteration — TEST INFRASTRUCTURE.

Used only by ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s
``cpu_baseline`` leg; never by the product path. It shares no code with the
HIP library. Inputs may be float32 arrays (the synthetic data); every
computation converts them to float64 first.

Paper: Ma & Belkin, "Kernel machines that adapt to GPUs for effective large
batch training" (SysML 2019, arXiv 1806.06144).

What each function follows
--------------------------
kernel_matrix      Appendix B: Gaussian exp(-|x-z|^2 / (2 sigma^2)) and
                   Laplacian exp(-|x-z| / sigma).
top_eigenpairs     the top q eigenpairs of K_s by a library routine (LAPACK
                   dense, or ARPACK Lanczos for large s).
setup              Algorithm 1 (initialisation: subsample r, top eigensystem
                   of K_s); Section 4 (Nystrom extension: lambda_i ~ sigma_i/s,
                   D = Sigma^-1 (1 - sigma_q Sigma^-1)); Section 3, Step 2
                   (beta(K_P) as the largest k_P(x, x) over subsample points,
                   lambda_1(K_P) = lambda_q); Section 2 (critical batch
                   m* = beta / lambda_1).
step_coefficient   Section 3, Step 3 and Appendix C, read as the optimal
                   per-coordinate step c(m) = 1 / (beta + (m - 1) lambda_q)
                   (see "Readings" below).
step               Algorithm 1, steps 1-5, in matrix form.
step_pointwise     Algorithm 1, steps 2-5, one point and one coordinate at a
                   time (pure Python loops; tiny cases only).
predict            Section 2: f(z) = sum_i alpha_i k(x_i, z).
interpolant        Section 2: alpha* = K^{-1} y, the unique interpolating
                   solution every iteration converges to.
with_rank          Section 3 Step 2 / Section 4: the adapted kernel of a lower
                   rank k' from the same eigensystem.
choose_rank        Section 3 Step 2, Eq. 7: the largest rank whose critical
                   batch does not exceed the resource batch m_G.
acceleration       Section 3 claim: beta(K)/beta(K_G) * m_G / m*(k).

Readings of the paper (shared with the HIP path by construction)
----------------------------------------------------------------
* q = k + 1: the top k + 1 eigenpairs of K_s are computed; V holds the top k
  eigenvectors and sigma_{k+1} is the flattening level. The paper's D has
  D_qq = 0, so this is the paper's update with q = k + 1.
* Step size: Algorithm 1 writes eta * 2/m and Section 3 Step 3 sets
  eta = m / beta, which puts the per-coordinate step at 2/beta, the edge of
  stability. Table 5's (m, eta) pairs satisfy m / eta ~ 2, i.e. a
  per-coordinate step of about 1/(2 beta) at m = m*, which is the optimal
  step 1 / (beta + (m - 1) lambda) of the interpolation analysis the paper
  relies on (Appendix C's denominator). The oracle uses
  c(m) = 1 / (beta_G + (m - 1) lambda_{k+1}) for both coordinate blocks, with
  the m of the batch at hand (a short last batch uses its own size).
* beta(K_G) is taken over the s subsample points, where k_P(x, x) has the
  closed form 1 - sum_j (sigma_j - sigma_{k+1}) V_ij^2.
* Both coordinate-block updates use the residual of the pre-step model and
  add; rows in both the batch and the subsample receive both.
* Squared distances use |a|^2 + |b|^2 - 2 a.b in float64 (a matrix product
  as a library step), clamped at zero so that the square root of the
  Laplacian kernel is defined when rounding makes the expansion negative.
  Where both sides index the same training row (the batch against all
  centres, the subsample against itself or against the batch) the distance
  is the direct sum of squared coordinate differences, which is exactly 0:
  a point's distance to itself is 0 by definition, and the expansion would
  leave rounding noise there (for the Laplacian kernel k(x, x) ~ 1 - 1e-8,
  the square root of that noise).
* Sums over the n centres are accumulated block by block over rows of X.

Parity pins live in tests/test_oracle_*.py.
"""

from dataclasses import dataclass

import numpy as np
import scipy.linalg
import scipy.sparse.linalg

GAUSSIAN = 0
LAPLACIAN = 1

_BLOCK = 16384


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def sq_dist(A, B, ids_a=None, ids_b=None):
    """All pairwise |a - b|^2 (float64), rows of A against rows of B.

    ``ids_a`` / ``ids_b`` (optional, distinct on each side) name the training
    row behind each row of A and B; pairs with equal ids get the direct sum
    of squared differences instead of the expansion."""
    A = _f64(A)
    B = _f64(B)
    an = np.einsum("ij,ij->i", A, A)
    bn = np.einsum("ij,ij->i", B, B)
    d2 = an[:, None] + bn[None, :] - 2.0 * (A @ B.T)
    np.maximum(d2, 0.0, out=d2)
    if ids_a is not None and ids_b is not None:
        _, pa, pb = np.intersect1d(np.asarray(ids_a, dtype=np.int64),
                                   np.asarray(ids_b, dtype=np.int64),
                                   assume_unique=True, return_indices=True)
        if pa.size:
            diff = A[pa] - B[pb]
            d2[pa, pb] = np.einsum("ij,ij->i", diff, diff)
    return d2


def kernel_matrix(A, B, kernel, bandwidth, ids_a=None, ids_b=None):
    """[k(a_i, b_j)] in float64 (Appendix B kernels); see ``sq_dist`` for the
    optional row ids."""
    d2 = sq_dist(A, B, ids_a, ids_b)
    if kernel == GAUSSIAN:
        return np.exp(-d2 / (2.0 * float(bandwidth) ** 2))
    if kernel == LAPLACIAN:
        return np.exp(-np.sqrt(d2) / float(bandwidth))
    raise ValueError(f"unknown kernel {kernel!r}")


def _kernel_times(Q, X, W, kernel, bandwidth, block=_BLOCK, q_ids=None):
    """sum_i k(q, x_i) W_i for every row q of Q, over all rows x_i of X,
    accumulated block by block over the rows of X. ``q_ids``: the training
    row of each query, if the queries are training points."""
    Q = _f64(Q)
    out = np.zeros((Q.shape[0], W.shape[1]), dtype=np.float64)
    for a in range(0, X.shape[0], block):
        b = min(X.shape[0], a + block)
        ids = None if q_ids is None else np.arange(a, b)
        out += kernel_matrix(Q, X[a:b], kernel, bandwidth, q_ids, ids) @ _f64(W[a:b])
    return out


@dataclass
class OracleState:
    """Setup products of Algorithm 1's initialisation and Section 3."""
    X: np.ndarray            # n x d training features (any float dtype)
    kernel: int
    bandwidth: float
    r: np.ndarray            # s subsample indices
    Xs: np.ndarray           # s x d, float64
    sigma: np.ndarray        # top k+1 eigenvalues of K_s, descending
    V: np.ndarray            # s x k top eigenvectors
    D: np.ndarray            # k: (1 - sigma_{k+1}/sigma_i) / sigma_i
    beta: float              # beta(K_G)
    lam: float               # lambda_{k+1} = sigma_{k+1} / s
    m_star: float            # beta / lambda
    m: int                   # min(n, max(1, floor(m*)))

    @property
    def s(self):
        return self.r.shape[0]

    @property
    def k(self):
        return self.V.shape[1]

    @property
    def n(self):
        return self.X.shape[0]


def beta_closed_form(sigma, V):
    """max over subsample points of k_P(x_ri, x_ri) = 1 - sum_j (sigma_j -
    sigma_{k+1}) V_ij^2 (Section 3 Step 2 with the Nystrom eigenfunctions
    e_j(x_ri) = sqrt(sigma_j) V_ij of Section 4; k(x, x) = 1)."""
    k = V.shape[1]
    if k == 0:
        return 1.0
    w = sigma[:k] - sigma[k]
    return float(np.max(1.0 - (V * V) @ w))


# subsample sizes up to which top_eigenpairs uses the dense routine
DENSE_EIG_MAX_S = 4000


def top_eigenpairs(K, q, method="auto"):
    """The q largest eigenvalues of the symmetric matrix K (descending) and
    their unit eigenvectors, by a library routine:

    dense    LAPACK's symmetric eigensolver (scipy.linalg.eigh) restricted to
             the top q; its reduction to tridiagonal form costs O(s^3) and
             takes minutes at s = 12000-20000;
    lanczos  ARPACK's implicitly restarted Lanczos iteration
             (scipy.sparse.linalg.eigsh) on K, which needs only products
             K v; a fixed seeded start vector makes it deterministic;
    auto     dense up to DENSE_EIG_MAX_S rows, else lanczos.
    """
    s = K.shape[0]
    if method == "auto":
        method = "dense" if s <= DENSE_EIG_MAX_S or q >= s else "lanczos"
    if method == "dense":
        w, U = scipy.linalg.eigh(K, subset_by_index=[s - q, s - 1])
    elif method == "lanczos":
        v0 = np.random.default_rng(12345).standard_normal(s)
        w, U = scipy.sparse.linalg.eigsh(K, k=q, which="LA", tol=1e-14, v0=v0,
                                         ncv=min(s, max(2 * q + 1, q + 64)))
    else:
        raise ValueError(f"unknown eigen method {method!r}")
    order = np.argsort(w)[::-1]
    return w[order].copy(), U[:, order].copy()


def setup(X, kernel, bandwidth, s, k, sub_idx, eig="auto"):
    """Algorithm 1 initialisation + Section 4 + Section 3 Steps 2-3."""
    n = X.shape[0]
    r = np.asarray(sub_idx, dtype=np.int64)
    if r.shape != (s,) or not (0 <= k < s <= n):
        raise ValueError("need 0 <= k < s <= n and s subsample indices")
    Xs = _f64(X[r])
    Ks = kernel_matrix(Xs, Xs, kernel, bandwidth, r, r)
    # top k+1 eigenpairs of K_s
    sigma, U = top_eigenpairs(Ks, k + 1, eig)
    V = U[:, :k].copy()
    D = (1.0 - sigma[k] / sigma[:k]) / sigma[:k]
    beta = beta_closed_form(sigma, V)
    lam = sigma[k] / s
    m_star = beta / lam
    m = int(min(n, max(1, np.floor(m_star))))
    return OracleState(X, kernel, float(bandwidth), r, Xs, sigma, V, D,
                       float(beta), float(lam), float(m_star), m)


def step_coefficient(beta, lam, m_b):
    """Per-coordinate step c(m) = 1 / (beta + (m - 1) lambda)."""
    return 1.0 / (beta + (m_b - 1) * lam)


def step(state, alpha, t, y_b, block=_BLOCK):
    """One iteration of Algorithm 1 (steps 1-5) from weights ``alpha``.

    Returns (alpha_next, F) with F the batch predictions before the update.
    """
    t = np.asarray(t, dtype=np.int64)
    alpha = _f64(alpha)
    y_b = _f64(y_b)
    Xb = _f64(state.X[t])
    # step 2: f(x_tj) = sum_i alpha_i k(x_i, x_tj)
    F = _kernel_times(Xb, state.X, alpha, state.kernel, state.bandwidth, block, q_ids=t)
    R = F - y_b
    c = step_coefficient(state.beta, state.lam, t.shape[0])
    # steps 4-5: sum_i (f(x_ti) - y_ti) V D V^T phi(x_ti)
    G = kernel_matrix(state.Xs, Xb, state.kernel, state.bandwidth, state.r, t) @ R
    H = state.V @ (state.D[:, None] * (state.V.T @ G))
    out = alpha.copy()
    out[t] -= c * R                 # step 3
    out[state.r] += c * H           # step 5
    return out, F


def step_pointwise(state, alpha, t, y_b):
    """Algorithm 1 steps 2-5 one point / one coordinate at a time (tiny
    inputs only)."""
    X = _f64(state.X)
    alpha = _f64(alpha)
    y_b = _f64(y_b)
    n, l = alpha.shape
    m = len(t)

    def k(a, b):
        diff = a - b
        d2 = float(np.dot(diff, diff))
        if state.kernel == GAUSSIAN:
            return np.exp(-d2 / (2.0 * state.bandwidth ** 2))
        return np.exp(-np.sqrt(d2) / state.bandwidth)

    f = np.zeros((m, l))
    for j in range(m):
        for i in range(n):
            f[j] += alpha[i] * k(X[i], X[t[j]])
    c = step_coefficient(state.beta, state.lam, m)
    out = alpha.copy()
    for j in range(m):
        out[t[j]] -= c * (f[j] - y_b[j])
    # V D V^T as an explicit s x s matrix
    P = np.zeros((state.s, state.s))
    for q in range(state.k):
        P += state.D[q] * np.outer(state.V[:, q], state.V[:, q])
    for j in range(m):
        phi = np.array([k(X[state.r[a]], X[t[j]]) for a in range(state.s)])
        upd = P @ phi
        for a in range(state.s):
            out[state.r[a]] += c * (f[j] - y_b[j]) * upd[a]
    return out, f


def predict(X, alpha, Z, kernel, bandwidth, block=_BLOCK, z_ids=None):
    """f(z) = sum_i alpha_i k(x_i, z) for every row z of Z (``z_ids``: the
    training row of each z, when the points predicted are training points)."""
    return _kernel_times(Z, X, _f64(alpha), kernel, bandwidth, block, q_ids=z_ids)


def run_epoch(state, alpha, batches, y_of):
    """Apply ``step`` over a list of index batches; ``y_of(t)`` gives the
    labels of a batch."""
    for t in batches:
        alpha, _ = step(state, alpha, t, y_of(t))
    return alpha


def interpolant(X, Y, kernel, bandwidth):
    """alpha* = K^{-1} Y (Section 2), by a dense solve."""
    ids = np.arange(X.shape[0])
    K = kernel_matrix(X, X, kernel, bandwidth, ids, ids)
    return np.linalg.solve(K, _f64(Y))


def with_rank(state, k):
    """The same subsample and eigensystem flattened at rank k <= state.k:
    V keeps its top k columns, sigma_{k+1} becomes the floor, and beta, m*,
    m are recomputed (Section 3 Step 2, Section 4)."""
    if not 0 <= k <= state.k:
        raise ValueError("rank outside [0, k]")
    sigma = state.sigma[:k + 1].copy()
    V = state.V[:, :k].copy()
    D = (1.0 - sigma[k] / sigma[:k]) / sigma[:k]
    beta = beta_closed_form(sigma, V)
    lam = sigma[k] / state.s
    m_star = beta / lam
    m = int(min(state.n, max(1, np.floor(m_star))))
    return OracleState(state.X, state.kernel, state.bandwidth, state.r, state.Xs, sigma, V, D,
                       float(beta), float(lam), float(m_star), m)


def choose_rank(state, m_G):
    """Eq. 7 with q = k+1: the largest k <= state.k with m*(k) <= m_G (0 if
    none)."""
    best = 0
    for k in range(state.k + 1):
        if with_rank(state, k).m_star <= m_G:
            best = k
    return best


def acceleration(state_k, m_G):
    """beta(K) / beta(K_G) * m_G / m*(k): beta(K) = 1 for the normalised
    kernels and m*(k) = s / sigma_1 for the original kernel."""
    return (1.0 / state_k.beta) * m_G / (state_k.s / state_k.sigma[0])
