"""Seeded draws for the synthetic workloads.

Every stream is a child of ``numpy.random.SeedSequence(seed)`` addressed by an
explicit spawn key, so any row range can be regenerated on its own and the
result does not depend on thread count or call order:

    (0, c)  features X, row chunk c          (2, c)  held-out Z, row chunk c
    (1,)    label map / class means          (3,)    subsample indices r
    (4, e)  permutation of epoch e           (5, c)  initial weights alpha0, chunk c

Draws are made directly in float32 (the precision both consumers read). The
label rule uses a float32 matrix product followed by an argmin/argmax with the
lowest index winning ties; labels are data, computed once and handed to both
sides, so the precision of that rule is not a parity question.
"""

from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass
import os

import numpy as np

from .configs import Config

CHUNK_ROWS = 1 << 16


def _ss(seed: int, *key: int) -> np.random.SeedSequence:
    return np.random.SeedSequence(seed, spawn_key=tuple(key))


def _rng(seed: int, *key: int) -> np.random.Generator:
    return np.random.default_rng(_ss(seed, *key))


def _threads() -> int:
    n = os.cpu_count() or 1
    return max(1, min(16, n))


def _draw_rows(rng: np.random.Generator, law: str, rows: int, d: int) -> np.ndarray:
    """One block of rows from a feature law (float32)."""
    if law == "normal_scaled":          # N(0,1)/sqrt(d)
        x = rng.standard_normal((rows, d), dtype=np.float32)
        x *= np.float32(1.0 / np.sqrt(d))
    elif law == "normal":               # standardised features
        x = rng.standard_normal((rows, d), dtype=np.float32)
    elif law == "uniform":              # pixels rescaled to [0, 1]
        x = rng.random((rows, d), dtype=np.float32)
    elif law == "uniform_sparse80":     # [0,1] pixels, 80 % of entries zero
        x = rng.random((rows, d), dtype=np.float32)
        x[rng.random((rows, d), dtype=np.float32) < np.float32(0.8)] = 0.0
    elif law == "halfnormal_sparse50":  # ReLU-like: |N(0,1)|, 50 % zero
        x = np.abs(rng.standard_normal((rows, d), dtype=np.float32))
        x[rng.random((rows, d), dtype=np.float32) < np.float32(0.5)] = 0.0
    else:
        raise ValueError(f"unknown feature law {law!r}")
    return x


def _chunked(seed: int, stream: int, law: str, rows: int, d: int) -> np.ndarray:
    out = np.empty((rows, d), dtype=np.float32)
    chunks = [(c, c * CHUNK_ROWS, min(rows, (c + 1) * CHUNK_ROWS))
              for c in range((rows + CHUNK_ROWS - 1) // CHUNK_ROWS)]

    def fill(job):
        c, a, b = job
        out[a:b] = _draw_rows(_rng(seed, stream, c), law, CHUNK_ROWS, d)[: b - a]

    if len(chunks) == 1:
        fill(chunks[0])
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(fill, chunks))
    return out


def features(cfg: Config, seed: int = 0, n: int = None) -> np.ndarray:
    """Training features X (n x d float32, row-major). ``n`` takes a row
    prefix of the same draw."""
    return _chunked(seed, 0, cfg.x_law, cfg.n if n is None else n, cfg.d)


def heldout(cfg: Config, seed: int = 0, n_z: int = None) -> np.ndarray:
    """Held-out prediction points Z from the same law as X."""
    return _chunked(seed, 2, cfg.x_law, cfg.n_z if n_z is None else n_z, cfg.d)


def _label_map(cfg: Config, seed: int):
    rng = _rng(seed, 1)
    if cfg.label_rule == "argmax_linear":
        return rng.standard_normal((cfg.d, cfg.l), dtype=np.float32)
    if cfg.label_rule == "nearest_mean":
        # class means drawn from the same law as the features
        return _draw_rows(rng, cfg.x_law, cfg.l, cfg.d)
    raise ValueError(cfg.label_rule)


def class_labels(cfg: Config, X: np.ndarray, seed: int = 0) -> np.ndarray:
    """Integer class of every row of X (int32)."""
    M = _label_map(cfg, seed)
    out = np.empty(X.shape[0], dtype=np.int32)
    if cfg.label_rule == "argmax_linear":
        for a in range(0, X.shape[0], CHUNK_ROWS):
            out[a:a + CHUNK_ROWS] = np.argmax(X[a:a + CHUNK_ROWS] @ M, axis=1)
        return out
    mnorm = np.einsum("ij,ij->i", M, M)
    chunks = list(range(0, X.shape[0], CHUNK_ROWS))

    def lab(a):
        xb = X[a:a + CHUNK_ROWS]
        # |x - c|^2 = |x|^2 + |c|^2 - 2 x.c ; |x|^2 is constant per row
        out[a:a + CHUNK_ROWS] = np.argmin(mnorm[None, :] - 2.0 * (xb @ M.T), axis=1)

    with ThreadPoolExecutor(max(1, _threads() // 4)) as ex:
        list(ex.map(lab, chunks))
    return out


def one_hot(labels: np.ndarray, l: int) -> np.ndarray:
    y = np.zeros((labels.shape[0], l), dtype=np.float32)
    y[np.arange(labels.shape[0]), labels] = 1.0
    return y


def subsample_indices(cfg: Config, seed: int = 0, n: int = None, s: int = None) -> np.ndarray:
    """r: s distinct indices drawn uniformly without replacement (int64)."""
    n = cfg.n if n is None else n
    s = cfg.s if s is None else s
    return _rng(seed, 3).choice(n, size=s, replace=False).astype(np.int64)


def epoch_permutation(n: int, epoch: int, seed: int = 0) -> np.ndarray:
    return _rng(seed, 4, epoch).permutation(n).astype(np.int64)


def epoch_batches(n: int, m: int, epoch: int, seed: int = 0):
    """Consecutive batches of m indices from the epoch's permutation; the
    last batch holds the remainder."""
    p = epoch_permutation(n, epoch, seed)
    return [p[a:a + m] for a in range(0, n, m)]


def initial_alpha(n: int, l: int, seed: int = 0) -> np.ndarray:
    """alpha0 ~ N(0, 1/n), float32, used to start one-step checks from a
    non-zero model."""
    out = np.empty((n, l), dtype=np.float32)
    for c, a in enumerate(range(0, n, CHUNK_ROWS)):
        b = min(n, a + CHUNK_ROWS)
        out[a:b] = _rng(seed, 5, c).standard_normal((b - a, l), dtype=np.float32)
    out *= np.float32(1.0 / np.sqrt(n))
    return out


@dataclass
class Workload:
    cfg: Config
    X: np.ndarray        # n x d float32
    labels: np.ndarray   # n int32
    r: np.ndarray        # s int64
    seed: int

    @property
    def n(self):
        return self.X.shape[0]

    def y(self, idx: np.ndarray) -> np.ndarray:
        return one_hot(self.labels[idx], self.cfg.l)


def make_workload(cfg: Config, seed: int = 0, n: int = None) -> Workload:
    X = features(cfg, seed, n)
    labels = class_labels(cfg, X, seed)
    r = subsample_indices(cfg, seed, n=X.shape[0])
    return Workload(cfg, X, labels, r, seed)
