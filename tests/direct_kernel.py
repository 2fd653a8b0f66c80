"""Kernel matrices from direct coordinate differences (scipy's cdist), an
evaluation route independent of the oracle's expansion |a|^2 + |b|^2 - 2 a.b:
the pins compare the oracle against it, and a row's distance to itself is
exactly zero here."""

import numpy as np
from scipy.spatial.distance import cdist

GAUSSIAN = 0
LAPLACIAN = 1


def kmat(A, B, kernel, bw):
    d2 = cdist(np.asarray(A, dtype=np.float64), np.asarray(B, dtype=np.float64), "sqeuclidean")
    if kernel == GAUSSIAN:
        return np.exp(-d2 / (2.0 * bw * bw))
    return np.exp(-np.sqrt(d2) / bw)
