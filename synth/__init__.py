"""Seeded synthetic workloads for the EigenPro 2.0 step.

This package holds input recipes and random draws only. It contains none of
the method's arithmetic (no kernel evaluation, no eigensystem, no step), so
both the fp64 oracle and the HIP path can consume the same arrays without
sharing any computation.
"""

from .configs import CONFIGS, Config, get_config
from .generate import (
    Workload,
    make_workload,
    features,
    heldout,
    class_labels,
    one_hot,
    subsample_indices,
    epoch_permutation,
    epoch_batches,
    initial_alpha,
)

__all__ = [
    "CONFIGS",
    "Config",
    "get_config",
    "Workload",
    "make_workload",
    "features",
    "heldout",
    "class_labels",
    "one_hot",
    "subsample_indices",
    "epoch_permutation",
    "epoch_batches",
    "initial_alpha",
]
