"""The five synthetic workload shapes.

Each stands in for one of the paper's data sets (Section 5 and Appendix A:
MNIST, CIFAR-10, TIMIT, ImageNet features) by its size, feature dimension,
label count and value distribution after the paper's preprocessing. None of
the real data sets is used or reproduced. Kernel, bandwidth, subsample size s
and EigenPro rank k follow the workload definitions; where a batch size is
not fixed, it is the analytic critical batch size computed at setup.
"""

from dataclasses import dataclass
from typing import Optional


@dataclass(frozen=True)
class Config:
    name: str
    n: int              # centres = training points
    d: int              # features
    l: int              # one-hot label columns
    x_law: str          # feature distribution, see synth.generate.features
    label_rule: str     # "argmax_linear" or "nearest_mean"
    kernel: str         # "gaussian" or "laplacian"
    bandwidth: float
    s: int              # subsample (fixed coordinate block) size
    k: int              # EigenPro rank: top-k directions flattened to sigma_{k+1}
    m: Optional[int]    # fixed batch size, or None for the analytic m*
    epochs: int         # epochs used by the one-epoch / multi-epoch checks
    n_z: int            # held-out prediction points

    @property
    def kernel_id(self) -> int:
        return {"gaussian": 0, "laplacian": 1}[self.kernel]


CONFIGS = {
    "tiny": Config("tiny", 2000, 64, 4, "normal_scaled", "argmax_linear",
                   "gaussian", 1.0, 500, 20, 256, 3, 500),
    "mnist": Config("mnist", 60000, 784, 10, "uniform_sparse80", "nearest_mean",
                    "gaussian", 5.0, 4000, 160, None, 1, 10000),
    "cifar": Config("cifar", 50000, 3072, 10, "uniform", "nearest_mean",
                    "laplacian", 10.0, 4000, 200, None, 1, 10000),
    "timit": Config("timit", 1100000, 440, 144, "normal", "nearest_mean",
                    "gaussian", 15.0, 12000, 160, None, 1, 10000),
    "imagenet": Config("imagenet", 1280000, 2048, 1000, "halfnormal_sparse50",
                       "nearest_mean", "gaussian", 20.0, 20000, 200, None, 1, 10000),
}


def get_config(name: str, **overrides) -> Config:
    """Return a named config, optionally with fields replaced (e.g. n for a
    row-prefix of the same workload)."""
    cfg = CONFIGS[name]
    if overrides:
        fields = {**cfg.__dict__, **overrides}
        cfg = Config(**fields)
    return cfg
