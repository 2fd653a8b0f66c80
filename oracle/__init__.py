"""fp64 CPU oracle for the EigenPro 2.0 iteration — TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package. The product (the HIP library and its
Python binding) never calls it and shares no code with it.

Everything here is a plain, slow, obviously correct NumPy/SciPy rendering of
the paper's definitions in float64. See ``oracle.eigenpro`` for the functions
and the passages each one follows.
"""

from .eigenpro import (
    GAUSSIAN,
    LAPLACIAN,
    OracleState,
    sq_dist,
    kernel_matrix,
    top_eigenpairs,
    DENSE_EIG_MAX_S,
    setup,
    step_coefficient,
    beta_closed_form,
    step,
    step_pointwise,
    predict,
    run_epoch,
    interpolant,
    with_rank,
    choose_rank,
    acceleration,
)

__all__ = [
    "GAUSSIAN",
    "LAPLACIAN",
    "OracleState",
    "sq_dist",
    "kernel_matrix",
    "top_eigenpairs",
    "DENSE_EIG_MAX_S",
    "setup",
    "step_coefficient",
    "beta_closed_form",
    "step",
    "step_pointwise",
    "predict",
    "run_epoch",
    "interpolant",
    "with_rank",
    "choose_rank",
    "acceleration",
]
