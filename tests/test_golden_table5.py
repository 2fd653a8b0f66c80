"""The step-size reading against the values printed in Table 5 (Appendix B).

Reading: eta(m) = m / (beta + (m - 1) lambda), applied as a per-coordinate
step eta/m. At the analytic batch m = m* = beta / lambda this gives
m / eta = 2 beta - lambda. With a normalised shift-invariant kernel
0 < beta <= 1 and 0 < lambda << 1 (lambda ~ 1/m*), so m / eta lies just
below 2. Section 3 Step 3 taken literally (eta = m / beta) would give
m / eta = beta <= 1 instead. Every printed row falls in the first band.
"""

import os

import numpy as np

import oracle

HERE = os.path.dirname(__file__)


def _rows():
    rows = []
    with open(os.path.join(HERE, "golden", "table5_parameters.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            name, q, qa, m, eta = line.split()
            rows.append((name, int(m), float(eta)))
    return rows


def test_printed_ratios_match_the_reading():
    rows = _rows()
    assert len(rows) == 4
    for name, m, eta in rows:
        ratio = m / eta
        # beta in [0.95, 1], lambda = beta / m
        lo = 2 * 0.95 - 1.0 / m
        hi = 2 * 1.0
        assert lo < ratio < hi, (name, ratio)
        assert ratio > 1.0, (name, ratio)   # the literal reading gives <= 1


def test_oracle_coefficient_at_critical_batch():
    # the oracle's coefficient reproduces the 2 beta - lambda band at m = m*
    rng = np.random.default_rng(0)
    X = rng.standard_normal((300, 20)) / np.sqrt(20)
    st = oracle.setup(X, oracle.GAUSSIAN, 1.0, 300, 10, np.arange(300))
    m = st.m_star
    eta = m * oracle.step_coefficient(st.beta, st.lam, m)
    assert m / eta == np.float64(2 * st.beta - st.lam) or abs(m / eta - (2 * st.beta - st.lam)) < 1e-12
