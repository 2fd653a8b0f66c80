"""Section 3 Step 1's compute-limited batch m_C: the knee of time per
iteration against batch size (ep_batch_knee, host-only, no GPU needed)."""

import numpy as np
import pytest

import paper_1806_06144_amd as ep

GRID = [2 ** j for j in range(4, 15)]


def test_exact_hinge_gives_its_knee():
    t0, a = 0.3, 1e-3                       # knee t0 / a = 300
    t = [max(t0, a * m) for m in GRID]
    mc, knee = ep.ep_batch_knee(GRID, t, 0.0)
    assert knee == pytest.approx(300.0, rel=1e-9)
    assert mc == 512                        # smallest power of two >= 300
    mc, _ = ep.ep_batch_knee(GRID, t, 0.5)  # (1 - tol) knee = 150
    assert mc == 256


def test_flat_and_linear_curves():
    assert ep.ep_batch_knee(GRID, [1.0] * len(GRID), 0.1)[0] == GRID[-1]
    assert ep.ep_batch_knee(GRID, [1e-3 * m for m in GRID], 0.1)[0] == GRID[0]


def test_reproducible_under_timing_noise():
    """A measured-shaped curve (flat, a soft transition, then linear) with
    3 % multiplicative noise, as the median of three noisy sweeps: the same
    m_C comes back for every draw, and the knee stays within 10 %."""
    base = np.array([0.306, 0.305, 0.304, 0.315, 0.343, 0.602, 1.115, 2.046, 3.915, 7.770,
                     15.460])
    ref_mc, ref_knee = ep.ep_batch_knee(GRID, base, 0.1)
    rng = np.random.default_rng(0)
    for _ in range(50):
        sweeps = base * (1.0 + 0.03 * rng.standard_normal((3, base.size)))
        mc, knee = ep.ep_batch_knee(GRID, np.median(sweeps, axis=0), 0.1)
        assert mc == ref_mc
        assert knee == pytest.approx(ref_knee, rel=0.1)


@pytest.mark.parametrize("ms,t,tol", [
    ([16], [1.0], 0.1), ([32, 16], [1.0, 1.0], 0.1), ([0, 16], [1.0, 1.0], 0.1),
    ([16, 32], [1.0, 0.0], 0.1), ([16, 32], [1.0, float("nan")], 0.1), ([16, 32], [1.0, 2.0], 1.0),
])
def test_rejects_bad_input(ms, t, tol):
    with pytest.raises(ep.EigenProError) as e:
        ep.ep_batch_knee(ms, t, tol)
    assert e.value.code == ep.EP_EINVAL
