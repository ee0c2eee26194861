"""The oracle's re-basing (Appendix E.2 protocol; Section 3.1) against what
the paper and the mathematics fix: the gradient against central differences,
the certified orbit minimum Phi = 200/9 (Theorem 1) with Gamma at its optimum
2 sqrt 2 + 16 / sqrt 3 from Strassen, the Winograd variant and random orbit
points of T*, stationarity of T* and of the cubic algorithm, exactness of the
terminal realizations, and the exactness gate on a corrupted realization."""
import math

import numpy as np
import pytest

import fmm_inputs as gen
from oracle import realizations as R
from oracle import rebase as RB

PHI_MIN = 200.0 / 9.0
GAMMA_MIN = 2.0 * math.sqrt(2.0) + 16.0 / math.sqrt(3.0)


@pytest.mark.parametrize("name", ["strassen", "winograd", "tstar", "cubic8"])
def test_gradient_matches_central_differences(name):
    D = R.builtin_f64(name)
    for x in [RB.IDENTITY] + list(gen.rebasing_starts(4, seed=3)):
        phi, grad = RB.phi_and_grad(D, x)
        fd = np.empty(12)
        for i in range(12):
            h = 1e-6 * max(1.0, abs(x[i]))
            e = np.zeros(12)
            e[i] = h
            fd[i] = (RB.phi_and_grad(D, x + e)[0] - RB.phi_and_grad(D, x - e)[0]) / (2 * h)
        assert np.max(np.abs(grad - fd)) <= 1e-6 * max(1.0, np.max(np.abs(fd))), (name, x)


def test_objective_is_phi_of_the_transformed_realization():
    D = R.builtin_f64("strassen")
    for x in gen.rebasing_starts(5, seed=4):
        g = tuple(np.asarray(x).reshape(3, 2, 2))
        assert RB.phi_and_grad(D, x)[0] == pytest.approx(R.phi_f64(R.act_f64(D, g)), rel=1e-13)


@pytest.mark.parametrize("name", ["tstar", "cubic8"])
def test_orbit_minima_are_stationary(name):
    # T* (moment map zero, Appendix A) and the cubic algorithm are critical points
    phi, grad = RB.phi_and_grad(R.builtin_f64(name), RB.IDENTITY)
    assert np.max(np.abs(grad)) < 1e-12 * phi
    assert phi == pytest.approx({"tstar": PHI_MIN, "cubic8": 8.0}[name], rel=1e-15)


@pytest.mark.parametrize("name", ["strassen", "winograd"])
def test_rebasing_reaches_the_certified_minimum(name):
    D = R.builtin_f64(name)
    best, phi, terminal = RB.rebase(D, gen.rebasing_starts(23, seed=0))
    assert phi == pytest.approx(PHI_MIN, rel=1e-12)
    assert R.gamma_f64(best) == pytest.approx(GAMMA_MIN, rel=1e-10)
    assert R.brent_residual_f64(best) <= 1e-12
    # Phi is geodesically convex on the orbit: every start ends at the minimum
    assert np.all(np.abs(terminal - PHI_MIN) <= 1e-9 * PHI_MIN)


def test_random_orbit_points_of_tstar_rebase_back():
    T = R.builtin_f64("tstar")
    for x in gen.rebasing_starts(3, seed=9):
        D = R.act_f64(T, tuple(np.asarray(x).reshape(3, 2, 2)))
        assert R.phi_f64(D) > PHI_MIN * (1 + 1e-3)
        best, phi, _ = RB.rebase(D)
        assert phi == pytest.approx(PHI_MIN, rel=1e-12)
        assert R.gamma_f64(best) == pytest.approx(GAMMA_MIN, rel=1e-10)


def test_cubic_orbit_minimum_is_eight():
    C = R.builtin_f64("cubic8")
    x = gen.rebasing_starts(1, seed=5)[0]
    D = R.act_f64(C, tuple(x.reshape(3, 2, 2)))
    assert R.phi_f64(D) > 8.5
    _, phi, _ = RB.rebase(D)
    assert phi == pytest.approx(8.0, rel=1e-12)


def test_exactness_gate_rejects_a_corrupted_realization():
    U, V, W = (np.array(M) for M in R.builtin_f64("strassen"))
    U[2, 0] = -U[2, 0]                      # one flipped sign: no longer a <2,2,2> algorithm
    best, phi, terminal = RB.rebase((U, V, W), gen.rebasing_starts(2, seed=0))
    assert best is None and np.isinf(phi) and np.all(np.isnan(terminal))
