"""Realizations of other shapes <m,k,n;R> in the C-ABI library, on the CPU:
the coefficients round-trip, Phi, Gamma and the Brent residual agree with
the oracle's, a perturbed coefficient is refused, the gauge agrees with the
oracle's formula applied to rows of length mk and kn, the calls that are
<2,2,2>'s alone say so, and plans are validated before any device call.
The realizations are fmm_inputs.shapes' constructions on each side's own
<2,2,2> tables (the library's builtins, the oracle's)."""
import os

import numpy as np
import pytest

from fmm_inputs import shapes as S
from oracle import realizations as R
from oracle import shapes as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2609_26077_amd", "libfmm8.so")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libfmm8.so not built")


@pytest.fixture(scope="module")
def fm():
    import paper_2609_26077_amd as fm
    return fm


def lib_base(fm):
    def base(which):
        return fm.fmm_realization_coefficients(fm.fmm_realization_builtin(which))
    return base


def lib_shaped(fm, name, tol=1e-9):
    (m, k, n), U, V, W = S.build(name, lib_base(fm))
    return fm.fmm_realization_create(U, V, W, tol=tol, shape=(m, k, n))


@pytest.mark.parametrize("name", sorted(S.CATALOG))
def test_coefficients_round_trip_and_metrics(fm, name):
    d = lib_shaped(fm, name)
    shape, rank = S.CATALOG[name]
    assert fm.fmm_realization_shape(d) == (shape, rank)
    assert fm.fmm_realization_terms(d, 1) == (rank, rank)
    D = S.build(name, R.builtin_f64)
    got = fm.fmm_realization_coefficients(d)
    for a, b in zip(got, D[1:]):
        assert np.array_equal(a, b)
    m = fm.fmm_realization_metrics(d, 1)
    assert m["phi"] == pytest.approx(O.phi(D), rel=1e-14)
    assert m["gamma"] == pytest.approx(O.gamma(D), rel=1e-14)
    # integer coefficients: every Brent sum is exact in binary64; T*'s to rounding
    assert m["brent_residual"] == 0.0 or (name == "223_tstar" and m["brent_residual"] < 1e-15)
    U, V, W = fm.fmm_realization_tables(d, 1)
    for a, b in zip((U, V, W), O.tables_f32(D)):
        assert a.dtype == np.float32 and np.array_equal(a, b)


def test_perturbed_coefficient_is_refused(fm):
    (m, k, n), U, V, W = S.build("333_26", lib_base(fm))
    for which in range(3):
        X = [U.copy(), V.copy(), W.copy()]
        X[which][20, 3] += 1e-6
        with pytest.raises(fm.FmmError) as e:
            fm.fmm_realization_create(*X, tol=1e-9, shape=(m, k, n))
        assert e.value.status == fm.FMM_ERR_NOT_EXACT
        d = fm.fmm_realization_create(*X, tol=1e-5, shape=(m, k, n))   # within a looser tolerance
        assert 0 < fm.fmm_realization_metrics(d, 1)["brent_residual"] <= 1e-5


def test_gauge_of_other_shapes(fm):
    """(U_r, V_r, W_r) -> (U_r / s_r, s_r V_r, W_r), s_r = sqrt(|U_r| / |V_r|),
    binary64; the result stays exact and its Phi does not change (the gauge
    keeps |U_r| |V_r|, hence each term's weight)."""
    d = lib_shaped(fm, "223_tstar")
    U, V, W = fm.fmm_realization_coefficients(d)
    g = fm.fmm_realization_rebalance(d)
    Ug, Vg, Wg = fm.fmm_realization_coefficients(g)
    for r in range(U.shape[0]):
        nu = np.sqrt(sum(float(x) * float(x) for x in U[r]))
        nv = np.sqrt(sum(float(x) * float(x) for x in V[r]))
        s = np.sqrt(nu / nv)
        assert np.array_equal(Ug[r], U[r] / s) and np.array_equal(Vg[r], V[r] * s)
    assert np.array_equal(Wg, W)
    mg = fm.fmm_realization_metrics(g, 1)
    assert mg["brent_residual"] < 1e-14
    assert mg["phi"] == pytest.approx(fm.fmm_realization_metrics(d, 1)["phi"], rel=1e-14)


def test_deeper_levels_refuse_other_shapes(fm):
    d = lib_shaped(fm, "223_11")
    for call in (lambda: fm.fmm_realization_metrics(d, 2),
                 lambda: fm.fmm_realization_terms(d, 2),
                 lambda: fm.fmm_realization_tables(d, 2)):
        with pytest.raises(fm.FmmError) as e:
            call()
        assert e.value.status == fm.FMM_ERR_UNSUPPORTED


@pytest.mark.parametrize("name", ["223_11", "232_11", "333_26", "525_46"])
def test_transform_matches_oracle(fm, name):
    """The orbit action u -> u (X (x) Y^-T) etc. over GL(m) x GL(k) x GL(n):
    the library (Gauss-Jordan inverses) against the oracle (numpy's) to
    rounding, and the result exact to rounding."""
    import fmm_inputs as gen
    d = lib_shaped(fm, name)
    D = S.build(name, R.builtin_f64)
    (m, k, n) = D[0]
    for g in gen.rebasing_starts_shape(4, m, k, n, seed=0, cfg=21):
        X, Y, Z = O.split_g(g, (m, k, n))
        got = fm.fmm_realization_coefficients(fm.fmm_realization_transform(d, X, Y, Z))
        want = O.act(D, X, Y, Z)[1:]
        for a, b in zip(got, want):
            assert np.allclose(a, b, rtol=1e-13, atol=1e-13 * np.abs(b).max())
        assert fm.fmm_realization_metrics(fm.fmm_realization_transform(d, X, Y, Z))["brent_residual"] < 1e-12


def test_transform_rejects_singular(fm):
    d = lib_shaped(fm, "223_11")
    Z = np.eye(3); Z[2] = Z[1]
    with pytest.raises(fm.FmmError) as e:
        fm.fmm_realization_transform(d, np.eye(2), np.eye(2), Z)
    assert e.value.status == fm.FMM_ERR_SINGULAR


@pytest.mark.parametrize("name", ["223_11", "333_26", "525_46"])
def test_phi_gradient_matches_oracle(fm, name):
    """The library's closed-form gradient (2 X^-T sum_r (b c U'U'^T -
    a b W'^T W') and its companions) against the oracle's chain rule through
    the Kronecker matrices."""
    import fmm_inputs as gen
    d = lib_shaped(fm, name)
    D = S.build(name, R.builtin_f64)
    (m, k, n) = D[0]
    for g in gen.rebasing_starts_shape(3, m, k, n, seed=0, cfg=22):
        phi, grad = fm.fmm_realization_phi_gradient(d, g)
        phi_o, grad_o = O.phi_and_grad(D, g)
        assert phi == pytest.approx(phi_o, rel=1e-13)
        assert np.allclose(grad, grad_o, rtol=1e-11, atol=1e-11 * np.abs(grad_o).max())


def test_optimize_matches_oracle(fm):
    """Re-basing <2,2,3;11> from the identity and 8 perturbed starts: the
    least terminal Phi equals the oracle's (scipy L-BFGS-B from the same
    starts), every start's terminal realization is exact, and Phi drops
    from 36."""
    import fmm_inputs as gen
    d = lib_shaped(fm, "223_11")
    D = S.build("223_11", R.builtin_f64)
    starts = gen.rebasing_starts_shape(8, 2, 2, 3, seed=0, cfg=23)
    best, phi, term = fm.fmm_realization_optimize(d, starts)
    _, phi_o, term_o = O.rebase(D, starts)
    assert phi == pytest.approx(phi_o, rel=1e-9)
    assert phi < 36.0 - 1.0
    assert fm.fmm_realization_metrics(best)["brent_residual"] < 1e-12
    assert np.all(np.isfinite(term))


def test_optimize_cubic_returns_mkn(fm):
    """The cubic algorithm's orbit minimum is mkn (the oracle's test states
    why): from random starts the library returns 24 for <2,3,4>."""
    import fmm_inputs as gen
    from paper_2609_26077_amd.controls import shaped_realization
    d = shaped_realization("cubic_234")
    best, phi, term = fm.fmm_realization_optimize(d, gen.rebasing_starts_shape(4, 2, 3, 4, seed=0, cfg=24))
    assert phi == pytest.approx(24.0, rel=1e-9)
    assert np.allclose(term, 24.0, rtol=1e-8)


@pytest.mark.parametrize("name,desc,status", [
    ("223_11", dict(M=512, K=256, N=768, depth=2), -3),              # one level only
    ("223_11", dict(M=512, K=256, N=768, flags=2), -3),              # no deployment granularity
    ("223_11", dict(M=512, K=256, N=768, flags=4), -3),
    ("223_11", dict(M=512, K=256, N=512), -2),                       # N not divisible by n = 3
    ("322_11", dict(M=512, K=256, N=512), -2),                       # M not divisible by m = 3
    ("232_11", dict(M=512, K=256, N=512), -2),                       # K not divisible by k = 3
    ("223_11", dict(M=512, K=96, N=768), -2),                        # K / k = 48 not / 32
    ("223_11", dict(M=512, K=256, N=384), -3),                       # N / n = 128: not whole 256-row tiles
    ("223_11", dict(M=384, K=256, N=768), -3),                       # M / m = 192
    ("223_11", dict(M=512, K=192, N=768, block=32), -3),             # K / k = 96: not whole 64-byte steps
    ("223_11", dict(M=512, K=64, N=768, block=16), -3),              # K / k = 32 at block 16
    ("223_11", dict(M=512, K=256, N=768, flags=16), -1),             # unknown flag bit
])
def test_plan_validation_before_device(fm, name, desc, status):
    d = lib_shaped(fm, name)
    kw = dict(batch=1, M=256, K=256, N=256, depth=1, block=32, rule="pow2_ceil")
    kw.update(desc)
    assert fm.fmm_plan_create_status(d, fm.make_desc(**kw)) == status
