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


def test_222_only_calls_refuse_other_shapes(fm):
    d = lib_shaped(fm, "223_11")
    I = np.eye(2).ravel()
    for call in (lambda: fm.fmm_realization_transform(d, I, I, I),
                 lambda: fm.fmm_realization_optimize(d),
                 lambda: fm.fmm_realization_phi_gradient(d, np.tile(I, 3)),
                 lambda: fm.fmm_realization_metrics(d, 2),
                 lambda: fm.fmm_realization_terms(d, 2),
                 lambda: fm.fmm_realization_tables(d, 2)):
        with pytest.raises(fm.FmmError) as e:
            call()
        assert e.value.status == fm.FMM_ERR_UNSUPPORTED


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
