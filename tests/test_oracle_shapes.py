"""The oracle for realizations of other shapes <m,k,n;R> (oracle/shapes.py),
pinned to what the mathematics fixes: the Brent equations in exact
arithmetic (and a perturbed coefficient fails them), the exact product on
integer matrices with and without the quantizer (any index mistake in the
grids or the cyclic third factor breaks it), Phi of a direct sum as the sum
of the parts' Phi and of the cubic algorithm as mkn, agreement bit for bit
with the <2,2,2> oracle, and the second-moment model of Appendix D
(E|dC|^2 / E|C|^2 ~ 2 s_q^2 Phi / (m k n))."""
import numpy as np
import pytest

import fmm_inputs as gen
from fmm_inputs import shapes as S
from oracle import e4m3, fmm, model, shapes
from oracle import realizations as R


def shaped(name):
    """A realization of fmm_inputs.shapes.CATALOG built on the oracle's
    <2,2,2> tables, or the oracle's Strassen itself."""
    if name == "222_strassen":
        return S.from_222(R.builtin_f64("strassen"))
    return S.build(name, R.builtin_f64)


@pytest.mark.parametrize("mkn", [(2, 2, 3), (3, 2, 2), (2, 3, 2), (3, 3, 3), (1, 2, 3), (2, 1, 1)])
def test_cubic_is_exact_with_phi_mkn(mkn):
    D = S.cubic(*mkn)
    assert len(D[1]) == mkn[0] * mkn[1] * mkn[2]
    assert shapes.brent_exact(D)
    assert shapes.phi(D) == mkn[0] * mkn[1] * mkn[2]


# Phi of a direct sum is the sum of the parts' Phi (the re-indexing keeps
# every norm): Strassen's terms give 8 + 6 * 4 = 32, T*'s 200/9, a cubic term 1
@pytest.mark.parametrize("name,phi", [("223_11", 32.0 + 4), ("322_11", 32.0 + 4), ("232_11", 32.0 + 4),
                                      ("223_tstar", 200 / 9 + 4), ("333_26", 32.0 + 19),
                                      ("333_27", 27.0), ("525_46", 4 * 32.0 + 18), ("454_80", 80.0)])
def test_catalog_is_exact_with_its_phi(name, phi):
    D = shaped(name)
    shape, rank = S.CATALOG[name]
    assert D[0] == shape and len(D[1]) == rank
    if name != "223_tstar":          # T*'s entries are irrational in binary64; exactness there is to rounding
        assert shapes.brent_exact(D)
    assert shapes.phi(D) == pytest.approx(phi, rel=1e-13)


def test_perturbed_direct_sum_fails_brent():
    for part in (1, 2, 3):
        D = list(shaped("223_11"))
        M = np.array(D[part])
        M[8, 0] = 1 - M[8, 0]                # flip one coefficient of a cubic term
        D[part] = M
        assert not shapes.brent_exact(tuple(D))


@pytest.mark.parametrize("name", ["223_11", "322_11", "232_11", "333_27"])
def test_bilinear_map_is_the_product_on_integers(name):
    D = shaped(name)
    m, k, n = D[0]
    rng = np.random.default_rng(7)
    A = rng.integers(-9, 10, size=(m * 6, k * 5)).astype(np.float64)
    B = rng.integers(-9, 10, size=(k * 5, n * 4)).astype(np.float64)
    assert np.array_equal(shapes.exact_product(A, B, D), A @ B)


@pytest.mark.parametrize("name", ["223_11", "322_11", "232_11"])
@pytest.mark.parametrize("rule", [e4m3.RULE_POW2_CEIL, e4m3.RULE_POW2_OCP])
def test_quantized_evaluation_exact_on_sign_operands(name, rule):
    """With +-1 and 0 operands and +-1 coefficients every combination is a
    small integer, exactly representable after either power-of-two scale, so
    the whole fused evaluation (split, combine, quantize, products,
    W-combine) must return A B exactly; a wrong block index anywhere breaks
    it."""
    D = shaped(name)
    m, k, n = D[0]
    rng = np.random.default_rng(11)
    A = rng.integers(-1, 2, size=(m * 8, k * 64)).astype(np.float32)
    B = rng.integers(-1, 2, size=(k * 64, n * 8)).astype(np.float32)
    o = shapes.fmm_shape(A, B, D, 32, rule)
    assert np.array_equal(o["C"], A.astype(np.float64) @ B.astype(np.float64))


def test_agrees_with_the_222_oracle_bit_for_bit():
    D = R.builtin_f64("strassen")
    A, B = gen.operands("gaussian", 1, 128, 256, 192, seed=0, cfg=16, trial=0)
    want = fmm.fmm(A[0], B[0], R.tables_f32(D, 1), 1, 32, e4m3.RULE_POW2_CEIL)
    got = shapes.fmm_shape(A[0], B[0], S.from_222(D), 32, e4m3.RULE_POW2_CEIL)
    assert np.array_equal(got["a"]["codes"], want["a"]["codes"])
    assert np.array_equal(got["b"]["codes"], want["b"]["codes"])
    assert np.array_equal(got["a"]["scales"], want["a"]["scales"])
    assert np.array_equal(got["b"]["scales"], want["b"]["scales"])
    assert np.array_equal(got["C"], want["C"])


@pytest.mark.parametrize("name", ["223_11", "223_tstar", "333_27"])
def test_model_predicts_measured(name):
    """Appendix D's model with the measured noise coefficients predicts the
    measured relative MSE within a few percent at shape <m,k,n> (mkn in place
    of 8)."""
    D = shaped(name)
    m, k, n = D[0]
    errs, refs, sa, sb = [], [], [], []
    for t in range(3):
        A, B = gen.operands("gaussian", 1, 64 * m, 64 * k, 64 * n, seed=0, cfg=17, trial=t)
        o = shapes.fmm_shape(A[0], B[0], D, 32, e4m3.RULE_POW2_CEIL)
        e2, r2 = fmm.error_sums(o["C"], fmm.reference(A[0], B[0]))
        errs.append(e2); refs.append(r2)
        sa.append(model.noise_coefficient(o["a"]["x"], o["a"]["deq"]))
        sb.append(model.noise_coefficient(o["b"]["x"], o["b"]["deq"]))
    rel = np.sum(errs) / np.sum(refs)
    s_a2, s_b2 = np.mean(sa), np.mean(sb)
    pred = (s_a2 + s_b2 + s_a2 * s_b2) * shapes.phi(D) / (m * k * n)
    assert pred / rel == pytest.approx(1.0, abs=0.06), (pred, rel)


# ---- the orbit GL(m) x GL(k) x GL(n) and re-basing ---------------------------

def rational_g(rng, shape):
    """A random rational (X, Y, Z) with nonzero determinants."""
    from fractions import Fraction
    out = []
    for size in shape:
        while True:
            M = [[Fraction(int(rng.integers(-4, 5)), int(rng.integers(1, 4))) + (1 if i == j else 0)
                  for j in range(size)] for i in range(size)]
            import sympy
            if sympy.Matrix(M).det() != 0:
                out.append(M)
                break
    return out


@pytest.mark.parametrize("name", ["223_11", "232_11", "333_26"])
def test_action_keeps_exactness_in_rational_arithmetic(name):
    """u -> u (X (x) Y^-T) and its cyclic companions keep the Brent equations
    exactly (<U', A> = <U, X A Y^-1>, so the trilinear form becomes
    tr(X A B C X^-1)); Y^-1 in place of Y^-T breaks them."""
    import sympy
    D = shaped(name)
    rng = np.random.default_rng(3)
    X, Y, Z = rational_g(rng, D[0])
    Dg = shapes.act_exact(D, X, Y, Z)
    assert shapes.brent_exact(Dg)
    # the plausible slip: no transpose on the inverse
    (m, k, n), U, V, W = D
    Ky = sympy.kronecker_product(sympy.Matrix(X), sympy.Matrix(Y).inv())
    bad = (D[0], [list(sympy.Matrix([[sympy.Rational(x) for x in r]]) * Ky) for r in np.asarray(U).astype(int).tolist()],
           Dg[2], Dg[3])
    assert not shapes.brent_exact(bad)


def test_action_at_222_is_the_222_oracles():
    D = R.builtin_f64("strassen")
    for g in gen.basis_changes(5, seed=0, cfg=17):
        _, U, V, W = shapes.act(S.from_222(D), *g)
        want = R.act_f64(D, g)
        for a, b in zip((U, V, W), want):
            assert np.allclose(a, np.asarray(b, float), rtol=1e-14, atol=1e-14)


@pytest.mark.parametrize("name", ["223_11", "333_26", "525_46"])
def test_gradient_against_central_differences(name):
    D = shaped(name)
    (m, k, n) = D[0]
    g = gen.rebasing_starts_shape(1, m, k, n, seed=0, cfg=18)[0]
    f, grad = shapes.phi_and_grad(D, g)
    h = 1e-6
    for i in range(0, g.size, max(1, g.size // 12)):
        e = np.zeros_like(g); e[i] = h
        fd = (shapes.phi_and_grad(D, g + e)[0] - shapes.phi_and_grad(D, g - e)[0]) / (2 * h)
        assert fd == pytest.approx(grad[i], rel=1e-6, abs=1e-6 * np.abs(grad).max())


@pytest.mark.parametrize("mkn", [(2, 2, 3), (2, 3, 4), (3, 3, 3)])
def test_cubic_orbit_minimum_is_mkn(mkn):
    """The cubic algorithm's orbit has Phi >= mkn, equality at g = 1: term
    (i, j, l) maps to rank-one matrices, |X^T e_i e_j^T Y^-T|^2 =
    |X^T e_i|^2 |Y^-1 e_j|^2, so Phi(cubic . g) factors into
    (sum_i |X^T e_i|^2 |X^-1 e_i|^2)(sum_j ...)(sum_l ...), and each summand
    is >= 1 by Cauchy-Schwarz, since row i of X times column i of X^-1 is 1.
    Random orbit points respect the bound and re-basing from random starts
    returns mkn."""
    m, k, n = mkn
    C = S.cubic(m, k, n)
    starts = gen.rebasing_starts_shape(6, m, k, n, seed=0, cfg=19)
    for g in starts:
        assert shapes.phi(shapes.act(C, *shapes.split_g(g, mkn))) >= m * k * n * (1 - 1e-12)
    _, best, term = shapes.rebase(C, starts)
    assert best == pytest.approx(m * k * n, rel=1e-9)
    assert np.allclose(term, m * k * n, rtol=1e-8)


def test_scalar_gauge_leaves_phi():
    D = shaped("333_26")
    I3 = np.eye(3)
    assert shapes.phi(shapes.act(D, 2.0 * I3, 0.5 * I3, 3.0 * I3)) == pytest.approx(shapes.phi(D), rel=1e-14)


def test_rebase_lowers_phi_and_stays_exact():
    D = shaped("223_11")
    best, phi, term = shapes.rebase(D, gen.rebasing_starts_shape(5, 2, 2, 3, seed=0, cfg=20))
    assert phi < shapes.phi(D) - 1.0
    assert shapes.brent_residual(best) < 1e-12
    ident = np.concatenate([np.eye(2).ravel(), np.eye(2).ravel(), np.eye(3).ravel()])
    _, grad = shapes.phi_and_grad(best, ident)          # stationary where it ended
    assert np.abs(grad).max() <= 1e-6 * phi
