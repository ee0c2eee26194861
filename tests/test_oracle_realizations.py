"""Pins of the oracle's coefficient algebra against what the paper fixes.

Every check here compares the oracle with an independent fact: the Brent
equations (exact arithmetic), the paper's printed coordinates and matrices
(tests/golden), closed forms of Section 3 and Appendices A and C, or an
invariance that holds by construction.
"""
import itertools

import mpmath as mp
import numpy as np
import pytest
import sympy as sp

from oracle import realizations as R
from tests.conftest import golden

NAMES = ["cubic8", "strassen", "winograd", "tstar"]


def _sym(s, extra=None):
    loc = {"sqrt": sp.sqrt, "xi": R.XI, "eta": R.ETA, "zeta": R.ZETA,
           "rho": R.RHO}
    if extra:
        loc.update(extra)
    return sp.sympify(s, locals=loc)


@pytest.mark.parametrize("name", NAMES)
def test_brent_exact(name):
    """Each named realization multiplies 2x2 matrices exactly (Section 2.1)."""
    assert R.brent_exact(R.builtin(name))


def test_brent_rejects_a_sign_flip():
    """The exactness check is not vacuous: one flipped coefficient fails."""
    U, V, W = R.builtin("strassen")
    W = W.copy(); W[4, 0] = -W[4, 0]
    assert not R.brent_exact((U, V, W))


def test_tstar_matches_printed_coordinates():
    g = golden("tstar.json")
    U, V, W = R.tstar()
    Ug = sp.Matrix([[_sym(x) for x in row] for row in g["U_star"]])
    assert sp.simplify(U - Ug) == sp.zeros(7, 4)
    for r in range(7):
        assert sp.simplify(V.row(r) - Ug.row(g["pi_V"][r] - 1)) == sp.zeros(1, 4)
        assert sp.simplify(W.row(r) - Ug.row(g["pi_W"][r] - 1)) == sp.zeros(1, 4)


def test_k_rho_is_the_printed_matrix():
    """K_rho = T_rho (x) T_rho^-T equals the display of Appendix A."""
    g = golden("k_rho.json")
    T = sp.Matrix([[_sym(x) for x in row] for row in g["T_rho"]])
    assert sp.simplify(T - R.t_rho()) == sp.zeros(2, 2)
    K = R.kron2(T, T.inv().T)
    Kg = sp.Matrix([[_sym(x) for x in row] for row in g["K_rho"]])
    assert sp.simplify(K - Kg) == sp.zeros(4, 4)


def test_tstar_is_strassen_under_the_balanced_sandwich():
    """T* = Strassen . (T_rho, T_rho, T_rho) (Theorem 1), exactly; this pins the
    order and signs of the Strassen table, which the paper does not print."""
    T = R.t_rho()
    got = R.act_exact(R.strassen(), (T, T, T))
    want = R.tstar()
    for a, b in zip(got, want):
        assert sp.simplify(a - b) == sp.zeros(7, 4)


def test_tstar_row_norms():
    """a_r = |U*_r|^2 = |V*_r|^2 = |W*_r|^2 = (2, 4/3, ..., 4/3) (eq. A.3)."""
    g = golden("tstar.json")
    want = [sp.Rational(x) for x in g["a_r"]]
    for M in R.tstar():
        assert R.row_sq_norms(M) == want


@pytest.mark.parametrize("name,phi,gam", [
    ("cubic8", "8", "8"),
    ("strassen", "32", "12 + 2*sqrt(2)"),
    ("winograd", "56", "7 + 4*sqrt(2) + 3*sqrt(3)"),
    ("tstar", "200/9", "2*sqrt(2) + 16/sqrt(3)"),
])
def test_phi_gamma_closed_forms(name, phi, gam):
    """Section 3.2 closed forms (cubic 8, Strassen 32, T* 200/9, Gamma_min)."""
    D = R.builtin(name)
    assert sp.simplify(R.phi_exact(D) - _sym(phi)) == 0
    assert sp.simplify(R.gamma_exact(D) - _sym(gam)) == 0


def test_phi_gamma_match_table_e2():
    g = golden("table_e2_named.json")["arms"]
    for arm, name in [("dps_acc", "tstar"), ("strassen_classic", "strassen"),
                      ("winograd_form", "winograd")]:
        D = R.builtin_f64(name)
        assert round(R.phi_f64(D), 4) == pytest.approx(g[arm]["phi"], abs=5e-5)
        assert round(R.gamma_f64(D), 4) == pytest.approx(g[arm]["gamma"], abs=5e-5)


def test_certificate_constants():
    g = golden("certificate.json")
    phi_t = R.phi_exact(R.tstar())
    phi_c = R.phi_exact(R.cubic8())
    assert phi_t == _sym(g["phi_min"])
    assert phi_t / phi_c == _sym(g["phi_ratio_min_over_cubic"])
    assert sp.sqrt(phi_t / phi_c) == _sym(g["rms_ratio_min_over_cubic"])
    assert sp.sqrt(R.phi_exact(R.strassen()) / phi_c) == 2
    assert float(R.gamma_exact(R.tstar())) == pytest.approx(g["gamma_min_decimal"], abs=5e-13)


def _reshape(row):
    return sp.Matrix([[row[0], row[1]], [row[2], row[3]]])


def test_moment_map_vanishes_at_tstar():
    """L_A = R_A = (100/9) I for A in {U*, V*, W*} (eq. A.4-A.6)."""
    val = _sym(golden("certificate.json")["moment_map_L_equals_R"])
    for M in R.tstar():
        a = R.row_sq_norms(M)
        L = sp.zeros(2, 2); Rm = sp.zeros(2, 2)
        for r in range(7):
            Ar = _reshape(list(M.row(r)))
            L += a[r] ** 2 * Ar * Ar.T
            Rm += a[r] ** 2 * Ar.T * Ar
        assert sp.simplify(L - val * sp.eye(2)) == sp.zeros(2, 2)
        assert sp.simplify(Rm - val * sp.eye(2)) == sp.zeros(2, 2)


def test_moment_map_control_rejects_perturbation():
    """Negative control: the identity fails away from T* (a tilted copy)."""
    T = sp.Matrix([[1, sp.Rational(1, 5)], [0, 1]])
    U, _, _ = R.act_exact(R.tstar(), (T, sp.eye(2), sp.eye(2)))
    a = R.row_sq_norms(U)
    L = sp.zeros(2, 2)
    for r in range(7):
        Ar = _reshape(list(U.row(r)))
        L += a[r] ** 2 * Ar * Ar.T
    assert sp.simplify(L - _sym("100/9") * sp.eye(2)) != sp.zeros(2, 2)


def test_gamma_stationarity():
    """sum_r sqrt(a_r) A_r A_r^T = sum_r sqrt(a_r) A_r^T A_r = (sqrt2 + 8/sqrt3) I
    (eq. C.2)."""
    val = _sym(golden("certificate.json")["gamma_stationarity"])
    for M in R.tstar():
        a = R.row_sq_norms(M)
        L = sp.zeros(2, 2); Rm = sp.zeros(2, 2)
        for r in range(7):
            Ar = _reshape(list(M.row(r)))
            L += sp.sqrt(a[r]) * Ar * Ar.T
            Rm += sp.sqrt(a[r]) * Ar.T * Ar
        assert sp.simplify(L - val * sp.eye(2)) == sp.zeros(2, 2)
        assert sp.simplify(Rm - val * sp.eye(2)) == sp.zeros(2, 2)


def _phi_at(t, D):
    """Phi(T* . (e^{H_X}, e^{H_Y}, e^{H_Z})) in 60-digit arithmetic;
    H(p, q) = 1/2 [[p, q], [q, -p]], t = (x1, y1, z1, x2, y2, z2) (eq. A.8)."""
    def expm(p, q):
        return mp.expm(mp.matrix([[p / 2, q / 2], [q / 2, -p / 2]]))
    X = expm(t[0], t[3]); Y = expm(t[1], t[4]); Z = expm(t[2], t[5])

    def kron(A, B):
        K = mp.matrix(4, 4)
        for i, j, ip, jp in itertools.product(range(2), repeat=4):
            K[2 * i + j, 2 * ip + jp] = A[i, ip] * B[j, jp]
        return K
    Ks = [kron(X, (Y ** -1).T), kron(Y, (Z ** -1).T), kron(Z, (X ** -1).T)]
    tot = mp.mpf(0)
    for r in range(7):
        prod = mp.mpf(1)
        for M, K in zip(D, Ks):
            row = mp.matrix([[M[r][c] for c in range(4)]])
            v = row * K
            prod *= sum(v[0, c] ** 2 for c in range(4))
        tot += prod
    return tot


def test_second_order_form_at_tstar():
    """Hessian of Phi_t at t = 0 equals 2 (8/9) diag(Q, Q); eigenvalues 128/9
    (twice) and 440/9 (four times) (eq. A.8)."""
    g = golden("certificate.json")
    mp.mp.dps = 60
    D = [[[mp.mpf(sp.N(M[r, c], 70)) for c in range(4)] for r in range(7)]
         for M in R.tstar()]
    h = mp.mpf("1e-12")
    H = mp.matrix(6, 6)
    f0 = _phi_at([0] * 6, D)
    assert abs(f0 - mp.mpf(200) / 9) < mp.mpf("1e-50")
    for i in range(6):
        for j in range(6):
            def f(a, b):
                t = [mp.mpf(0)] * 6
                t[i] += a * h; t[j] += b * h
                return _phi_at(t, D)
            H[i, j] = (f(1, 1) - f(1, -1) - f(-1, 1) + f(-1, -1)) / (4 * h * h)
    Q = sp.Matrix([[_sym(x) for x in row] for row in g["Q"]])
    scale = 2 * _sym(g["second_order_scale"])
    want = sp.zeros(6, 6)
    want[:3, :3] = scale * Q
    want[3:, 3:] = scale * Q
    for i in range(6):
        for j in range(6):
            assert abs(H[i, j] - mp.mpf(sp.N(want[i, j], 40))) < mp.mpf("1e-15")
    ev = sorted(float(x) for x in mp.eig(H)[0])
    assert ev == pytest.approx([128 / 9] * 2 + [440 / 9] * 4, rel=1e-12)
    qev = Q.eigenvals()
    assert {str(k): v for k, v in qev.items()} == g["Q_eigenvalues"]


# --------------------------------------------------------------------------
# Orbit, gauge and Kronecker structure in binary64
# --------------------------------------------------------------------------

def _rand_g(rng):
    out = []
    for _ in range(3):
        while True:
            g = np.eye(2) + 0.45 * rng.standard_normal((2, 2))
            if abs(np.linalg.det(g)) >= 1e-3:
                out.append(g); break
    return out


def test_orbit_floor_and_exactness():
    """Phi(D . g) >= 200/9 on the orbit of Strassen (Theorem 1), and the action
    preserves exactness (Section 2.1)."""
    rng = np.random.default_rng(1)
    S = R.builtin_f64("strassen")
    for _ in range(300):
        Dg = R.act_f64(S, _rand_g(rng))
        assert R.phi_f64(Dg) >= 200 / 9 - 1e-12
        assert R.brent_residual_f64(Dg) < 1e-9


def test_right_action_composes():
    """D . (g h) = (D . g) . h (Section 2.1)."""
    rng = np.random.default_rng(2)
    S = R.builtin_f64("tstar")
    g, h = _rand_g(rng), _rand_g(rng)
    gh = [a @ b for a, b in zip(g, h)]
    A = R.act_f64(S, gh)
    B = R.act_f64(R.act_f64(S, g), h)
    for a, b in zip(A, B):
        assert np.max(np.abs(a - b)) < 1e-11


def test_act_f64_agrees_with_exact_action():
    X = sp.Matrix([[2, 1], [1, 1]]); Y = sp.Matrix([[1, -1], [1, 2]])
    Z = sp.Matrix([[3, 0], [1, 1]])
    ex = R.act_exact(R.strassen(), (X, Y, Z))
    nm = R.act_f64(R.builtin_f64("strassen"),
                   [np.array(M.tolist(), dtype=float) for M in (X, Y, Z)])
    for a, b in zip(ex, nm):
        assert np.max(np.abs(R.to_f64(a) - b)) < 1e-14


def test_gauge_invariance_of_phi():
    """O(2)^3 sandwich, term permutation and product-one rescaling leave Phi
    unchanged (Section 2.1; Appendix B, DG2-DG3: drift about 1e-15)."""
    rng = np.random.default_rng(3)
    D = R.builtin_f64("tstar")
    base = R.phi_f64(D)
    for _ in range(20):
        Qs = []
        for _ in range(3):
            q, _ = np.linalg.qr(rng.standard_normal((2, 2)))
            Qs.append(q)
        assert abs(R.phi_f64(R.act_f64(D, Qs)) / base - 1) < 1e-14
        perm = rng.permutation(7)
        assert abs(R.phi_f64(tuple(M[perm] for M in D)) / base - 1) < 1e-15
        al = np.exp(rng.standard_normal(7)); be = np.exp(rng.standard_normal(7))
        ga = 1 / (al * be)
        Dr = (D[0] * al[:, None], D[1] * be[:, None], D[2] * ga[:, None])
        assert abs(R.phi_f64(Dr) / base - 1) < 1e-14


def test_general_sandwich_moves_phi():
    """A non-orthogonal sandwich is not a gauge: it changes Phi."""
    D = R.builtin_f64("tstar")
    g = [np.array([[1.0, 0.3], [0.0, 1.0]]), np.eye(2), np.eye(2)]
    assert R.phi_f64(R.act_f64(D, g)) > 200 / 9 + 1e-3


def test_rebalance():
    """The canonical gauge equalizes |U_r| and |V_r|, keeps W and Phi; T* is
    already balanced (eq. A.3), so it is a fixed point."""
    D = R.builtin_f64("winograd")
    B = R.rebalance_f64(D)
    nu = np.linalg.norm(B[0], axis=1); nv = np.linalg.norm(B[1], axis=1)
    assert np.allclose(nu, nv, rtol=1e-15)
    assert np.array_equal(B[2], D[2])
    assert R.phi_f64(B) == pytest.approx(56.0, rel=1e-15)
    T = R.builtin_f64("tstar")
    for a, b in zip(R.rebalance_f64(T), T):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("name,depth", [("cubic8", 2), ("strassen", 2), ("winograd", 2),
                                        ("strassen", 3), ("cubic8", 3)])
def test_flattening_is_exact_for_integer_realizations(name, depth):
    """The flattened depth-l realization satisfies the <2^l,2^l,2^l> Brent
    equations exactly (integer coefficients: binary64 is exact)."""
    F = R.flatten_f64(R.builtin_f64(name), depth)
    assert R.brent_residual_f64(F, depth) == 0.0


def test_flattening_tstar_depth2():
    """Phi(T* (x) T*) = 40000/81 (Section 3.2, Kronecker multiplicativity)."""
    g = golden("certificate.json")
    F = R.flatten_f64(R.builtin_f64("tstar"), 2)
    assert R.brent_residual_f64(F, 2) < 1e-14
    assert R.phi_f64(F) == pytest.approx(float(_sym(g["phi_kronecker_square_tstar"])), rel=1e-14)
    F3 = R.flatten_f64(R.builtin_f64("tstar"), 3)
    assert R.phi_f64(F3) == pytest.approx((200 / 9) ** 3, rel=1e-13)


def test_flattening_index_convention_is_kronecker():
    """Level 1 is the most significant digit of both the term and the block
    index: the depth-2 table is the Kronecker product of row vectors arranged
    over the 4x4 grid (checked element by element against a permuted kron)."""
    U = R.builtin_f64("strassen")[0]
    F = R.flatten_f64((U, U, U), 2)[0]
    for r1, r2 in itertools.product(range(7), repeat=2):
        A1 = U[r1].reshape(2, 2); A2 = U[r2].reshape(2, 2)
        grid = np.kron(A1, A2)               # block (i1,j1) scaled copy of A2
        assert np.array_equal(F[7 * r1 + r2], grid.reshape(-1))


def test_tables_f32_single_rounding():
    """The fp32 table is the one-time rounding of the binary64 flattening."""
    T = R.builtin_f64("tstar")
    F64 = R.flatten_f64(T, 2)
    F32 = R.tables_f32(T, 2)
    for a, b in zip(F64, F32):
        assert b.dtype == np.float32
        assert np.array_equal(a.astype(np.float32), b)
    xi = F32[0][1, 4]                    # U*[0,0] * U*[1,2] = 1 * xi (P=1, Q=0)
    assert xi == np.float32(1 / np.sqrt(3.0))
