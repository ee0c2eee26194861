"""Coefficient algebra of <2,2,2;R> realizations (oracle; test infrastructure only).

Conventions (Appendix A, the paragraph introducing eq. A.1):

* rv(A) = (a11, a12, a21, a22): an A-block coefficient vector U_r has index
  b = 2*i + j for block (i, j); a B-block vector V_r has index 2*j + k.
* The third factor is cyclic: w_r = rv(W_r^T), so output block (i, k)
  receives w[r, 2*k + i] * P_r.
* The bilinear algorithm of Section 2.1 is c = sum_r <U_r,a><V_r,b> W_r.

A realization here is a triple (U, V, w) of R x 4 arrays (sympy matrices for
exact work, numpy float64 for numeric work).

Parity pins: the tests check this module against the Brent equations in
exact arithmetic, the paper's printed T* coordinates and K_rho matrix
(Appendix A, eq. A.2 and the K_rho display), Phi/Gamma of Section 3.2 and
Table E.2, the moment-map identity (eq. A.4-A.6), the second-order form
(eq. A.8) and the Gamma stationarity identity (eq. C.2).
"""
from __future__ import annotations

import itertools
import math

import numpy as np
import sympy as sp

# ---------------------------------------------------------------------------
# The named realizations, exact
# ---------------------------------------------------------------------------


def cubic8():
    """The cubic <2,2,2;8> algorithm: one term per (i, j, k) in lexicographic
    order, u = e_{2i+j}, v = e_{2j+k}, w = e_{2k+i} (Section 3.2: Phi = 8)."""
    U, V, W = [], [], []
    for i, j, k in itertools.product(range(2), repeat=3):
        u = [0] * 4; u[2 * i + j] = 1
        v = [0] * 4; v[2 * j + k] = 1
        w = [0] * 4; w[2 * k + i] = 1
        U.append(u); V.append(v); W.append(w)
    return sp.Matrix(U), sp.Matrix(V), sp.Matrix(W)


def strassen():
    """Strassen's 1969 products M1..M7 in their classical order.

    M1=(A11+A22)(B11+B22), M2=(A21+A22)B11, M3=A11(B12-B22), M4=A22(B21-B11),
    M5=(A11+A12)B22, M6=(A21-A11)(B11+B12), M7=(A12-A22)(B21+B22);
    C11=M1+M4-M5+M7, C12=M3+M5, C21=M2+M4, C22=M1-M2+M3+M6.

    The paper cites this decomposition without printing it (Section 3.1).
    This order and sign convention is the one for which U*K_rho, V*K_rho and
    w*K_rho reproduce the printed T* coordinates exactly (Appendix A), which
    the tests check; Phi = 32 and Gamma = 12 + 2*sqrt(2) (Section 3.2,
    Table E.2 row strassen_classic).
    """
    U = [[1, 0, 0, 1], [0, 0, 1, 1], [1, 0, 0, 0], [0, 0, 0, 1],
         [1, 1, 0, 0], [-1, 0, 1, 0], [0, 1, 0, -1]]
    V = [[1, 0, 0, 1], [1, 0, 0, 0], [0, 1, 0, -1], [-1, 0, 1, 0],
         [0, 0, 0, 1], [1, 1, 0, 0], [0, 0, 1, 1]]
    # columns of w: (C11, C21, C12, C22) = index 2k+i
    W = [[1, 0, 0, 1], [0, 1, 0, -1], [0, 0, 1, 1], [1, 1, 0, 0],
         [-1, 0, 1, 0], [0, 0, 0, 1], [1, 0, 0, 0]]
    return sp.Matrix(U), sp.Matrix(V), sp.Matrix(W)


def winograd():
    """The Strassen-Winograd variant in its raw (unrebalanced) gauge.

    M1=A11 B11, M2=A12 B21, M3=(A11+A12-A21-A22) B22,
    M4=A22 (B11-B12-B21+B22), M5=(A21+A22)(B12-B11),
    M6=(A21+A22-A11)(B11-B12+B22), M7=(A11-A21)(B22-B12);
    C11=M1+M2, C12=M1+M3+M5+M6, C21=M1-M4+M6+M7, C22=M1+M5+M6+M7.

    The paper names this arm (winograd_form) without printing it; its row of
    Table E.2 fixes Phi = 56 and Gamma = 17.8530 = 7 + 4 sqrt2 + 3 sqrt3,
    which the tests check.  Appendix E.3 notes the panel used the canonically
    rebalanced representative; this is the raw form.
    """
    U = [[1, 0, 0, 0], [0, 1, 0, 0], [1, 1, -1, -1], [0, 0, 0, 1],
         [0, 0, 1, 1], [-1, 0, 1, 1], [1, 0, -1, 0]]
    V = [[1, 0, 0, 0], [0, 0, 1, 0], [0, 0, 0, 1], [1, -1, -1, 1],
         [-1, 1, 0, 0], [1, -1, 0, 1], [0, -1, 0, 1]]
    #      C11 C21 C12 C22
    W = [[1, 1, 1, 1], [1, 0, 0, 0], [0, 0, 1, 0], [0, -1, 0, 0],
         [0, 0, 1, 1], [0, 1, 1, 1], [0, 1, 0, 1]]
    return sp.Matrix(U), sp.Matrix(V), sp.Matrix(W)


XI = 1 / sp.sqrt(3)
ETA = sp.sqrt(3) / 2
ZETA = 1 / (2 * sp.sqrt(3))
PI_V = (1, 3, 7, 6, 4, 5, 2)   # Appendix A, after eq. A.2 (1-based)
PI_W = (1, 7, 2, 5, 6, 4, 3)


def tstar():
    """The Phi-optimal realization T* from its printed coordinates (eq. A.2):
    U* as displayed, V*_r = U*_{pi_V(r)}, w*_r = U*_{pi_W(r)}."""
    h = sp.Rational(1, 2)
    Us = sp.Matrix([
        [1, 0, 0, 1],
        [0, 0, XI, 1],
        [1, 0, XI, 0],
        [0, 0, -XI, 1],
        [h, ETA, ZETA, h],
        [-1, 0, XI, 0],
        [-h, ETA, ZETA, -h],
    ])
    Vs = sp.Matrix([list(Us.row(p - 1)) for p in PI_V])
    Ws = sp.Matrix([list(Us.row(p - 1)) for p in PI_W])
    return Us, Vs, Ws


BUILTINS = {"cubic8": cubic8, "strassen": strassen, "winograd": winograd,
            "tstar": tstar}


def builtin(name: str):
    return BUILTINS[name]()


# ---------------------------------------------------------------------------
# Exact change of basis (eq. A.1), T_rho and K_rho (Appendix A)
# ---------------------------------------------------------------------------

RHO = (sp.Rational(4, 3)) ** sp.Rational(1, 4)


def t_rho():
    """T_rho = [[rho^-1, rho/2], [0, rho]], rho = (4/3)^(1/4) (Theorem 1)."""
    return sp.Matrix([[1 / RHO, RHO / 2], [0, RHO]])


def kron2(X, M):
    """Kronecker product of two 2x2 matrices: entry ((2i+j),(2i'+j')) is
    X[i,i'] * M[j,j'].  Works for sympy matrices."""
    out = sp.zeros(4, 4)
    for i, j, ip, jp in itertools.product(range(2), repeat=4):
        out[2 * i + j, 2 * ip + jp] = X[i, ip] * M[j, jp]
    return out


def act_exact(D, g):
    """D . g for g = (X, Y, Z) by eq. A.1, exactly:
    u -> u (X kron Y^-T), v -> v (Y kron Z^-T), w -> w (Z kron X^-T)."""
    U, V, W = D
    X, Y, Z = [sp.Matrix(m) for m in g]
    KU = kron2(X, Y.inv().T)
    KV = kron2(Y, Z.inv().T)
    KW = kron2(Z, X.inv().T)
    return (sp.simplify(U * KU), sp.simplify(V * KV), sp.simplify(W * KW))


# ---------------------------------------------------------------------------
# Exact functionals
# ---------------------------------------------------------------------------


def row_sq_norms(M):
    return [sp.nsimplify(sp.expand(sum(M[r, c] ** 2 for c in range(M.cols))))
            for r in range(M.rows)]


def phi_exact(D):
    """Phi(D) = sum_r |U_r|^2 |V_r|^2 |W_r|^2 (Section 2.1)."""
    a, b, c = (row_sq_norms(M) for M in D)
    return sp.nsimplify(sp.expand(sum(x * y * z for x, y, z in zip(a, b, c))))


def gamma_exact(D):
    """Gamma(D) = sum_r |U_r| |V_r| |W_r| (Section 2.1, Phi_1)."""
    a, b, c = (row_sq_norms(M) for M in D)
    return sp.radsimp(sum(sp.sqrt(x * y * z) for x, y, z in zip(a, b, c)))


def matmul_tensor(n: int):
    """The <n,n,n> tensor in the cyclic convention: entry
    [(I n + J), (J' n + K), (K' n + I')] = d(J,J') d(K,K') d(I,I')."""
    T = np.zeros((n * n, n * n, n * n), dtype=np.int64)
    for I, J, K in itertools.product(range(n), repeat=3):
        T[I * n + J, J * n + K, K * n + I] = 1
    return T


def brent_exact(D) -> bool:
    """True iff sum_r U_r (x) V_r (x) w_r equals the <2,2,2> tensor exactly."""
    U, V, W = D
    target = matmul_tensor(2)
    for a, b, c in itertools.product(range(4), repeat=3):
        s = sum(U[r, a] * V[r, b] * W[r, c] for r in range(U.rows))
        if sp.simplify(s - int(target[a, b, c])) != 0:
            return False
    return True


# ---------------------------------------------------------------------------
# Binary64 versions (the numbers the fp32 tables are rounded from)
# ---------------------------------------------------------------------------


def to_f64(M) -> np.ndarray:
    """Round every exact entry to the nearest binary64 value."""
    return np.array([[float(sp.N(M[r, c], 40)) for c in range(M.cols)]
                     for r in range(M.rows)], dtype=np.float64)


def builtin_f64(name: str):
    return tuple(to_f64(M) for M in builtin(name))


def inverse_f64(G) -> np.ndarray:
    """2x2 inverse by the adjugate, in this order of binary64 operations:
    det = a*d - b*c; inv = [[d/det, -b/det], [-c/det, a/det]]."""
    a, b, c, d = float(G[0][0]), float(G[0][1]), float(G[1][0]), float(G[1][1])
    det = a * d - b * c
    return [[d / det, (-b) / det], [(-c) / det, a / det]]


def kron_f64(X, M) -> list:
    """4x4 Kronecker product; entry ((2i+j),(2i'+j')) = X[i][i'] * M[j][j']."""
    K = [[0.0] * 4 for _ in range(4)]
    for i, j, ip, jp in itertools.product(range(2), repeat=4):
        K[2 * i + j][2 * ip + jp] = float(X[i][ip]) * float(M[j][jp])
    return K


def _transpose(M):
    return [[M[0][0], M[1][0]], [M[0][1], M[1][1]]]


def _rowtimes(u, K) -> list:
    """u K for a 4-vector and a 4x4 matrix; each output entry summed in
    ascending input index, one rounding per multiply and per add."""
    out = []
    for c in range(4):
        s = float(u[0]) * K[0][c]
        for a in range(1, 4):
            s = s + float(u[a]) * K[a][c]
        out.append(s)
    return out


def act_f64(D, g):
    """D . g by eq. A.1 in binary64, with the operation order fixed above:
    Y^-1 by the adjugate, M = (Y^-1)^T, K = X kron M, u' = u K summed in
    ascending index.  Raises ValueError for |det| < 1e-12 (singular)."""
    U, V, W = (np.asarray(M, dtype=np.float64) for M in D)
    X, Y, Z = ([[float(m[0][0]), float(m[0][1])], [float(m[1][0]), float(m[1][1])]]
               for m in g)
    for G in (X, Y, Z):
        det = G[0][0] * G[1][1] - G[0][1] * G[1][0]
        if not (abs(det) >= 1e-12):
            raise ValueError("singular basis change")
    KU = kron_f64(X, _transpose(inverse_f64(Y)))
    KV = kron_f64(Y, _transpose(inverse_f64(Z)))
    KW = kron_f64(Z, _transpose(inverse_f64(X)))
    U2 = np.array([_rowtimes(U[r], KU) for r in range(U.shape[0])])
    V2 = np.array([_rowtimes(V[r], KV) for r in range(V.shape[0])])
    W2 = np.array([_rowtimes(W[r], KW) for r in range(W.shape[0])])
    return U2, V2, W2


def _norm(row) -> float:
    s = 0.0
    for x in row:
        s = s + float(x) * float(x)
    return math.sqrt(s)


def rebalance_f64(D):
    """The canonical rebalanced gauge (Appendix E.2):
    (U_r, V_r, W_r) -> (U_r / s_r, s_r V_r, W_r), s_r = sqrt(|U_r| / |V_r|),
    norms summed in ascending index; rows with a zero norm are left alone."""
    U, V, W = (np.array(M, dtype=np.float64) for M in D)
    for r in range(U.shape[0]):
        nu, nv = _norm(U[r]), _norm(V[r])
        if nu == 0.0 or nv == 0.0:
            continue
        s = math.sqrt(nu / nv)
        U[r] = U[r] / s
        V[r] = V[r] * s
    return U, V, W


def phi_f64(D) -> float:
    U, V, W = (np.asarray(M, dtype=np.float64) for M in D)
    return float(np.sum((U ** 2).sum(1) * (V ** 2).sum(1) * (W ** 2).sum(1)))


def gamma_f64(D) -> float:
    U, V, W = (np.asarray(M, dtype=np.float64) for M in D)
    return float(np.sum(np.sqrt((U ** 2).sum(1) * (V ** 2).sum(1) * (W ** 2).sum(1))))


def brent_residual_f64(D, depth: int = 1) -> float:
    """max |sum_r U (x) V (x) w - <n,n,n>| with n = 2^depth (tables as given)."""
    U, V, W = (np.asarray(M, dtype=np.float64) for M in D)
    T = np.einsum("ra,rb,rc->abc", U, V, W)
    return float(np.max(np.abs(T - matmul_tensor(2 ** depth))))


# ---------------------------------------------------------------------------
# Kronecker flattening (Section 3.2; the kernels flatten, Section 4.3)
# ---------------------------------------------------------------------------


def flatten_f64(D, depth: int):
    """Depth-l Kronecker power as one nonrecursive realization.

    Term (r_1..r_l) becomes r = sum_t r_t R^(l-t) (level 1 most significant).
    A sub-block (I, J) of the 2^l x 2^l grid has I = sum_t i_t 2^(l-t) and
    index I*2^l + J; its coefficient is prod_t U[r_t, 2 i_t + j_t], multiplied
    left to right (t = 1..l) in binary64.  V uses (J, K) and w the cyclic
    (K, I) with index K*2^l + I, in the same way.
    """
    U, V, W = (np.asarray(M, dtype=np.float64) for M in D)
    R = U.shape[0]
    n = 2 ** depth
    T = R ** depth
    out = [np.zeros((T, n * n)), np.zeros((T, n * n)), np.zeros((T, n * n))]
    for r in range(T):
        digits = [(r // R ** (depth - 1 - t)) % R for t in range(depth)]
        for P, Q in itertools.product(range(n), repeat=2):
            pb = [(P >> (depth - 1 - t)) & 1 for t in range(depth)]
            qb = [(Q >> (depth - 1 - t)) & 1 for t in range(depth)]
            for dst, src in zip(out, (U, V, W)):
                c = float(src[digits[0], 2 * pb[0] + qb[0]])
                for t in range(1, depth):
                    c = c * float(src[digits[t], 2 * pb[t] + qb[t]])
                dst[r, P * n + Q] = c
    return tuple(out)


def tables_f32(D, depth: int):
    """The fp32 coefficient tables the quantized evaluation uses: the binary64
    flattening rounded once, to nearest, to binary32."""
    return tuple(np.asarray(M, dtype=np.float64).astype(np.float32)
                 for M in flatten_f64(D, depth))
