"""Realizations of <m,k,n;R> other than <2,2,2> and their fused block-scaled
e4m3 evaluation at one level (oracle; test infrastructure only).

Conventions (Section 2.1; Appendix A's cyclic third factor, generalised):
A (M x K) is split into an m x k grid of sub-blocks, block (i, j) with index
i k + j; B (K x N) into a k x n grid, block (j, l) with index j n + l; C into
an m x n grid, block (i, l).  A realization is R terms (U_r, V_r, W_r) with
U_r of length m k, V_r of length k n and W_r of length n m indexed cyclically
by l m + i, and is exact when the Brent equations hold:

    sum_r U_r[i k + j] V_r[j' n + l] W_r[l' m + i'] = [j = j'] [l = l'] [i = i'].

Then C block (i, l) = sum_r W_r[l m + i] P_r with P_r = (sum_b U_r[b] A_b)
(sum_b V_r[b] B_b).  At <2,2,2> these are the conventions of
oracle/realizations.py (2i + j, 2j + k, 2k + i).

The paper tabulates errors for decompositions of other shapes (Table E.1)
whose coefficients are not printed.  The realizations run here are inputs
(fmm_inputs/shapes.py builds them from the cubic algorithm and direct sums,
e.g. <2,2,3;11> = Strassen (+) cubic <2,2,1;4> along n); this module checks
them (the Brent equations in exact arithmetic) and evaluates them.
A realization is ((m, k, n), U, V, W) with U, V, W arrays of R rows.

The evaluation follows oracle/fmm.py step by step (fp32 combination in
ascending block index, no fused multiply-add; quantization along the
contracted axis; sub-products and W-combine in binary64 with W rounded to
fp32).
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np
import sympy

from . import e4m3, fmm


def brent_exact(D) -> bool:
    """The Brent equations in exact rational arithmetic."""
    (m, k, n), U, V, W = D
    for i in range(m):
        for j in range(k):
            for j2 in range(k):
                for l in range(n):
                    for l2 in range(n):
                        for i2 in range(m):
                            s = sum(Fraction(U[r][i * k + j]) * Fraction(V[r][j2 * n + l]) *
                                    Fraction(W[r][l2 * m + i2]) for r in range(len(U)))
                            want = 1 if (j == j2 and l == l2 and i == i2) else 0
                            if s != want:
                                return False
    return True


def phi(D) -> float:
    """Phi = sum_r |U_r|^2 |V_r|^2 |W_r|^2 (Section 2.1), binary64."""
    _, U, V, W = D
    return float(sum(np.dot(u, u) * np.dot(v, v) * np.dot(w, w) for u, v, w in
                     zip(np.asarray(U, float), np.asarray(V, float), np.asarray(W, float))))


def gamma(D) -> float:
    """Gamma = sum_r |U_r| |V_r| |W_r|."""
    _, U, V, W = D
    return float(sum(np.linalg.norm(u) * np.linalg.norm(v) * np.linalg.norm(w) for u, v, w in
                     zip(np.asarray(U, float), np.asarray(V, float), np.asarray(W, float))))


def tables_f32(D):
    """The fp32 coefficient tables (R x mk, R x kn, R x nm)."""
    _, U, V, W = D
    return tuple(np.asarray(M, dtype=np.float64).astype(np.float32) for M in (U, V, W))


def split_grid(M: np.ndarray, rows: int, cols: int):
    """Sub-blocks of a matrix in a rows x cols grid; block (P, Q) has index
    P cols + Q."""
    r, c = M.shape
    if r % rows or c % cols:
        raise ValueError("matrix dimensions must be divisible by the grid")
    rb, cb = r // rows, c // cols
    return [M[P * rb:(P + 1) * rb, Q * cb:(Q + 1) * cb] for P in range(rows) for Q in range(cols)]


def encode_side(M: np.ndarray, table: np.ndarray, grid, bs: int, rule: int, side: str):
    """Encode and quantize one operand for every term (as fmm.encode_side at
    one level): A blocks in the m x k grid, B blocks in the k x n grid with
    each combination transposed so the contracted axis is last."""
    blocks = [np.asarray(b, dtype=np.float32) for b in split_grid(M, *grid)]
    codes, scales, deqs, xs = [], [], [], []
    for r in range(table.shape[0]):
        x = fmm.combine(blocks, table[r])
        if side == "B":
            x = np.ascontiguousarray(x.T)
        c, st, _, dq = e4m3.quantize_rows(x, bs, rule)
        codes.append(c); scales.append(st); deqs.append(dq); xs.append(x)
    return {"codes": np.stack(codes), "scales": np.stack(scales), "deq": deqs, "x": xs}


def wcombine(P, wtab: np.ndarray, shape, M: int, N: int) -> np.ndarray:
    """C block (i, l) = sum_r w[r, l m + i] P_r, binary64, ascending r."""
    m, _, n = shape
    mb, nb = M // m, N // n
    C = np.zeros((M, N), dtype=np.float64)
    w64 = np.asarray(wtab, dtype=np.float32).astype(np.float64)
    for r, Pr in enumerate(P):
        for i in range(m):
            for l in range(n):
                c = w64[r, l * m + i]
                if c != 0.0:
                    C[i * mb:(i + 1) * mb, l * nb:(l + 1) * nb] += c * Pr
    return C


def fmm_shape(A: np.ndarray, B: np.ndarray, D, bs: int, rule: int):
    """The fused evaluation of realization D at one level: codes, scales,
    dequantized operands and C (binary64)."""
    (m, k, n) = D[0]
    U, V, W = tables_f32(D)
    ea = encode_side(A, U, (m, k), bs, rule, "A")
    eb = encode_side(B, V, (k, n), bs, rule, "B")
    P = fmm.products(ea["deq"], eb["deq"])
    return {"a": ea, "b": eb, "C": wcombine(P, W, (m, k, n), A.shape[0], B.shape[1])}


def exact_product(A: np.ndarray, B: np.ndarray, D) -> np.ndarray:
    """The realization's bilinear map with no quantization, in binary64 (for
    the exactness check on integer matrices)."""
    (m, k, n), U, V, W = D
    Ab = split_grid(np.asarray(A, np.float64), m, k)
    Bb = split_grid(np.asarray(B, np.float64), k, n)
    P = [sum(u[b] * Ab[b] for b in range(m * k)) @ sum(v[b] * Bb[b] for b in range(k * n))
         for u, v in zip(U, V)]
    return wcombine(P, np.asarray(W, np.float64), (m, k, n), A.shape[0], B.shape[1])


# ---- the change-of-basis orbit GL(m) x GL(k) x GL(n) -------------------------
#
# eq. A.1's right action written for any shape: u -> u (X (x) Y^-T),
# v -> v (Y (x) Z^-T), w -> w (Z (x) X^-T) with the Kronecker index order of
# the flattened grids (u index i k + j pairs X's row index i with Y^-T's j).
# Re-basing (Section 3.1; Appendix E.2's protocol) minimizes Phi(D . g) over
# it; here by scipy's L-BFGS-B with the gradient by the chain rule through
# the Kronecker matrices (as oracle/rebase.py does at <2,2,2>).

def split_g(g, shape):
    m, k, n = shape
    g = np.asarray(g, dtype=np.float64)
    return (g[:m * m].reshape(m, m), g[m * m:m * m + k * k].reshape(k, k), g[m * m + k * k:].reshape(n, n))


def kron_parts(P, Q):
    """K = P (x) Q^-T and N = Q^-T (numpy's inverse)."""
    N = np.linalg.inv(Q).T
    return np.kron(P, N), N


def act(D, X, Y, Z):
    """D . (X, Y, Z) in binary64: each row times its Kronecker matrix."""
    shape, U, V, W = D
    KU, _ = kron_parts(np.asarray(X, float), np.asarray(Y, float))
    KV, _ = kron_parts(np.asarray(Y, float), np.asarray(Z, float))
    KW, _ = kron_parts(np.asarray(Z, float), np.asarray(X, float))
    return shape, np.asarray(U, float) @ KU, np.asarray(V, float) @ KV, np.asarray(W, float) @ KW


def act_exact(D, X, Y, Z):
    """D . (X, Y, Z) in rational arithmetic (X, Y, Z of Fractions or ints)."""
    shape, U, V, W = D

    def kron_inv_t(P, Q):
        Ni = sympy.Matrix(Q).inv().T
        return sympy.kronecker_product(sympy.Matrix(P), Ni)

    def rows(M, K):
        return [list(sympy.Matrix([[sympy.Rational(str(Fraction(x))) for x in r]]) * K) for r in np.asarray(M).tolist()]
    X, Y, Z = ([[sympy.Rational(str(Fraction(x))) for x in r] for r in M] for M in (X, Y, Z))
    return (shape, rows(U, kron_inv_t(X, Y)), rows(V, kron_inv_t(Y, Z)), rows(W, kron_inv_t(Z, X)))


def phi_and_grad(D, g):
    """Phi(D . g) and its gradient over the m^2 + k^2 + n^2 entries of g."""
    (m, k, n), U, V, W = D
    U, V, W = (np.asarray(M, dtype=np.float64) for M in (U, V, W))
    X, Y, Z = split_g(g, (m, k, n))
    KU, NY = kron_parts(X, Y)
    KV, NZ = kron_parts(Y, Z)
    KW, NX = kron_parts(Z, X)
    uK, vK, wK = U @ KU, V @ KV, W @ KW
    a, b, c = (np.sum(M * M, axis=1) for M in (uK, vK, wK))
    phi = float(np.sum(a * b * c))
    HU = 2.0 * np.einsum("r,ra,rc->ac", b * c, U, uK)      # dPhi/dK_U
    HV = 2.0 * np.einsum("r,ra,rc->ac", a * c, V, vK)
    HW = 2.0 * np.einsum("r,ra,rc->ac", a * b, W, wK)

    def parts(H, P, N):
        p, q = P.shape[0], N.shape[0]
        H4 = H.reshape(p, q, p, q)                          # [i, j, i', j']
        return np.einsum("ijkl,jl->ik", H4, N), np.einsum("ijkl,ik->jl", H4, P)

    dX1, dNY = parts(HU, X, NY)
    dY1, dNZ = parts(HV, Y, NZ)
    dZ1, dNX = parts(HW, Z, NX)
    dY2 = -NY @ dNY.T @ NY          # N = Q^-T: dN = -N dQ^T N
    dZ2 = -NZ @ dNZ.T @ NZ
    dX2 = -NX @ dNX.T @ NX
    return phi, np.concatenate([(dX1 + dX2).ravel(), (dY1 + dY2).ravel(), (dZ1 + dZ2).ravel()])


def brent_residual(D) -> float:
    """max |sum_r U_r (x) V_r (x) W_r - <m,k,n>| in binary64."""
    (m, k, n), U, V, W = D
    T = np.einsum("ra,rb,rc->abc", np.asarray(U, float), np.asarray(V, float), np.asarray(W, float))
    want = np.zeros_like(T)
    for i in range(m):
        for j in range(k):
            for l in range(n):
                want[i * k + j, j * n + l, l * m + i] = 1.0
    return float(np.abs(T - want).max())


def rebase(D, starts=None, max_iter: int = 1000, gtol: float = 1e-10, tol: float = 1e-9):
    """(D . g of least Phi, that Phi, terminal Phi per start) over the identity
    start and ``starts``; NaN marks a start that ended singular, non-finite or
    not exact within ``tol``."""
    from scipy.optimize import minimize
    (m, k, n) = D[0]
    ident = np.concatenate([np.eye(m).ravel(), np.eye(k).ravel(), np.eye(n).ravel()])
    xs = [ident] + ([] if starts is None else list(np.asarray(starts, dtype=np.float64)))

    def f(x):
        try:
            return phi_and_grad(D, x)
        except np.linalg.LinAlgError:
            return np.inf, np.zeros_like(x)
    best, best_phi, terminal = None, np.inf, []
    for x0 in xs:
        res = minimize(f, np.array(x0), jac=True, method="L-BFGS-B",
                       options={"maxiter": max_iter, "gtol": gtol, "ftol": 1e-16, "maxcor": 10})
        t = np.nan
        try:
            Dg = act(D, *split_g(res.x, (m, k, n)))
            p = phi(Dg)
            if np.isfinite(p) and brent_residual(Dg) <= tol:
                t = p
                if p < best_phi:
                    best, best_phi = Dg, p
        except np.linalg.LinAlgError:
            pass
        terminal.append(t)
    return best, best_phi, np.array(terminal)
