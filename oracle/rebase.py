"""Re-basing (oracle; test infrastructure only): minimization of Phi over a
realization's change-of-basis orbit.

Protocol (Appendix E.2, the re-basing paragraph): start from the realization
itself and from perturbed starts g = (X, Y, Z), each I + 0.45 N(0,1) with
|det| >= 1e-3 (drawn by ``fmm_inputs.rebasing_starts``); drive every start
by limited-memory BFGS with a strong-Wolfe line search in binary64; keep the
least finite terminal Phi whose realization passes the exactness check.
Here the minimizer is scipy's L-BFGS-B without bounds (its line search is
the More-Thuente search, which enforces the strong Wolfe conditions).

Objective: Phi(D . g) = sum_r a_r b_r c_r with a_r = |u_r K_U|^2,
b_r = |v_r K_V|^2, c_r = |w_r K_W|^2 (Section 2.1), K_U = X (x) Y^-T,
K_V = Y (x) Z^-T, K_W = Z (x) X^-T (the right action of eq. A.1, as
``realizations.act_f64`` applies it).  Gradient, by the chain rule:
  dPhi/dK_U = sum_r b_r c_r 2 u_r^T (u_r K_U)          (4 x 4), likewise K_V, K_W;
  for K = P (x) N, K[2i+j, 2i'+j'] = P[i,i'] N[j,j']:
    dPhi/dP[i,i'] = sum_{j,j'} dPhi/dK[2i+j, 2i'+j'] N[j,j'],
    dPhi/dN[j,j'] = sum_{i,i'} dPhi/dK[2i+j, 2i'+j'] P[i,i'];
  for N = Q^-T, dN = -N dQ^T N, so dPhi/dQ = -N (dPhi/dN)^T N.
Each factor X, Y, Z enters one Kronecker matrix as P and another as Q.

Parity pins (tests/test_oracle_rebase.py): the gradient against central
differences; Strassen 1969, the Winograd variant and random orbit points of
T* re-base to Phi = 200/9 with Gamma = 2 sqrt 2 + 16 / sqrt 3 (Theorem 1 and
the Gamma optimum of Section 3.1); the cubic algorithm and T* itself are
stationary (Phi 8 and 200/9); the terminal realizations satisfy the Brent
equations.
"""
from __future__ import annotations

import numpy as np
from scipy.optimize import minimize

from . import realizations as R


def _split(g):
    g = np.asarray(g, dtype=np.float64).reshape(3, 2, 2)
    return g[0], g[1], g[2]


def _kron_parts(P, Q):
    """K = P (x) Q^-T and N = Q^-T."""
    N = np.linalg.inv(Q).T
    K = np.einsum("ik,jl->ijkl", P, N).reshape(4, 4)
    return K, N


def phi_and_grad(D, g):
    """Phi(D . g) and its gradient over the 12 entries of g (X, Y, Z row-major)."""
    U, V, W = (np.asarray(M, dtype=np.float64) for M in D)
    X, Y, Z = _split(g)
    KU, NY = _kron_parts(X, Y)
    KV, NZ = _kron_parts(Y, Z)
    KW, NX = _kron_parts(Z, X)
    uK, vK, wK = U @ KU, V @ KV, W @ KW
    a = np.sum(uK * uK, axis=1)
    b = np.sum(vK * vK, axis=1)
    c = np.sum(wK * wK, axis=1)
    phi = float(np.sum(a * b * c))
    # dPhi/dK for each Kronecker matrix
    HU = 2.0 * np.einsum("r,ra,rc->ac", b * c, U, uK)
    HV = 2.0 * np.einsum("r,ra,rc->ac", a * c, V, vK)
    HW = 2.0 * np.einsum("r,ra,rc->ac", a * b, W, wK)

    def parts(H, P, N):
        H4 = H.reshape(2, 2, 2, 2)                       # [i, j, i', j']
        dP = np.einsum("ijkl,jl->ik", H4, N)
        dN = np.einsum("ijkl,ik->jl", H4, P)
        return dP, dN

    dX1, dNY = parts(HU, X, NY)      # X as P in K_U, Y through N_Y
    dY1, dNZ = parts(HV, Y, NZ)
    dZ1, dNX = parts(HW, Z, NX)
    dY2 = -NY @ dNY.T @ NY
    dZ2 = -NZ @ dNZ.T @ NZ
    dX2 = -NX @ dNX.T @ NX
    grad = np.concatenate([(dX1 + dX2).ravel(), (dY1 + dY2).ravel(), (dZ1 + dZ2).ravel()])
    return phi, grad


def _objective(D):
    def f(x):
        X, Y, Z = _split(x)
        for M in (X, Y, Z):
            if abs(M[0, 0] * M[1, 1] - M[0, 1] * M[1, 0]) < 1e-300:
                return np.inf, np.zeros(12)
        return phi_and_grad(D, x)
    return f


IDENTITY = np.array([1, 0, 0, 1] * 3, dtype=np.float64)


def rebase(D, starts=None, max_iter: int = 1000, gtol: float = 1e-10, tol: float = 1e-9):
    """(D . g of least Phi, that Phi, terminal Phi per start) over the identity
    start and ``starts`` (an (n, 12) array); NaN marks a start whose terminal
    realization was not exact within ``tol`` or not finite."""
    xs = [IDENTITY] + ([] if starts is None else list(np.asarray(starts, dtype=np.float64)))
    best, best_phi = None, np.inf
    terminal = []
    f = _objective(D)
    for x0 in xs:
        res = minimize(f, np.array(x0), jac=True, method="L-BFGS-B",
                       options={"maxiter": max_iter, "gtol": gtol, "ftol": 1e-16, "maxcor": 10})
        X, Y, Z = _split(res.x)
        t = np.nan
        try:
            Dg = R.act_f64(D, (X, Y, Z))
            phi = R.phi_f64(Dg)
            if np.isfinite(phi) and R.brent_residual_f64(Dg) <= tol:
                t = phi
                if phi < best_phi:
                    best, best_phi = Dg, phi
        except (np.linalg.LinAlgError, ZeroDivisionError, ValueError):
            pass
        terminal.append(t)
    return best, best_phi, np.array(terminal)
