"""The second-moment model (oracle; test infrastructure only).

Section 2.2 and Appendix D: under Assumption 1,
E|dC|^2 / E|C|^2 = (s_A^2 + s_B^2 + s_A^2 s_B^2) Phi / (m k n)   (eq. D.8),
and keeping the leading operand-side terms with s_A = s_B = s_q,
E|dC|^2 / E|C|^2 ~ 2 s_q^2 Phi / (m k n)                          (eq. D.9).
For <2,2,2> at depth l, m k n = 8^l and Phi is the flattened Phi.

s_A^2 is the operand-side rounding noise coefficient: the rounding energy
of the encoded combinations relative to their energy (eq. D.1), measured
over every term of the run.
"""
from __future__ import annotations

import numpy as np


def noise_coefficient(x_list, deq_list) -> float:
    """s^2 = sum_r sum (xhat_r - x_r)^2 / sum_r sum x_r^2."""
    num = 0.0
    den = 0.0
    for x, xh in zip(x_list, deq_list):
        x64 = np.asarray(x, np.float64)
        d = np.asarray(xh, np.float64) - x64
        num += float(np.sum(d * d))
        den += float(np.sum(x64 * x64))
    return num / den


def predicted_rel_mse(s_a2: float, s_b2: float, phi: float, depth: int,
                      full: bool = True) -> float:
    mkn = 8.0 ** depth
    if full:
        return (s_a2 + s_b2 + s_a2 * s_b2) * phi / mkn
    s2 = 0.5 * (s_a2 + s_b2)
    return 2.0 * s2 * phi / mkn


def cross_r_residual(ea, eb, w_table) -> float:
    """The share of the error's linear part that the diagonal sum defining
    Phi leaves out (Appendix D, the cross-r covariance measurement):
    (|L|^2 - diag) / |L|^2 from cross_r_sums."""
    L2, diag = cross_r_sums(ea, eb, w_table)
    return (L2 - diag) / L2


def cross_r_sums(ea, eb, w_table):
    """(|L|^2, diag) of the cross-r covariance measurement (Appendix D).

    With X_r, Y_r the fp32 combinations and dX_r, dY_r their rounding
    residuals (encode_side outputs, B side transposed back), the part of the
    sub-product error linear in the residuals is t_r = dX_r Y_r + X_r dY_r,
    and that of output block q is L_q = sum_r w[r, q] t_r.  |L|^2 =
    sum_q |L_q|^2 and diag = sum_{r,q} w[r, q]^2 |t_r|^2 (binary64
    throughout)."""
    w = np.asarray(w_table, dtype=np.float64)
    T, nq = w.shape
    t = []
    for r in range(T):
        X = np.asarray(ea["x"][r], np.float64)
        dX = ea["deq"][r] - X
        Y = np.asarray(eb["x"][r], np.float64).T
        dY = eb["deq"][r].T - Y
        t.append(dX @ Y + X @ dY)
    L2 = 0.0
    diag = 0.0
    for q in range(nq):
        Lq = sum(w[r, q] * t[r] for r in range(T) if w[r, q] != 0.0)
        if not isinstance(Lq, np.ndarray):
            continue
        L2 += float(np.sum(Lq * Lq))
        diag += sum(float(w[r, q] ** 2 * np.sum(t[r] * t[r])) for r in range(T))
    return L2, diag
