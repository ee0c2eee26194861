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
