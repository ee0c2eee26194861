"""Realizations of shapes <m,k,n;R> other than <2,2,2>, built as inputs.

The paper tabulates errors for decompositions of other shapes (Table E.1)
whose coefficients it does not print.  The realizations here are exact by
construction, from two pieces: the cubic algorithm of any shape, and direct
sums along one dimension of two realizations (Section 2.1's tensor view:
C = A [B1 B2] = [A B1, A B2] along n, C = [A1; A2] B along m,
C = A1 B1 + A2 B2 along k).  Both place given coefficients at new indices
and do no arithmetic; exactness is checked by the oracle (the Brent
equations in rational arithmetic), not assumed.

Conventions (Section 2.1, with Appendix A's cyclic third factor): U_r has
m k entries, A block (i, j) at i k + j; V_r has k n, B block (j, l) at
j n + l; W_r has n m, C block (i, l) at l m + i.  A realization is
((m, k, n), U, V, W) with U, V, W float64 arrays of R rows.

``build(name, base)`` returns the named realization; ``base(which)`` must
return the (U, V, W) rows of a <2,2,2> realization ("strassen" or "tstar"),
so each side (the oracle, the library) supplies its own copy of those.
"""
from __future__ import annotations

import numpy as np


def cubic(m: int, k: int, n: int):
    """The cubic <m,k,n; mkn> algorithm: term (i, j, l), in lexicographic
    order, multiplies A block (i, j) by B block (j, l) into C block (i, l)."""
    R = m * k * n
    U = np.zeros((R, m * k)); V = np.zeros((R, k * n)); W = np.zeros((R, n * m))
    r = 0
    for i in range(m):
        for j in range(k):
            for l in range(n):
                U[r, i * k + j] = 1.0
                V[r, j * n + l] = 1.0
                W[r, l * m + i] = 1.0
                r += 1
    return (m, k, n), U, V, W


def from_222(UVW):
    """A <2,2,2> realization's rows (U, V, W; 4 columns each) in this form."""
    U, V, W = (np.array(x, dtype=np.float64).reshape(-1, 4) for x in UVW)
    return (2, 2, 2), U, V, W


def direct_sum(D1, D2, axis: str):
    """<m,k,n1+n2> from <m,k,n1> and <m,k,n2> (axis 'n'), <m1+m2,k,n> (axis
    'm') or <m,k1+k2,n> (axis 'k'): the terms of D1 followed by those of D2,
    each placed at its block's index in the larger grids."""
    (m1, k1, n1), _, _, _ = D1
    (m2, k2, n2), _, _, _ = D2
    if axis == "n":
        if (m1, k1) != (m2, k2):
            raise ValueError("direct sum along n needs equal m, k")
        shape, offs = (m1, k1, n1 + n2), ((0, 0, 0), (0, 0, n1))
    elif axis == "m":
        if (k1, n1) != (k2, n2):
            raise ValueError("direct sum along m needs equal k, n")
        shape, offs = (m1 + m2, k1, n1), ((0, 0, 0), (m1, 0, 0))
    elif axis == "k":
        if (m1, n1) != (m2, n2):
            raise ValueError("direct sum along k needs equal m, n")
        shape, offs = (m1, k1 + k2, n1), ((0, 0, 0), (0, k1, 0))
    else:
        raise ValueError(axis)
    m, k, n = shape
    Us, Vs, Ws = [], [], []
    for ((mm, kk, nn), U, V, W), (om, ok, on) in zip((D1, D2), offs):
        R = U.shape[0]
        nU = np.zeros((R, m * k)); nV = np.zeros((R, k * n)); nW = np.zeros((R, n * m))
        for i in range(mm):
            for j in range(kk):
                nU[:, (i + om) * k + (j + ok)] = U[:, i * kk + j]
        for j in range(kk):
            for l in range(nn):
                nV[:, (j + ok) * n + (l + on)] = V[:, j * nn + l]
        for i in range(mm):
            for l in range(nn):
                nW[:, (l + on) * m + (i + om)] = W[:, l * mm + i]
        Us.append(nU); Vs.append(nV); Ws.append(nW)
    return shape, np.vstack(Us), np.vstack(Vs), np.vstack(Ws)


# name -> (shape, rank); built by build()
CATALOG = {
    "223_11": ((2, 2, 3), 11),      # Strassen (+)n cubic <2,2,1>
    "322_11": ((3, 2, 2), 11),      # Strassen (+)m cubic <1,2,2>
    "232_11": ((2, 3, 2), 11),      # Strassen (+)k cubic <2,1,2>
    "223_tstar": ((2, 2, 3), 11),   # T* (+)n cubic <2,2,1>
    "333_26": ((3, 3, 3), 26),      # 3 = 2 + 1 along every dimension, Strassen on the 2 x 2 x 2 part
    "333_27": ((3, 3, 3), 27),      # cubic
    "525_46": ((5, 2, 5), 46),      # four Strassens on the 4 x 2 x 4 part, cubic on the rest
    "454_80": ((4, 5, 4), 80),      # cubic (A and B grids of 20 blocks)
}


def build(name: str, base):
    """The named realization of CATALOG; base(which) gives a <2,2,2> one."""
    if name == "223_11":
        return direct_sum(from_222(base("strassen")), cubic(2, 2, 1), "n")
    if name == "322_11":
        return direct_sum(from_222(base("strassen")), cubic(1, 2, 2), "m")
    if name == "232_11":
        return direct_sum(from_222(base("strassen")), cubic(2, 1, 2), "k")
    if name == "223_tstar":
        return direct_sum(from_222(base("tstar")), cubic(2, 2, 1), "n")
    if name == "333_26":
        s223 = direct_sum(from_222(base("strassen")), cubic(2, 2, 1), "n")
        s233 = direct_sum(s223, cubic(2, 1, 3), "k")
        return direct_sum(s233, cubic(1, 3, 3), "m")
    if name == "333_27":
        return cubic(3, 3, 3)
    if name == "525_46":
        s = from_222(base("strassen"))
        s225 = direct_sum(direct_sum(s, s, "n"), cubic(2, 2, 1), "n")
        return direct_sum(direct_sum(s225, s225, "m"), cubic(1, 2, 5), "m")
    if name == "454_80":
        return cubic(4, 5, 4)
    raise KeyError(name)
