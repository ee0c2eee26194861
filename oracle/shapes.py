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
whose coefficients are not printed.  The shapes here are built from exact
pieces: the cubic algorithm of any shape, and direct sums along one
dimension (C = A [B1 B2] = [A B1, A B2] along n, and the like along m and
k), e.g. <2,2,3;11> = Strassen (x) cubic <2,2,1;4> along n.

The evaluation follows oracle/fmm.py step by step (fp32 combination in
ascending block index, no fused multiply-add; quantization along the
contracted axis; sub-products and W-combine in binary64 with W rounded to
fp32).
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np

from . import e4m3, fmm


def cubic(m: int, k: int, n: int):
    """The cubic <m,k,n; mkn> algorithm: term (i, j, l) in lexicographic order
    multiplies A block (i, j) by B block (j, l) into C block (i, l)."""
    U, V, W = [], [], []
    for i in range(m):
        for j in range(k):
            for l in range(n):
                u = [0] * (m * k); u[i * k + j] = 1
                v = [0] * (k * n); v[j * n + l] = 1
                w = [0] * (n * m); w[l * m + i] = 1
                U.append(u); V.append(v); W.append(w)
    return (m, k, n), U, V, W


def from_222(D):
    """A <2,2,2> realization (U, V, w lists of rows) in this module's form."""
    U, V, W = D
    return (2, 2, 2), [list(r) for r in U], [list(r) for r in V], [list(r) for r in W]


def direct_sum(D1, D2, axis: str):
    """<m,k,n1+n2> from <m,k,n1> and <m,k,n2> (axis 'n': C = A [B1 B2]),
    <m1+m2,k,n> (axis 'm': C = [A1; A2] B) or <m,k1+k2,n> (axis 'k':
    C = A1 B1 + A2 B2): the terms of D1 followed by those of D2, each
    re-indexed into the larger grids."""
    (m1, k1, n1), U1, V1, W1 = D1
    (m2, k2, n2), U2, V2, W2 = D2
    if axis == "n":
        assert (m1, k1) == (m2, k2)
        m, k, n = m1, k1, n1 + n2
        a_map = lambda part, i, j: (i, j)
        b_map = lambda part, j, l: (j, l + (0 if part == 0 else n1))
        c_map = lambda part, i, l: (i, l + (0 if part == 0 else n1))
    elif axis == "m":
        assert (k1, n1) == (k2, n2)
        m, k, n = m1 + m2, k1, n1
        a_map = lambda part, i, j: (i + (0 if part == 0 else m1), j)
        b_map = lambda part, j, l: (j, l)
        c_map = lambda part, i, l: (i + (0 if part == 0 else m1), l)
    elif axis == "k":
        assert (m1, n1) == (m2, n2)
        m, k, n = m1, k1 + k2, n1
        a_map = lambda part, i, j: (i, j + (0 if part == 0 else k1))
        b_map = lambda part, j, l: (j + (0 if part == 0 else k1), l)
        c_map = lambda part, i, l: (i, l)
    else:
        raise ValueError(axis)
    U, V, W = [], [], []
    for part, ((mm, kk, nn), Us, Vs, Ws) in enumerate((D1, D2)):
        for u, v, w in zip(Us, Vs, Ws):
            nu = [0] * (m * k); nv = [0] * (k * n); nw = [0] * (n * m)
            for i in range(mm):
                for j in range(kk):
                    I, J = a_map(part, i, j)
                    nu[I * k + J] = u[i * kk + j]
            for j in range(kk):
                for l in range(nn):
                    J, L = b_map(part, j, l)
                    nv[J * n + L] = v[j * nn + l]
            for i in range(mm):
                for l in range(nn):
                    I, L = c_map(part, i, l)
                    nw[L * m + I] = w[l * mm + i]
            U.append(nu); V.append(nv); W.append(nw)
    return (m, k, n), U, V, W


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
