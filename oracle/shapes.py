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
