"""Fused block-scaled e4m3 evaluation of a realization (oracle; test
infrastructure only).

This follows the regime of Assumption 1 (Section 2.2) and the emulator of
Appendix E.2: the original operand blocks stay unquantized; for every term
the encoded combinations x_r = <U_r, a> and y_r = <V_r, b> are formed in
fp32, quantized per block along the contracted axis (1 x bs on both sides),
multiplied, and the products are decoded into C by the W coefficients.

Readings (where the paper fixes no detail):

* combine order: the nonzero coefficients of a term are visited in
  ascending sub-block index; acc = fl32(c_1 a_1), then
  acc = fl32(acc + fl32(c_j a_j)) -- a multiply and an add, never a fused
  multiply-add.  A term with no nonzero coefficient combines to +0.
* depth l: the flattened (nonrecursive) realization is evaluated; each
  flattened term is quantized once (Section 4.3 notes the kernels flatten
  the Kronecker construction).
* the sub-products of dequantized operands and the W-combine are formed in
  binary64 (the dequantized values code * scale are exact in binary64), with
  the W coefficients rounded to fp32, summed over terms in ascending order.

Layouts match the GPU workspace so results compare byte for byte:
x codes (T, m', k') and y codes transposed (T, n', k'), both with the
contracted axis last; scales (T, m', k'/bs) and (T, n', k'/bs).
"""
from __future__ import annotations

import numpy as np

from . import e4m3


def split(M: np.ndarray, depth: int):
    """Sub-blocks of a (rows, cols) matrix in a 2^l x 2^l grid; block (P, Q)
    has index P * 2^l + Q."""
    n = 2 ** depth
    r, c = M.shape
    if r % n or c % n:
        raise ValueError("matrix dimensions must be divisible by 2^depth")
    rb, cb = r // n, c // n
    return [M[P * rb:(P + 1) * rb, Q * cb:(Q + 1) * cb]
            for P in range(n) for Q in range(n)]


def combine(blocks, coeffs) -> np.ndarray:
    """fp32 combination sum_b coeffs[b] * blocks[b] in the pinned order."""
    acc = None
    for b, c in enumerate(coeffs):
        c = np.float32(c)
        if c == 0:
            continue
        t = c * blocks[b]                          # fl32(c * a), elementwise
        acc = t if acc is None else (acc + t)      # fl32(acc + t)
    if acc is None:
        acc = np.zeros_like(blocks[0], dtype=np.float32)
    return acc.astype(np.float32, copy=False)


def encode_side(M: np.ndarray, table: np.ndarray, depth: int, bs: int,
                rule: int, side: str, want_deq: bool = True, row_block: int = 1,
                bf16: bool = False):
    """Encode and quantize one operand for every flattened term.

    side 'A': M is A (M x K), blocks (I, J), output rows p, contracted l.
    side 'B': M is B (K x N), blocks (J, K); the combination y (k' x n') is
    transposed (exactly) so its contracted axis is last.
    Deployment granularity (Appendix E, weight-scale granularity): with
    bf16 each combination is first rounded to bfloat16; with row_block > 1
    one scale covers row_block rows x bs positions, its maximum taken over the
    combination (scales stored per row, replicated over each block's rows).
    Returns dict(codes (T, r, k'), scales (T, r, k'/bs) stored form,
    s (float32 scales), deq (float64, if want_deq), x (fp32 combos list if
    want_deq)).
    """
    blocks = [np.asarray(b, dtype=np.float32) for b in split(M, depth)]
    T = table.shape[0]
    codes, scales, s_all, deqs, xs = [], [], [], [], []
    for r in range(T):
        x = combine(blocks, table[r])
        if side == "B":
            x = np.ascontiguousarray(x.T)
        xq = e4m3.bf16_round(x) if bf16 else x       # x itself stays the fp32 combination
        if row_block > 1:
            c, st, s, dq = e4m3.quantize_blocks2d(xq, row_block, bs, rule)
        else:
            c, st, s, dq = e4m3.quantize_rows(xq, bs, rule)
        codes.append(c); scales.append(st); s_all.append(s)
        if want_deq:
            deqs.append(dq); xs.append(x)
    out = {"codes": np.stack(codes), "scales": np.stack(scales),
           "s": np.stack(s_all)}
    if want_deq:
        out["deq"] = deqs
        out["x"] = xs
    return out


def products(xdeq, ydeq):
    """P_r = xhat_r yhat_r^T in binary64 for every term (y stored n' x k')."""
    return [xr @ yr.T for xr, yr in zip(xdeq, ydeq)]


def wcombine(P, wtab: np.ndarray, depth: int, M: int, N: int) -> np.ndarray:
    """C block (I, K) = sum_r w[r, K 2^l + I] P_r, binary64, ascending r."""
    n = 2 ** depth
    mb, nb = M // n, N // n
    C = np.zeros((M, N), dtype=np.float64)
    w64 = np.asarray(wtab, dtype=np.float32).astype(np.float64)
    for r, Pr in enumerate(P):
        for I in range(n):
            for K in range(n):
                c = w64[r, K * n + I]
                if c != 0.0:
                    C[I * mb:(I + 1) * mb, K * nb:(K + 1) * nb] += c * Pr
    return C


def fmm(A: np.ndarray, B: np.ndarray, tables, depth: int, bs: int, rule: int,
        keep: bool = True, b_rows: int = 1, b_bf16: bool = False):
    """One product: the full quantized evaluation for a single (A, B) pair.

    tables = (U, V, w) fp32 flattened tables (T x 4^l).  Returns a dict with
    C (binary64), and the codes/scales of both sides; with keep=True also
    the fp32 combinations and dequantized operands (for the noise model).
    b_rows, b_bf16: the weight (B) side's deployment granularity -- scale
    blocks of b_rows columns of B x bs, and a bfloat16 pre-round of each
    encoded B combination (Appendix E, weight-scale granularity).
    """
    U, V, W = tables
    Mdim, Kdim = A.shape
    Kb, Ndim = B.shape
    if Kb != Kdim:
        raise ValueError("inner dimensions differ")
    ea = encode_side(A, U, depth, bs, rule, "A")
    eb = encode_side(B, V, depth, bs, rule, "B", row_block=b_rows, bf16=b_bf16)
    P = products(ea["deq"], eb["deq"])
    C = wcombine(P, W, depth, Mdim, Ndim)
    out = {"C": C, "a": ea, "b": eb}
    if not keep:
        for side in (ea, eb):
            side.pop("deq"); side.pop("x")
    return out


def fmm_unquantized(A, B, tables, depth: int) -> np.ndarray:
    """The same evaluation with the quantizer bypassed (xhat = x): the fp32
    combinations are multiplied in binary64 and W-combined.  On small integer
    operands with integer coefficients every step is exact, so the result is
    exactly A B for an exact realization (the Brent equations)."""
    U, V, W = tables
    xa = [combine(split(np.asarray(A, np.float32), depth), U[r]).astype(np.float64)
          for r in range(U.shape[0])]
    yb = [combine(split(np.asarray(B, np.float32), depth), V[r]).astype(np.float64).T
          for r in range(V.shape[0])]
    return wcombine(products(xa, yb), W, depth, A.shape[0], B.shape[1])


def reference(A, B) -> np.ndarray:
    """C_ref = A B in binary64 from the float32 operands."""
    return np.asarray(A, np.float64) @ np.asarray(B, np.float64)


def error_sums(C, Cref):
    """(err2, ref2) = (sum (C - C_ref)^2, sum C_ref^2), binary64."""
    C = np.asarray(C, np.float64)
    d = C - Cref
    return float(np.sum(d * d)), float(np.sum(Cref * Cref))


def summarize(err2, ref2):
    """Batch statistics: relMSE as a ratio of sums (the ratio of expectations
    of Appendix D), its square root, and the mean per-product relative
    Frobenius error (the statistic of Table E.1)."""
    err2 = np.asarray(err2, np.float64)
    ref2 = np.asarray(ref2, np.float64)
    rel_mse = float(err2.sum() / ref2.sum())
    return {"rel_mse": rel_mse, "rel_rms": float(np.sqrt(rel_mse)),
            "mean_rel_fro": float(np.mean(np.sqrt(err2 / ref2)))}
