"""Seeded synthetic inputs shared by the oracle, the tests and the benchmark.

This module draws random numbers and nothing else: it holds none of the
method's arithmetic (no combine, no quantizer, no product).  Both the CPU
oracle and the GPU path receive the arrays it returns as inputs.

Streams: every array comes from its own
``numpy.random.Generator(PCG64(SeedSequence([seed, cfg, trial, operand])))``
so that any one trial of any configuration can be regenerated alone, and the
same operands serve every arm (realization) of a configuration (paired
comparison, as in the paper's emulator protocol, Appendix E.2).

Operand families (the paper's synthetic family is "signed-uniform",
Appendix E.2; the others are the benchmark configurations' families):

* ``gaussian``   iid N(0,1)
* ``uniform``    iid Uniform[-1, 1]
* ``student_t3`` iid Student-t with nu=3, divided by sqrt(3) so the variance
  is one (Var t_nu = nu/(nu-2) = 3)
* ``rowscaled``  iid N(0,1), then every row multiplied by 10**U(-2, 2)
  (a log-uniform factor over [1e-2, 1e2]); the factor is applied in float64
  before the cast to float32.  For B the rows run along the contracted axis.

Random basis changes g = (X, Y, Z) in GL(2)^3 follow the paper's restart
distribution for re-basing (Appendix E.2): each factor is I + 0.45 * N(0,1)
entrywise, and a draw whose determinant has absolute value below 1e-3 is
rejected and redrawn from the same stream.
"""
from __future__ import annotations

import numpy as np

FAMILIES = ("gaussian", "uniform", "student_t3", "rowscaled")

# operand ids inside the SeedSequence
OPERAND_A = 0
OPERAND_B = 1
OPERAND_G = 4  # basis changes


def generator(seed: int, cfg: int, trial: int, operand: int) -> np.random.Generator:
    """The PCG64 stream for one (seed, config, trial, operand) key."""
    ss = np.random.SeedSequence([int(seed), int(cfg), int(trial), int(operand)])
    return np.random.Generator(np.random.PCG64(ss))


def draw(family: str, shape, rng: np.random.Generator) -> np.ndarray:
    """Draw one float32 array of ``shape`` from ``family``.

    ``shape`` is (..., rows, cols); for ``rowscaled`` one factor is drawn per
    row of every trailing matrix.
    """
    shape = tuple(int(s) for s in shape)
    if family == "gaussian":
        return rng.standard_normal(shape, dtype=np.float32)
    if family == "uniform":
        return rng.uniform(-1.0, 1.0, size=shape).astype(np.float32)
    if family == "student_t3":
        x = rng.standard_t(3.0, size=shape) / np.sqrt(3.0)
        return x.astype(np.float32)
    if family == "rowscaled":
        x = rng.standard_normal(shape)  # float64
        f = 10.0 ** rng.uniform(-2.0, 2.0, size=shape[:-1] + (1,))
        return (x * f).astype(np.float32)
    if family == "rademacher":
        return np.where(rng.integers(0, 2, size=shape) == 0, -1.0, 1.0).astype(np.float32)
    if family == "rademacher10":
        return np.where(rng.integers(0, 2, size=shape) == 0, -10.0, 10.0).astype(np.float32)
    if family == "laplace":
        return (rng.laplace(0.0, 1.0 / np.sqrt(2.0), size=shape)).astype(np.float32)
    if family == "ones":
        # a control, not a workload: every encoded combination of a term is
        # one constant, so every code of the term is the same byte
        return np.ones(shape, dtype=np.float32)
    raise ValueError(f"unknown operand family {family!r}")


def operands(family: str, batch: int, M: int, K: int, N: int,
             seed: int = 0, cfg: int = 0, trial: int = 0):
    """(A, B) float32, C-contiguous, shapes (batch, M, K) and (batch, K, N)."""
    A = draw(family, (batch, M, K), generator(seed, cfg, trial, OPERAND_A))
    B = draw(family, (batch, K, N), generator(seed, cfg, trial, OPERAND_B))
    return np.ascontiguousarray(A), np.ascontiguousarray(B)


def basis_change(rng: np.random.Generator, scale: float = 0.45,
                 min_abs_det: float = 1e-3):
    """One g = (X, Y, Z): three float64 2x2 matrices, each I + scale*N(0,1)."""
    out = []
    for _ in range(3):
        while True:
            g = np.eye(2) + scale * rng.standard_normal((2, 2))
            if abs(g[0, 0] * g[1, 1] - g[0, 1] * g[1, 0]) >= min_abs_det:
                out.append(g)
                break
    return tuple(out)


def basis_changes(count: int, seed: int = 0, cfg: int = 4):
    """``count`` basis changes; change i is drawn from key [seed, cfg, i, 4]."""
    return [basis_change(generator(seed, cfg, i, OPERAND_G)) for i in range(count)]


def rebasing_starts(count: int, seed: int = 0, cfg: int = 6) -> np.ndarray:
    """``count`` re-basing starts as a (count, 12) float64 array: row i is
    (X, Y, Z) of basis change i (drawn as in ``basis_changes`` from key
    [seed, cfg, i, 4]), each 2x2 flattened row-major."""
    out = np.empty((count, 12), dtype=np.float64)
    for i, g in enumerate(basis_changes(count, seed=seed, cfg=cfg)):
        out[i] = np.concatenate([m.reshape(-1) for m in g])
    return out


def rebasing_starts_shape(count: int, m: int, k: int, n: int, seed: int = 0, cfg: int = 16) -> np.ndarray:
    """``count`` re-basing starts for a realization of another shape <m,k,n>,
    as a (count, m^2 + k^2 + n^2) float64 array: row i is (X, Y, Z), each
    I + 0.45 N(0,1) of size m, k, n (flattened row-major), a factor with
    |det| < 1e-3 redrawn from the same stream (key [seed, cfg, i, 4]), as the
    <2,2,2> starts are drawn."""
    out = np.empty((count, m * m + k * k + n * n), dtype=np.float64)
    for i in range(count):
        rng = generator(seed, cfg, i, OPERAND_G)
        parts = []
        for size in (m, k, n):
            while True:
                g = np.eye(size) + 0.45 * rng.standard_normal((size, size))
                if abs(np.linalg.det(g)) >= 1e-3:
                    parts.append(g.reshape(-1))
                    break
        out[i] = np.concatenate(parts)
    return out
