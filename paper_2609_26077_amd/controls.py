"""Synthetic error controls on the batched path (Appendix D; Table E.8).

Each control runs the library's own kernels (encode, sub-products, W-combine,
the fp64 reference and error sums, the operand-noise measurement) and reports
simple statistics of what they return:

* calibration transport: R(F, S, D) = s_q sqrt(2 Phi(D) / mkn) / e_meas
  (the predicted-to-measured ratio of the model's leading term, Appendix D),
  with s_q^2 the mean of the two sides' measured noise coefficients and
  e_meas the relative RMS error, over operand families F and shapes S; the
  spreads 100 (max R - min R) / mean R within a family across shapes and
  within a shape across families;
* orbit-ratio stability: R over exact orbit members D . g of Strassen (random
  g in GL(2)^3), one shape, signed-uniform operands; its coefficient of
  variation;
* designed Rademacher cells: +-1 operands at unit scale and at scale 10 on
  three shapes; whether classic Strassen's measured error is below T*'s;
* cross-r covariance residual: the share of the error's linear part that the
  diagonal sum defining Phi leaves out, (|L|^2 - diag) / |L|^2 from the
  library's cross-term kernels, on six arms (cubic, Strassen, Winograd raw
  and rebalanced, T*, a random orbit member of Strassen) at n = 512, Gaussian
  operands, four seeds, 1 x 128 blocks with fp32 amax/448 scales; the
  armwise means (the paper reports -0.085% to 0.201%).

Usage: python -m paper_2609_26077_amd.controls [--quick]  (prints one JSON object)
"""
from __future__ import annotations

import argparse
import json
import math

import numpy as np
import torch

from . import (fmm_realization_builtin, fmm_realization_metrics, fmm_realization_rebalance,
               fmm_realization_transform)
from .runner import FMM, error_stats, reference_f64

FAMILIES = ("gaussian", "uniform", "student_t3", "laplace", "rowscaled")


def measure(real, A, B, depth=1, block=32, rule="pow2_ceil"):
    """(relMSE, s_A^2, s_B^2, Phi) of one batched run on device operands."""
    b, M, K = A.shape
    N = B.shape[2]
    f = FMM(real, b, M, K, N, depth, block, rule)
    f.encode(A, B)
    noise = f.encode_noise(A, B)
    C = f.multiply()
    err2, ref2 = error_stats(C, reference_f64(A, B))
    sa2 = noise[:, 0, :, 0].sum() / noise[:, 0, :, 1].sum()
    sb2 = noise[:, 1, :, 0].sum() / noise[:, 1, :, 1].sum()
    phi = fmm_realization_metrics(f.real, depth)["phi"]
    return float(err2.sum() / ref2.sum()), float(sa2), float(sb2), float(phi)


def ratio(rel_mse, sa2, sb2, phi, depth=1):
    s_q2 = 0.5 * (sa2 + sb2)
    return math.sqrt(s_q2) * math.sqrt(2.0 * phi / 8.0 ** depth) / math.sqrt(rel_mse)


def spread(values):
    v = np.asarray(values, dtype=np.float64)
    return float(100.0 * (v.max() - v.min()) / v.mean())


def device_operands(family, b, M, K, N, seed, cfg, trial=0):
    import fmm_inputs as gen
    A, B = gen.operands(family, b, M, K, N, seed=seed, cfg=cfg, trial=trial)
    return torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()


def calibration_transport(shapes, families=FAMILIES, realization="tstar", batch=2, seed=0):
    table = {}
    for fam in families:
        for (M, K, N) in shapes:
            A, B = device_operands(fam, batch, M, K, N, seed, 11)
            table[(fam, (M, K, N))] = ratio(*measure(realization, A, B))
    within_family = max(spread([table[(f, s)] for s in shapes]) for f in families)
    within_shape = max(spread([table[(f, s)] for f in families]) for s in shapes)
    return {"ratios": {f"{f}/{s[0]}x{s[1]}x{s[2]}": r for (f, s), r in table.items()},
            "max_within_family_across_shape_spread_pct": within_family,
            "max_within_shape_across_family_spread_pct": within_shape}


def orbit_stability(n_members=15, shape=(1024, 1024, 1024), batch=2, seed=0):
    import fmm_inputs as gen
    base = fmm_realization_builtin("strassen")
    M, K, N = shape
    A, B = device_operands("uniform", batch, M, K, N, seed, 12)
    rs, phis = [], []
    for g in gen.basis_changes(n_members, seed=seed, cfg=12):
        d = fmm_realization_transform(base, *g)
        rel, sa2, sb2, phi = measure(d, A, B)
        rs.append(ratio(rel, sa2, sb2, phi))
        phis.append(phi)
    rs = np.array(rs)
    return {"ratios": rs.tolist(), "phi": phis, "cv_pct": float(100.0 * rs.std() / rs.mean())}


def rademacher_cells(shapes, batch=2, seed=0):
    cells = []
    for fam in ("rademacher", "rademacher10"):
        for (M, K, N) in shapes:
            A, B = device_operands(fam, batch, M, K, N, seed, 13)
            rs = measure("strassen", A, B)[0]
            rt = measure("tstar", A, B)[0]
            cells.append({"family": fam, "shape": [M, K, N], "rel_mse_strassen": rs, "rel_mse_tstar": rt,
                          "strassen_wins": bool(rs < rt)})
    return {"cells": cells, "strassen_wins": sum(c["strassen_wins"] for c in cells), "of": len(cells)}


def cross_r_residual(n=512, seeds=4):
    import fmm_inputs as gen
    s = fmm_realization_builtin("strassen")
    arms = {"cubic8": fmm_realization_builtin("cubic8"), "strassen": s,
            "winograd": fmm_realization_builtin("winograd"),
            "winograd/rebalanced": fmm_realization_rebalance(fmm_realization_builtin("winograd")),
            "tstar": fmm_realization_builtin("tstar"),
            "strassen.g": fmm_realization_transform(s, *gen.basis_changes(1, seed=0, cfg=14)[0])}
    out = {}
    for label, real in arms.items():
        vals = []
        for seed in range(seeds):
            A, B = device_operands("gaussian", 1, n, n, n, seed, 14)
            f = FMM(real, 1, n, n, n, 1, 128, "fp32_amax")
            f.encode(A, B)
            L2, diag = f.cross_terms(A, B)[0]
            vals.append(float((L2 - diag) / L2))
        out[label] = {"mean_pct": 100.0 * float(np.mean(vals)), "per_seed_pct": [100.0 * v for v in vals]}
    means = [v["mean_pct"] for v in out.values()]
    return {"arms": out, "armwise_mean_range_pct": [min(means), max(means)],
            "paper_range_pct": [-0.085, 0.201]}


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--quick", action="store_true", help="small shapes (a smoke run)")
    args = ap.parse_args()
    if args.quick:
        shapes = [(256, 256, 256), (512, 256, 384), (384, 512, 256)]
        orbit = dict(n_members=4, shape=(256, 256, 256))
    else:
        shapes = [(1024, 1024, 1024), (2048, 1024, 1536), (1536, 2048, 1024)]
        orbit = dict(n_members=15, shape=(1024, 1024, 1024))
    out = {"calibration_transport": calibration_transport(shapes),
           "orbit_stability": orbit_stability(**orbit),
           "rademacher": rademacher_cells(shapes),
           "cross_r_residual": cross_r_residual(seeds=1 if args.quick else 4)}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
