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
  armwise means (the paper reports -0.085% to 0.201%);
* cross-shape predictor (Section 3's breadth test; Appendix E's protocol and
  Table E.1's setting): over realizations of several shapes <m,k,n;R> (the
  <2,2,2> builtins and fmm_inputs.shapes' constructions), one level, signed-
  uniform operands, eight paired samples at block edge 256, 1 x 128 blocks
  with fp32 amax/448 scales, the mean relative Frobenius error e of each and
  of the cubic algorithm of its shape on the same operands, and the
  Spearman correlation (average ranks for ties) of e with the coefficient-
  only predictors sqrt(Phi / mkn), sqrt(Phi) and GQ_chi (Appendix E: each
  term rescaled to |U_r| = |V_r| = 1 with the magnitude moved into W_r;
  chi_r^A = 0 when the rescaled U_r has exactly one entry of magnitude
  >= 1e-6, else 1, chi_r^B likewise; GQ_chi = (mean_q sum_r W_rq^2
  (chi_r^A + chi_r^B))^(1/2)); and the intervention of Section 3: each
  realization re-based over its own orbit GL(m) x GL(k) x GL(n) (the
  identity and 23 perturbed starts, Appendix E.2's protocol) and measured on
  the same operands, e_reb / e_cubic beside e_lib / e_cubic.

Usage: python -m paper_2609_26077_amd.controls [--quick] [--only NAME]  (prints one JSON object)
"""
from __future__ import annotations

import argparse
import json
import math

import numpy as np
import torch

from . import (fmm_realization_builtin, fmm_realization_coefficients, fmm_realization_create,
               fmm_realization_metrics, fmm_realization_optimize, fmm_realization_rebalance,
               fmm_realization_shape, fmm_realization_transform)
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


def shaped_realization(name):
    """A realization of fmm_inputs.shapes.CATALOG (or the cubic algorithm
    "cubic_<m><k><n>") built on the library's own <2,2,2> tables."""
    from fmm_inputs import shapes as S
    if name.startswith("cubic_"):
        (m, k, n), U, V, W = S.cubic(*(int(c) for c in name[6:]))
    else:
        (m, k, n), U, V, W = S.build(
            name, lambda which: fmm_realization_coefficients(fmm_realization_builtin(which)))
    return fmm_realization_create(U, V, W, tol=1e-9, shape=(m, k, n))


def gq_chi(real):
    """Appendix E's coefficient-growth heuristic GQ_chi of a realization."""
    U, V, W = fmm_realization_coefficients(real)
    nu = np.linalg.norm(U, axis=1)
    nv = np.linalg.norm(V, axis=1)
    ok = (nu > 0) & (nv > 0)
    Ur = U[ok] / nu[ok, None]
    Vr = V[ok] / nv[ok, None]
    Wr = W[ok] * (nu[ok] * nv[ok])[:, None]
    chi_a = (np.count_nonzero(np.abs(Ur) >= 1e-6, axis=1) != 1).astype(np.float64)
    chi_b = (np.count_nonzero(np.abs(Vr) >= 1e-6, axis=1) != 1).astype(np.float64)
    return float(np.sqrt(np.mean(np.sum(Wr ** 2 * (chi_a + chi_b)[:, None], axis=0))))


def spearman(x, y):
    """Spearman correlation with average ranks for ties."""
    from scipy.stats import rankdata
    rx, ry = rankdata(x), rankdata(y)
    return float(np.corrcoef(rx, ry)[0, 1])


CROSS_SHAPE_ROWS = ("strassen", "winograd", "tstar", "223_11", "223_tstar", "322_11", "232_11",
                    "333_26", "525_46")


def cross_shape_predictor(rows=CROSS_SHAPE_ROWS, samples=8, edge=256, seed=0, rebase_starts=23):
    import fmm_inputs as gen
    rows_out, cubic_e = [], {}
    for name in rows:
        real = fmm_realization_builtin(name) if name in ("strassen", "winograd", "tstar") else shaped_realization(name)
        (m, k, n), R = fmm_realization_shape(real)
        M, K, N = m * edge, k * edge, n * edge
        A, B = device_operands("uniform", samples, M, K, N, seed, 15)

        def mean_rel_fro(d):
            f = FMM(d, samples, M, K, N, 1, 128, "fp32_amax")
            err2, ref2 = error_stats(f.matmul(A, B), reference_f64(A, B))
            return float(np.mean(np.sqrt(err2 / ref2)))

        key = (m, k, n, seed)
        if key not in cubic_e:
            cub = fmm_realization_builtin("cubic8") if (m, k, n) == (2, 2, 2) else shaped_realization(f"cubic_{m}{k}{n}")
            cubic_e[key] = mean_rel_fro(cub)
        e = mean_rel_fro(real)
        phi = fmm_realization_metrics(real, 1)["phi"]
        row = {"realization": name, "shape": [m, k, n], "rank": R, "phi": phi,
               "sqrt_phi_over_mkn": math.sqrt(phi / (m * k * n)), "gq_chi": gq_chi(real),
               "e": e, "e_cubic": cubic_e[key], "e_over_e_cubic": e / cubic_e[key]}
        if rebase_starts is not None:
            starts = gen.rebasing_starts_shape(rebase_starts, m, k, n, seed=seed, cfg=16)
            reb, phi_reb, _ = fmm_realization_optimize(real, starts)
            e_reb = mean_rel_fro(reb)
            row.update({"phi_rebased": phi_reb, "e_rebased": e_reb, "e_rebased_over_e_cubic": e_reb / cubic_e[key]})
        rows_out.append(row)
    e = [r["e"] for r in rows_out]
    out_reb = {}
    if rebase_starts is not None:
        moved = [r for r in rows_out if r["phi_rebased"] < r["phi"] * (1 - 1e-9)]
        out_reb = {"rebased_rows": len(moved), "error_lowered_rows": sum(r["e_rebased"] < r["e"] for r in moved),
                   "min_error_reduction": min((r["e"] / r["e_rebased"] for r in moved), default=None),
                   "rebase_starts": rebase_starts}
    return {"rows": rows_out, **out_reb,
            "spearman_sqrt_phi_over_mkn": spearman([r["sqrt_phi_over_mkn"] for r in rows_out], e),
            "spearman_sqrt_phi": spearman([math.sqrt(r["phi"]) for r in rows_out], e),
            "spearman_gq_chi": spearman([r["gq_chi"] for r in rows_out], e),
            "setting": {"family": "uniform", "samples": samples, "edge": edge, "block": 128,
                        "rule": "fp32_amax", "depth": 1}}


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--quick", action="store_true", help="small shapes (a smoke run)")
    ap.add_argument("--only", choices=("calibration_transport", "orbit_stability", "rademacher",
                                       "cross_r_residual", "cross_shape_predictor"),
                    help="run one control")
    args = ap.parse_args()
    if args.only == "cross_shape_predictor":
        print(json.dumps({args.only: cross_shape_predictor(samples=2 if args.quick else 8)}), flush=True)
        return
    if args.only == "cross_r_residual":
        print(json.dumps({args.only: cross_r_residual(seeds=1 if args.quick else 4)}), flush=True)
        return
    if args.quick:
        shapes = [(256, 256, 256), (512, 256, 384), (384, 512, 256)]
        orbit = dict(n_members=4, shape=(256, 256, 256))
    else:
        shapes = [(1024, 1024, 1024), (2048, 1024, 1536), (1536, 2048, 1024)]
        orbit = dict(n_members=15, shape=(1024, 1024, 1024))
    if args.only == "calibration_transport":
        print(json.dumps({args.only: calibration_transport(shapes)}), flush=True)
        return
    if args.only == "orbit_stability":
        print(json.dumps({args.only: orbit_stability(**orbit)}), flush=True)
        return
    if args.only == "rademacher":
        print(json.dumps({args.only: rademacher_cells(shapes)}), flush=True)
        return
    out = {"calibration_transport": calibration_transport(shapes),
           "orbit_stability": orbit_stability(**orbit),
           "rademacher": rademacher_cells(shapes),
           "cross_r_residual": cross_r_residual(seeds=1 if args.quick else 4),
           "cross_shape_predictor": cross_shape_predictor(samples=2 if args.quick else 8)}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
