"""The operand-side rounding energy (fmm_encode_noise; Appendix D, eq. D.1)
against the oracle: per batch element, side and term, the sums of
(xhat - x)^2 and x^2 over the encoded combination, where x is the fp32
combination (before any bfloat16 pre-round) and xhat its decoded e4m3 value;
repeat calls agree bit for bit; the second-moment model of eq. D.8 built
from the GPU's own noise coefficients predicts its measured relative MSE."""
import numpy as np
import pytest

import fmm_inputs as gen
from oracle import e4m3, fmm, model
from oracle import realizations as R

pytestmark = pytest.mark.gpu


def gpu_noise(name, family, b, M, K, N, depth, bs, rule, flags=0, seed=0, cfg=10):
    import torch
    from paper_2609_26077_amd.runner import FMM
    A, B = gen.operands(family, b, M, K, N, seed=seed, cfg=cfg, trial=0)
    dA, dB = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
    f = FMM(name, b, M, K, N, depth, bs, rule, flags=flags)
    f.encode(dA, dB)
    return A, B, f, dA, dB, f.encode_noise(dA, dB)


def oracle_noise(A, B, name, depth, bs, rule, b_rows=1, b_bf16=False):
    U, V, _ = R.tables_f32(R.builtin_f64(name), depth)
    out = []
    for side, (M, tab) in enumerate(((A, U), (B, V))):
        e = fmm.encode_side(M, tab, depth, bs, rule, "AB"[side],
                            row_block=b_rows if side else 1, bf16=b_bf16 and side == 1)
        rows = []
        for x, dq in zip(e["x"], e["deq"]):
            x64 = np.asarray(x, np.float64)
            d = dq - x64
            rows.append((np.sum(d * d), np.sum(x64 * x64)))
        out.append(rows)
    return np.array(out)                      # [2][T][2]


@pytest.mark.parametrize("case", [
    ("tstar", "gaussian", 2, 256, 256, 256, 1, 32, 1, 0),
    ("strassen", "student_t3", 1, 130, 192, 66, 1, 16, 0, 0),      # ragged, fp32 scales, block 16
    ("tstar", "uniform", 1, 256, 512, 256, 2, 32, 2, 0),           # depth 2
    ("winograd", "gaussian", 1, 512, 256, 512, 1, 32, 1, 8),       # large-tile layout (forced)
    ("tstar", "gaussian", 1, 1024, 512, 1024, 2, 32, 1, 8),        # large-tile layout at depth 2
    ("strassen", "gaussian", 1, 512, 256, 512, 1, 32, 0, 8),       # large-tile layout, fp32 scales
    ("tstar", "rowscaled", 1, 256, 512, 256, 1, 128, 1, 0),        # 128 x 128 tile layout, block 128
    ("tstar", "student_t3", 1, 384, 512, 320, 1, 128, 0, 2 | 4),   # deployment granularity
])
def test_noise_matches_oracle(case):
    name, family, b, M, K, N, depth, bs, rule, flags = case
    A, B, f, _, _, g = gpu_noise(name, family, b, M, K, N, depth, bs, rule, flags)
    for i in range(b):
        o = oracle_noise(A[i], B[i], name, depth, bs, rule, b_rows=128 if flags & 2 else 1, b_bf16=bool(flags & 4))
        assert np.allclose(g[i], o, rtol=1e-12, atol=0), (i, np.max(np.abs(g[i] / o - 1)))


def test_noise_is_deterministic():
    A, B, f, dA, dB, g1 = gpu_noise("tstar", "gaussian", 1, 512, 512, 512, 1, 32, 1)
    g2 = f.encode_noise(dA, dB)
    assert np.array_equal(g1, g2)


def test_noise_model_predicts_the_measured_error():
    """eq. D.8: relMSE = (s_A^2 + s_B^2 + s_A^2 s_B^2) Phi / 8 at depth 1; the
    oracle tests hold the oracle's own prediction within 6%."""
    from paper_2609_26077_amd.runner import error_stats, reference_f64
    for name in ("cubic8", "strassen", "tstar"):
        A, B, f, dA, dB, g = gpu_noise(name, "gaussian", 2, 1024, 1024, 1024, 1, 32, 1, seed=1)
        C = f.multiply()
        err2, ref2 = error_stats(C, reference_f64(dA, dB))
        measured = err2.sum() / ref2.sum()
        sa2 = g[:, 0, :, 0].sum() / g[:, 0, :, 1].sum()
        sb2 = g[:, 1, :, 0].sum() / g[:, 1, :, 1].sum()
        phi = R.phi_f64(R.builtin_f64(name))
        predicted = model.predicted_rel_mse(sa2, sb2, phi, 1)
        assert abs(predicted / measured - 1) < 0.08, (name, predicted, measured)


def test_noise_depth3_is_unsupported():
    import paper_2609_26077_amd as fm
    from paper_2609_26077_amd.runner import FMM
    f = FMM("tstar", 1, 64, 128, 64, 3, 16, 1)
    with pytest.raises(fm.FmmError):
        fm.fmm_encode_noise_scratch_size(f.plan)


def test_controls_quick_run():
    """The error-controls driver end to end on small shapes: Rademacher
    cells (Strassen's +-1 combinations are exact in e4m3, T*'s are not, so
    Strassen wins every cell), a small orbit sweep and the calibration
    spreads."""
    from paper_2609_26077_amd import controls
    shapes = [(256, 256, 256), (512, 256, 384)]
    rad = controls.rademacher_cells(shapes)
    assert rad["strassen_wins"] == rad["of"] == 4
    orb = controls.orbit_stability(n_members=4, shape=(256, 256, 256))
    assert orb["cv_pct"] < 5.0
    cal = controls.calibration_transport(shapes, families=("gaussian", "uniform"))
    assert 0 < cal["max_within_family_across_shape_spread_pct"] < 20
    print(rad, orb, cal, flush=True)
