"""GPU parity for realizations of other shapes <m,k,n;R> (the rows of Table
E.1 beyond <2,2,2>): the library's encoder over m x k and k x n sub-block
grids, its large-tile sub-products and its W-combine over the m x n grid of
C against the oracle's fused evaluation (oracle/shapes.py) on the same
seeded inputs, to the bars of tests/gpu_helpers.py: identical codes and
scales, every element of C within the dot-product bound and within
1e-5 |C|_F, the relative MSE within 1% of the oracle's.

The realizations are fmm_inputs.shapes' constructions, each side on its own
<2,2,2> tables.  Grids covered: up to 16 blocks per operand side (the
16-position encoder tile), 20 (the 4-position tile, <4,5,4;80>), a C grid of
25 blocks (the one-column W-combine, <5,2,5;46>), and the others of at most
16 (the four-column W-combine)."""
import numpy as np
import pytest

import fmm_inputs as gen
from fmm_inputs import shapes as S
from gpu_helpers import MSE_REL_TOL, REL_FRO_TOL
from oracle import e4m3, fmm
from oracle import realizations as R
from oracle import shapes as O

pytestmark = pytest.mark.gpu

RULES = {"fp32_amax": e4m3.RULE_FP32_AMAX, "pow2_ceil": e4m3.RULE_POW2_CEIL, "pow2_ocp": e4m3.RULE_POW2_OCP}
CFG = 31       # the input streams of these cases


def lib_realization(name):
    import paper_2609_26077_amd as fm

    def base(which):
        return fm.fmm_realization_coefficients(fm.fmm_realization_builtin(which))
    (m, k, n), U, V, W = S.build(name, base)
    return fm.fmm_realization_create(U, V, W, tol=1e-9, shape=(m, k, n))


def run_case(name, family, batch, mp, kp, np_, bs, rule, exact, trial=0, A=None, B=None):
    import torch
    from paper_2609_26077_amd import FMM_LAYOUT_TILE256x64
    from paper_2609_26077_amd import fmm_operand_views
    from paper_2609_26077_amd.runner import FMM, error_stats, reference_f64
    (m, k, n), _ = S.CATALOG[name]
    M, K, N = m * mp, k * kp, n * np_
    if A is None:
        A, B = gen.operands(family, batch, M, K, N, seed=0, cfg=CFG, trial=trial)
    print(f"shape case {name} {family} batch={batch} M={M} K={K} N={N} bs={bs} rule={rule} exact={exact}",
          flush=True)
    f = FMM(lib_realization(name), batch, M, K, N, 1, bs, rule, exact_dot=exact)
    assert fmm_operand_views(f.plan, f.ws)[0].code_layout == FMM_LAYOUT_TILE256x64
    dA, dB = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
    C = f.matmul(dA, dB)
    Cref = reference_f64(dA, dB)
    err2, ref2 = error_stats(C, Cref)
    torch.cuda.synchronize()
    ops = [t.cpu().numpy() for t in f.operands()]
    return A, B, C.cpu().numpy(), Cref.cpu().numpy(), err2, ref2, ops


def check(name, family, batch, mp, kp, np_, bs, rule_name, exact, trial=0):
    rule = RULES[rule_name]
    mx = (not exact) and rule != e4m3.RULE_FP32_AMAX and bs in (32, 128)
    g_dot = 2.0 ** -10 if mx else 2.0 ** -19
    A, B, Cg, Cr, err2, ref2, ops = run_case(name, family, batch, mp, kp, np_, bs, rule_name, exact, trial)
    D = S.build(name, R.builtin_f64)
    (m, k, n), U = D[0], D[1]
    T = U.shape[0]
    Wt = O.tables_f32(D)[2]
    errs, refs = [], []
    for b in range(batch):
        o = O.fmm_shape(A[b], B[b], D, bs, rule)
        assert np.array_equal(ops[0][b], o["a"]["codes"]), "A codes differ"
        assert np.array_equal(ops[2][b], o["b"]["codes"]), "B codes differ"
        if rule == e4m3.RULE_FP32_AMAX:
            assert np.array_equal(ops[1][b].view(np.uint32), o["a"]["scales"].view(np.uint32))
            assert np.array_equal(ops[3][b].view(np.uint32), o["b"]["scales"].view(np.uint32))
        else:
            assert np.array_equal(ops[1][b], o["a"]["scales"]), "A scales differ"
            assert np.array_equal(ops[3][b], o["b"]["scales"]), "B scales differ"
        Co = o["C"]
        diff = np.abs(Cg[b].astype(np.float64) - Co)
        fro = np.linalg.norm(Co)
        assert diff.max() <= REL_FRO_TOL * fro, (diff.max() / fro)
        Pabs = [np.abs(x) @ np.abs(y).T for x, y in zip(o["a"]["deq"], o["b"]["deq"])]
        Sb = O.wcombine(Pabs, np.abs(Wt), (m, k, n), A.shape[1], B.shape[2])
        bound = (g_dot + (kp + T + 8) * 2.0 ** -24) * Sb
        assert np.count_nonzero(diff > bound) == 0, "elements beyond the dot-product bound"
        ref = fmm.reference(A[b], B[b])
        assert np.allclose(Cr[b], ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())
        e2, r2 = fmm.error_sums(Co, ref)
        errs.append(e2); refs.append(r2)
    rel_gpu = err2.sum() / ref2.sum()
    rel_orc = np.sum(errs) / np.sum(refs)
    assert abs(rel_gpu / rel_orc - 1) <= MSE_REL_TOL, (rel_gpu, rel_orc)
    return rel_gpu


@pytest.mark.parametrize("exact", [False, True], ids=["fp8", "exact"])
@pytest.mark.parametrize("name", sorted(S.CATALOG))
def test_shape_matches_oracle(name, exact):
    check(name, "gaussian", 2, 256, 128, 256, 32, "pow2_ceil", exact)


@pytest.mark.parametrize("name", ["223_11", "333_26", "525_46", "454_80"])
def test_table_e1_setting(name):
    """Table E.1's emulator setting: signed-uniform operands, fp32 amax/448
    scales, blocks of 128 (the fp32-scale exact-dot kernel)."""
    check(name, "uniform", 2, 256, 256, 256, 128, "fp32_amax", False)


@pytest.mark.parametrize("name,bs,rule,exact", [("223_tstar", 16, "pow2_ocp", False),
                                                ("322_11", 128, "pow2_ocp", False),
                                                ("232_11", 128, "pow2_ceil", True),
                                                ("333_27", 16, "fp32_amax", False)])
def test_rules_and_blocks(name, bs, rule, exact):
    check(name, "gaussian", 1, 256, 256, 256, bs, rule, exact)


def test_several_tiles_per_block():
    """Sub-blocks of 512 x 512 by 256: two 256-row tiles per block side and
    several K steps, a batch of three."""
    check("223_11", "gaussian", 3, 512, 256, 512, 32, "pow2_ceil", False)


@pytest.mark.parametrize("name", ["223_11", "525_46", "454_80"])
@pytest.mark.parametrize("exact", [False, True], ids=["fp8", "exact"])
def test_sign_operands_exact(name, exact):
    """+-1 / 0 operands: every combination is a small integer, exact after a
    power-of-two scale, so C must equal A B exactly on either path."""
    (m, k, n), _ = S.CATALOG[name]
    rng = np.random.default_rng(5)
    M, K, N = m * 256, k * 128, n * 256
    A = rng.integers(-1, 2, size=(1, M, K)).astype(np.float32)
    B = rng.integers(-1, 2, size=(1, K, N)).astype(np.float32)
    _, _, Cg, _, _, _, _ = run_case(name, "sign", 1, 256, 128, 256, 32, "pow2_ceil", exact, A=A, B=B)
    assert np.array_equal(Cg[0].astype(np.float64), A[0].astype(np.float64) @ B[0].astype(np.float64))


def test_empty_contraction_and_batch():
    """K = 0: C = 0 with nothing encoded; batch 0: nothing to do."""
    import torch
    from paper_2609_26077_amd.runner import FMM
    f = FMM(lib_realization("525_46"), 2, 1280, 0, 1280, 1, 32, "pow2_ceil")
    C = torch.full((2, 1280, 1280), 7.0, device="cuda")
    f.matmul(torch.empty((2, 1280, 0), device="cuda"), torch.empty((2, 0, 1280), device="cuda"), C)
    torch.cuda.synchronize()
    assert torch.count_nonzero(C).item() == 0
    f0 = FMM(lib_realization("223_11"), 0, 512, 256, 768, 1, 32, "pow2_ceil")
    f0.matmul(torch.empty((0, 512, 256), device="cuda"), torch.empty((0, 256, 768), device="cuda"))
    torch.cuda.synchronize()


def test_cross_shape_predictor_matches_oracle():
    """The cross-shape control (Table E.1's setting) on three rows and two
    samples: each row's mean relative Frobenius error e, its cubic reference
    e_cubic and the error of its re-based realization equal the oracle's on
    the same operands to 1% (the re-based realization, the library's
    optimizer's output from the control's own starts, is the oracle's input),
    and the reported Phi are the realizations' own."""
    import math
    import fmm_inputs as gen_
    import paper_2609_26077_amd as fm
    from paper_2609_26077_amd import controls
    out = controls.cross_shape_predictor(rows=("strassen", "223_11", "333_26"), samples=2, edge=256)
    for row in out["rows"]:
        name = row["realization"]
        m, k, n = row["shape"]
        A, B = gen.operands("uniform", 2, m * 256, k * 256, n * 256, seed=0, cfg=15)
        if name == "strassen":
            D = S.from_222(R.builtin_f64("strassen"))
            C = S.from_222(R.builtin_f64("cubic8"))
            lib = fm.fmm_realization_builtin("strassen")
        else:
            D = S.build(name, R.builtin_f64)
            C = S.cubic(m, k, n)
            lib = controls.shaped_realization(name)
        reb, phi_reb, _ = fm.fmm_realization_optimize(lib, gen_.rebasing_starts_shape(23, m, k, n, seed=0, cfg=16))
        Dreb = ((m, k, n),) + tuple(fm.fmm_realization_coefficients(reb))
        for real, key in ((D, "e"), (C, "e_cubic"), (Dreb, "e_rebased")):
            rel = []
            for b in range(2):
                o = O.fmm_shape(A[b], B[b], real, 128, e4m3.RULE_FP32_AMAX)
                e2, r2 = fmm.error_sums(o["C"], fmm.reference(A[b], B[b]))
                rel.append(math.sqrt(e2 / r2))
            assert row[key] == pytest.approx(np.mean(rel), rel=0.01), (name, key)
        assert row["phi"] == pytest.approx(O.phi(D), rel=1e-14)
        assert row["phi_rebased"] == pytest.approx(phi_reb, rel=1e-14)
        assert row["phi_rebased"] < row["phi"] * (1 - 1e-9)
    assert out["error_lowered_rows"] == out["rebased_rows"] == 3
    print(out, flush=True)
