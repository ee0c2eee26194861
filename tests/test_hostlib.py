"""The C-ABI library on the CPU: it loads, exports every declared symbol, and
its host-side realization code agrees with the oracle bit for bit (binary64
coefficients and the fp32 tables the kernels use).  No device call here."""
import ctypes
import os
import re

import numpy as np
import pytest

import fmm_inputs as gen
from oracle import realizations as R

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2609_26077_amd", "libfmm8.so")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libfmm8.so not built")


@pytest.fixture(scope="module")
def fm():
    import paper_2609_26077_amd as fm
    return fm


def declared_symbols():
    src = open(os.path.join(ROOT, "include", "fmm8.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(fmm_[a-z0-9_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported(fm):
    lib = ctypes.CDLL(LIB)
    syms = declared_symbols()
    assert len(syms) >= 20
    for s in syms:
        assert hasattr(lib, s), s
    assert set(syms) == set(fm.EXPORTS)


NAMES = {"cubic8": 0, "strassen": 1, "winograd": 2, "tstar": 3}


@pytest.mark.parametrize("name", list(NAMES))
def test_builtin_coefficients_match_oracle(fm, name):
    d = fm.fmm_realization_builtin(name)
    U, V, W = fm.fmm_realization_coefficients(d)
    Uo, Vo, Wo = R.builtin_f64(name)
    assert np.array_equal(U, Uo) and np.array_equal(V, Vo) and np.array_equal(W, Wo)


@pytest.mark.parametrize("name", list(NAMES))
@pytest.mark.parametrize("depth", [1, 2, 3])
def test_tables_match_oracle_bitwise(fm, name, depth):
    d = fm.fmm_realization_builtin(name)
    got = fm.fmm_realization_tables(d, depth)
    want = R.tables_f32(R.builtin_f64(name), depth)
    for a, b in zip(got, want):
        assert a.dtype == np.float32 and np.array_equal(a.view(np.uint32), b.view(np.uint32))


@pytest.mark.parametrize("name,phi,gam", [("cubic8", 8, 8), ("strassen", 32, 14.828427124746190),
                                          ("winograd", 56, 17.853006672199010),
                                          ("tstar", 200 / 9, 12.066031431780)])
def test_metrics(fm, name, phi, gam):
    d = fm.fmm_realization_builtin(name)
    m = fm.fmm_realization_metrics(d, 1)
    assert m["phi"] == pytest.approx(phi, rel=1e-14)
    assert m["gamma"] == pytest.approx(gam, rel=1e-11)
    assert m["brent_residual"] < 1e-15
    m2 = fm.fmm_realization_metrics(d, 2)
    assert m2["phi"] == pytest.approx(phi ** 2, rel=1e-14)


def test_transform_matches_oracle_bitwise(fm):
    """The library evaluates eq. A.1 in the stated binary64 order; the oracle's
    independent implementation of the same order gives identical bits, for
    the 64 random basis changes of the batched sweep and more."""
    base = fm.fmm_realization_builtin("strassen")
    So = R.builtin_f64("strassen")
    gs = gen.basis_changes(64, seed=0) + gen.basis_changes(64, seed=123)
    for X, Y, Z in gs:
        d = fm.fmm_realization_transform(base, X, Y, Z)
        got = fm.fmm_realization_coefficients(d)
        want = R.act_f64(So, (X, Y, Z))
        for a, b in zip(got, want):
            assert np.array_equal(a, b)
        for depth in (1, 2):
            t1 = fm.fmm_realization_tables(d, depth)
            t2 = R.tables_f32(want, depth)
            for a, b in zip(t1, t2):
                assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_transform_rejects_singular(fm):
    base = fm.fmm_realization_builtin("strassen")
    with pytest.raises(fm.FmmError) as e:
        fm.fmm_realization_transform(base, [1, 2, 2, 4], np.eye(2), np.eye(2))
    assert e.value.status == fm.FMM_ERR_SINGULAR


def test_rebalance_matches_oracle(fm):
    for name in ("winograd", "tstar", "strassen"):
        d = fm.fmm_realization_rebalance(fm.fmm_realization_builtin(name))
        got = fm.fmm_realization_coefficients(d)
        want = R.rebalance_f64(R.builtin_f64(name))
        for a, b in zip(got, want):
            assert np.array_equal(a, b)


def test_create_checks_exactness(fm):
    U, V, W = R.builtin_f64("strassen")
    d = fm.fmm_realization_create(U, V, W, tol=0.0)
    assert fm.fmm_realization_terms(d, 2) == (7, 49)
    W2 = W.copy(); W2[3, 1] += 1e-6
    with pytest.raises(fm.FmmError) as e:
        fm.fmm_realization_create(U, V, W2, tol=1e-9)
    assert e.value.status == fm.FMM_ERR_NOT_EXACT
    fm.fmm_realization_create(U, V, W2, tol=1e-5)      # accepted at a looser tolerance
    with pytest.raises(fm.FmmError):
        fm.fmm_realization_create(U, V, W, tol=-1.0)


def test_create_shape_limits(fm):
    """Sizes below one are argument errors; grids of more than 64 blocks
    (m k, k n or n m) are unsupported; both are refused before the
    coefficients are read.  <2,2,2> takes R <= 8, other shapes R <= 4096."""
    import ctypes
    U, V, W = R.builtin_f64("strassen")
    for shape, R_, status in (((0, 2, 2), 7, fm.FMM_ERR_ARG), ((2, -1, 2), 7, fm.FMM_ERR_ARG),
                              ((9, 8, 1), 72, fm.FMM_ERR_UNSUPPORTED), ((1, 8, 9), 72, fm.FMM_ERR_UNSUPPORTED),
                              ((9, 1, 8), 72, fm.FMM_ERR_UNSUPPORTED), ((2, 2, 2), 9, fm.FMM_ERR_ARG),
                              ((2, 2, 3), 4097, fm.FMM_ERR_ARG), ((2, 2, 3), 11, fm.FMM_ERR_ARG)):
        m, k, n = shape
        h = ctypes.c_void_p()
        st = fm._lib.fmm_realization_create(m, k, n, R_, None, None, None, 0.0, ctypes.byref(h))
        assert st == status and not h.value, (shape, st)
    d = fm.fmm_realization_create(U, V, W, tol=0.0, shape=(2, 2, 2))
    assert fm.fmm_realization_terms(d, 1) == (7, 7)
    assert fm.fmm_realization_shape(d) == ((2, 2, 2), 7)


@pytest.mark.parametrize("desc,status", [
    (dict(batch=1, M=256, K=256, N=256, depth=4), -1),        # depth out of range
    (dict(batch=1, M=256, K=256, N=256, block=64), -1),       # block not 16/32/128
    (dict(batch=1, M=256, K=256, N=256, rule=7), -1),         # unknown rule
    (dict(batch=-1, M=256, K=256, N=256), -1),
    (dict(batch=1, M=255, K=256, N=256), -2),                 # M not divisible by 2
    (dict(batch=1, M=256, K=256, N=256, depth=3, block=128), -2),   # k' = 32 not / 128
    (dict(batch=1, M=256, K=96, N=256, block=32), -2),        # k' = 48 not / 32
    (dict(batch=70000, M=2, K=64, N=2), -3),                  # batch beyond the grid
    (dict(batch=1, M=256, K=256, N=256, flags=16), -1),       # unknown flag bit
    (dict(batch=1, M=256, K=256, N=256, depth=2, flags=2), -3),   # 128-row B blocks: depth 1 only
    (dict(batch=1, M=256, K=256, N=256, depth=2, flags=4), -3),   # bfloat16 pre-round: depth 1 only
])
def test_plan_validation_before_device(fm, desc, status):
    d = fm.fmm_realization_builtin("tstar")
    kw = dict(batch=1, M=256, K=256, N=256, depth=1, block=32, rule="pow2_ceil")
    kw.update(desc)
    st = fm.fmm_plan_create_status(d, fm.make_desc(**kw))
    assert st == status


def test_status_strings(fm):
    for s in range(0, -10, -1):
        assert fm.fmm_status_string(s) != "unknown status"
    assert fm.fmm_status_string(-99) == "unknown status"


# ---- re-basing (fmm_realization_optimize, fmm_realization_phi_gradient) -----

PHI_MIN = 200.0 / 9.0
GAMMA_MIN = 2.0 * np.sqrt(2.0) + 16.0 / np.sqrt(3.0)


@pytest.mark.parametrize("name", ["strassen", "winograd", "tstar", "cubic8"])
def test_phi_gradient_matches_oracle(fm, name):
    from oracle import rebase as RB
    d = fm.fmm_realization_builtin(name)
    D = R.builtin_f64(name)
    for x in [RB.IDENTITY] + list(gen.rebasing_starts(6, seed=11)):
        phi, grad = fm.fmm_realization_phi_gradient(d, x)
        ophi, ograd = RB.phi_and_grad(D, x)
        assert phi == pytest.approx(ophi, rel=1e-13)
        assert np.max(np.abs(grad - ograd)) <= 1e-11 * max(1.0, np.max(np.abs(ograd)))


@pytest.mark.parametrize("name", ["strassen", "winograd"])
def test_optimize_matches_oracle(fm, name):
    from oracle import rebase as RB
    starts = gen.rebasing_starts(23, seed=0)
    best, phi, start_phi = fm.fmm_realization_optimize(fm.fmm_realization_builtin(name), starts)
    obest, ophi, oterm = RB.rebase(R.builtin_f64(name), starts)
    # the minimum value is unique (Theorem 1); the minimizer is not (gauge orbit)
    assert phi == pytest.approx(ophi, rel=1e-12)
    assert phi == pytest.approx(PHI_MIN, rel=1e-12)
    assert np.allclose(start_phi, oterm, rtol=1e-10, atol=0)
    m = fm.fmm_realization_metrics(best, 1)
    assert m["phi"] == pytest.approx(phi, rel=1e-15)
    assert m["gamma"] == pytest.approx(GAMMA_MIN, rel=1e-10)
    assert m["brent_residual"] <= 1e-12


def test_optimize_random_orbit_points(fm):
    t = fm.fmm_realization_builtin("tstar")
    for x in gen.rebasing_starts(4, seed=13):
        X, Y, Z = x.reshape(3, 2, 2)
        d = fm.fmm_realization_transform(t, X, Y, Z)
        assert fm.fmm_realization_metrics(d, 1)["phi"] > PHI_MIN * (1 + 1e-3)
        best, phi, _ = fm.fmm_realization_optimize(d)
        assert phi == pytest.approx(PHI_MIN, rel=1e-12)
        assert fm.fmm_realization_metrics(best, 1)["brent_residual"] <= 1e-12


def test_optimize_argument_and_exactness_errors(fm):
    import ctypes
    d = fm.fmm_realization_builtin("strassen")
    out, phi = ctypes.c_void_p(), ctypes.c_double()
    starts = gen.rebasing_starts(1, seed=0)
    sp = starts.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
    lib = fm._lib
    assert lib.fmm_realization_optimize(d.handle, -1, None, 10, 1e-10, 1e-9, ctypes.byref(out), None, None) == fm.FMM_ERR_ARG
    assert lib.fmm_realization_optimize(d.handle, 1, None, 10, 1e-10, 1e-9, ctypes.byref(out), None, None) == fm.FMM_ERR_ARG
    assert lib.fmm_realization_optimize(d.handle, 1, sp, 0, 1e-10, 1e-9, ctypes.byref(out), None, None) == fm.FMM_ERR_ARG
    assert lib.fmm_realization_optimize(d.handle, 1, sp, 10, 0.0, 1e-9, ctypes.byref(out), None, None) == fm.FMM_ERR_ARG
    assert lib.fmm_realization_optimize(d.handle, 1, sp, 10, 1e-10, -1.0, ctypes.byref(out), None, None) == fm.FMM_ERR_ARG
    assert lib.fmm_realization_optimize(None, 1, sp, 10, 1e-10, 1e-9, ctypes.byref(out), None, None) == fm.FMM_ERR_ARG
    # a realization that is not a <2,2,2> algorithm: no start ends exact
    U, V, W = (np.array(M) for M in R.builtin_f64("strassen"))
    U[2, 0] = -U[2, 0]
    bad = fm.fmm_realization_create(U, V, W, tol=10.0)
    st = lib.fmm_realization_optimize(bad.handle, 1, sp, 100, 1e-10, 1e-9, ctypes.byref(out), ctypes.byref(phi), None)
    assert st == fm.FMM_ERR_NOT_EXACT and not out.value


def test_one_hip_runtime_whatever_the_import_order():
    """Importing the package before torch must not map a second HIP runtime
    (the library takes torch's device pointers, so both must use one)."""
    import subprocess
    import sys
    code = ("import paper_2609_26077_amd, torch\n"
            "libs = {l.split()[-1] for l in open('/proc/self/maps') if 'libamdhip64' in l}\n"
            "print(len(libs))\n")
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, cwd=ROOT, timeout=300)
    assert out.returncode == 0, out.stderr
    assert out.stdout.strip().splitlines()[-1] == "1", out.stdout


def test_noalloc_error_stats_rejects_before_any_device_call(fm):
    """The allocation-free reduction refuses a batch beyond its static
    scratch, and bad sizes, without touching a device (this runs on a CPU)."""
    n = fm.FMM_ERROR_STATS_NOALLOC_MAX_BATCH + 1
    st = fm._lib.fmm_error_stats_noalloc(n, 4, 4, None, None, None, None)
    assert st == fm.FMM_ERR_WORKSPACE
    assert b"exceeds the static scratch" in fm._lib.fmm_last_error_detail()
    assert fm._lib.fmm_error_stats_noalloc(-1, 4, 4, None, None, None, None) == fm.FMM_ERR_ARG
    assert fm._lib.fmm_error_stats_noalloc(0, 4, 4, None, None, None, None) == fm.FMM_OK
    assert fm._lib.fmm_error_stats_noalloc(2, 4, 4, None, None, None, None) == fm.FMM_ERR_ARG


def test_error_stats_scratch_checks_before_any_device_call(fm):
    """fmm_error_stats refuses a scratch that is too small or not 8-byte
    aligned, and bad sizes, before any device call (the pointers below are
    never dereferenced; this runs on a CPU)."""
    lib = fm._lib
    need = ctypes.c_size_t(0)
    assert lib.fmm_error_stats_scratch_size(3, 64, 64, ctypes.byref(need)) == fm.FMM_OK
    assert need.value > 0
    fake = 1 << 40                                   # non-null, 256-byte aligned
    args = (3, 64, 64, fake, fake, fake)
    assert lib.fmm_error_stats(*args, fake, need.value - 1, None) == fm.FMM_ERR_WORKSPACE
    assert lib.fmm_error_stats(*args, fake + 4, need.value, None) == fm.FMM_ERR_WORKSPACE
    assert lib.fmm_error_stats(*args, None, need.value, None) == fm.FMM_ERR_WORKSPACE
    assert lib.fmm_error_stats(-1, 64, 64, fake, fake, fake, fake, need.value, None) == fm.FMM_ERR_ARG
    assert lib.fmm_error_stats(3, 64, 64, fake, fake, None, fake, need.value, None) == fm.FMM_ERR_ARG
    assert lib.fmm_error_stats(0, 64, 64, None, None, None, None, 0, None) == fm.FMM_OK
