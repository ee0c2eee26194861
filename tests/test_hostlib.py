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


@pytest.mark.parametrize("desc,status", [
    (dict(batch=1, M=256, K=256, N=256, depth=4), -1),        # depth out of range
    (dict(batch=1, M=256, K=256, N=256, block=64), -1),       # block not 16/32/128
    (dict(batch=1, M=256, K=256, N=256, rule=7), -1),         # unknown rule
    (dict(batch=-1, M=256, K=256, N=256), -1),
    (dict(batch=1, M=255, K=256, N=256), -2),                 # M not divisible by 2
    (dict(batch=1, M=256, K=256, N=256, depth=3, block=128), -2),   # k' = 32 not / 128
    (dict(batch=1, M=256, K=96, N=256, block=32), -2),        # k' = 48 not / 32
    (dict(batch=70000, M=2, K=64, N=2), -3),                  # batch beyond the grid
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
