"""Pins of the oracle's e4m3 codec and block-scale rules.

The codec is checked against brute-force nearest-code search over exact
rationals (the definition), against closed-form special values of the OCP
E4M3 format, and the plain-C twin against the numpy version.  The scale
rules are checked against their definitions by direct search and against
homogeneity: a power-of-two factor moves the scale and leaves the codes.
"""
import ctypes
import os
import subprocess
from fractions import Fraction

import numpy as np
import pytest

from oracle import e4m3

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def oracle_c_lib():
    """Build (if needed) and load the plain-C codec of the oracle."""
    src = os.path.join(ROOT, "oracle", "e4m3_ref.c")
    so = os.path.join(ROOT, "oracle", "libe4m3_ref.so")
    if not os.path.exists(so) or os.path.getmtime(so) < os.path.getmtime(src):
        subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-ffp-contract=off",
                               "-fno-fast-math", src, "-o", so, "-lm"])
    lib = ctypes.CDLL(so)
    lib.oracle_e4m3_encode.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t]
    lib.oracle_e4m3_sweep.argtypes = [ctypes.c_uint32, ctypes.c_size_t, ctypes.c_void_p]
    lib.oracle_e4m3_sweep_pow2.argtypes = [ctypes.c_uint32, ctypes.c_size_t, ctypes.c_int,
                                           ctypes.c_void_p]
    return lib


def test_format_constants():
    vals = e4m3.DECODE
    finite = vals[~np.isnan(vals)]
    assert len(finite) == 254
    assert np.isnan(vals[0x7F]) and np.isnan(vals[0xFF])
    assert finite.max() == 448.0 and finite.min() == -448.0
    pos = np.sort(finite[finite > 0])
    assert pos[0] == 2.0 ** -9                    # smallest subnormal
    assert vals[0x08] == 2.0 ** -6                # smallest normal
    assert vals[0x80] == 0.0 and np.signbit(vals[0x80])
    assert vals[0x7E] == 448.0


def _random_inputs(n, rng):
    """float32 values concentrated where the codec's decisions are made."""
    mag = 2.0 ** rng.uniform(-12, 10, n)
    v = (mag * rng.choice([-1, 1], n)).astype(np.float32)
    # exact midpoints between neighbouring codes, and their float32 neighbours
    pos = np.sort(e4m3.DECODE[:0x7F])
    mids = ((pos[1:] + pos[:-1]) / 2).astype(np.float32)
    extra = np.concatenate([mids, np.nextafter(mids, np.float32(0)),
                            np.nextafter(mids, np.float32(1e9)), -mids,
                            np.float32([0.0, -0.0, 448, 449, 463.99, 464, 464.01, 480,
                                        500, 1e6, -1e6, 2 ** -10, -(2 ** -10),
                                        1.5 * 2 ** -10, 1e-30, -1e-30, 3.4e38])])
    return np.concatenate([v, extra]).astype(np.float32)


def test_encode_matches_bruteforce():
    rng = np.random.default_rng(0)
    v = _random_inputs(3000, rng)
    got = e4m3.encode(v)
    want = np.array([e4m3.encode_bruteforce(float(x)) for x in v], dtype=np.uint8)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, [(float(v[i]), hex(got[i]), hex(want[i])) for i in bad[:5]]


@pytest.mark.parametrize("v,code", [
    (0.0, 0x00), (-0.0, 0x80), (448.0, 0x7E), (-448.0, 0xFE),
    (464.0, 0x7E),            # midpoint to the (absent) 480: saturates
    (1e9, 0x7E), (-1e9, 0xFE),
    (2.0 ** -9, 0x01), (2.0 ** -10, 0x00),     # tie between 0 and 2^-9 -> even (0)
    (-(2.0 ** -10), 0x80),                       # negative zero keeps the sign
    (3 * 2.0 ** -10, 0x02),                      # tie 1 vs 2 (x 2^-9) -> even 2
    (1.0, 0x38), (1.0625, 0x38), (1.1875, 0x3A),  # ties to even mantissa
    (17.0, 0x58), (240.0, 0x77), (256.0, 0x78),
])
def test_encode_special_values(v, code):
    assert int(e4m3.encode(np.float32([v]))[0]) == code
    assert e4m3.encode_bruteforce(v) == code


def test_c_codec_matches_numpy_codec():
    lib = oracle_c_lib()
    rng = np.random.default_rng(1)
    bits = rng.integers(0, 2 ** 32, 2_000_000, dtype=np.uint64).astype(np.uint32)
    v = bits.view(np.float32)
    v = v[np.isfinite(v)]
    v = np.concatenate([v, _random_inputs(200000, rng)])
    out = np.empty(v.size, dtype=np.uint8)
    lib.oracle_e4m3_encode(v.ctypes.data, out.ctypes.data, v.size)
    assert np.array_equal(out, e4m3.encode(v))
    # the sweep entry point enumerates bit patterns
    start = 0x3F7FFF00
    sw = np.empty(4096, dtype=np.uint8)
    lib.oracle_e4m3_sweep(start, 4096, sw.ctypes.data)
    pat = (start + np.arange(4096, dtype=np.uint64)).astype(np.uint32).view(np.float32)
    assert np.array_equal(sw, e4m3.encode(pat))


def test_decode_encode_roundtrip():
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], dtype=np.uint8)
    vals = e4m3.decode(codes).astype(np.float32)
    assert np.array_equal(e4m3.encode(vals), codes)


# --------------------------------------------------------------------------
# Scale rules
# --------------------------------------------------------------------------

def _ceil_by_search(a):
    e = -200
    while Fraction(float(a)) > 448 * Fraction(2) ** e:
        e += 1
    return e


def _floor_log2_by_search(a):
    e = -200
    while Fraction(2) ** (e + 1) <= Fraction(float(a)):
        e += 1
    return e


def test_pow2_rules_match_definitions():
    rng = np.random.default_rng(2)
    a = (2.0 ** rng.uniform(-40, 40, 400)).astype(np.float32)
    a = np.concatenate([a, np.float32([448, 448 * 2.0 ** -3, np.nextafter(np.float32(448), np.float32(1e9)),
                                       1.75, 1.7500001, 1.0, 1e-12, 3e38])]).astype(np.float32)
    ec = e4m3.pow2_ceil_exponent(a)
    eo = e4m3.pow2_ocp_exponent(a)
    for x, c, o in zip(a, ec, eo):
        assert c == _ceil_by_search(x)
        assert o == _floor_log2_by_search(x) - 8


def test_fp32_amax_scale_is_one_division():
    a = np.float32([1.0, 3.0, 448.0, 7.0, 1e-3])
    s, st = e4m3.block_scales(a, e4m3.RULE_FP32_AMAX)
    for x, y in zip(a, s):
        assert y == np.float32(Fraction(float(x)) / 448)    # RNE of the exact quotient
    assert st.dtype == np.float32


def test_clamp_and_zero_block():
    """amax is clamped at fl32(1e-12) before the scale (Appendix E.2); an
    all-zero block gets the clamp's scale and zero codes (sign kept)."""
    x = np.zeros((2, 32), np.float32); x[1, 3] = -0.0
    for rule in (0, 1, 2):
        codes, stored, s, deq = e4m3.quantize_rows(x, 32, rule)
        assert np.all(codes[0] == 0) and codes[1, 3] == 0x80
        s_clamp, _ = e4m3.block_scales(np.float32([1e-12]), rule)
        assert np.all(s == s_clamp[0])
    s, st = e4m3.block_scales(np.float32([1e-12]), e4m3.RULE_POW2_CEIL)
    assert int(st[0]) == 127 + _ceil_by_search(np.float32(1e-12))


def test_ocp_rule_saturates_and_ceil_never_does():
    """POW2_OCP maps the top of a block to [256, 512) and clips it to 448;
    POW2_CEIL keeps every scaled value within 448."""
    rng = np.random.default_rng(3)
    x = rng.standard_normal((64, 32)).astype(np.float32)
    for rule in (1, 2):
        codes, stored, s, deq = e4m3.quantize_rows(x, 32, rule)
        v = x.reshape(64, 1, 32) / s[:, :, None]
        if rule == 1:
            assert np.abs(v).max() <= 448
        else:
            assert np.abs(v).max() >= 256
            assert np.any((codes & 0x7F) == 0x7E)


@pytest.mark.parametrize("rule", [0, 1, 2])
def test_power_of_two_homogeneity(rule):
    """A per-block dynamic scale is positively homogeneous (Appendix E.2):
    multiplying a block by 2^k leaves its codes unchanged and multiplies its
    scale by 2^k (while the clamp stays disengaged)."""
    rng = np.random.default_rng(4)
    x = rng.standard_normal((16, 128)).astype(np.float32)
    c0, st0, s0, d0 = e4m3.quantize_rows(x, 32, rule)
    for k in (-20, -3, 5, 30):
        f = np.float32(2.0 ** k)
        c1, st1, s1, d1 = e4m3.quantize_rows(x * f, 32, rule)
        assert np.array_equal(c0, c1)
        assert np.array_equal(s1, (s0 * f).astype(np.float32))
        assert np.array_equal(d1, d0 * float(f))


# ---- deployment granularity: bfloat16 pre-round, 2-D weight blocks ----------

def test_bf16_round_matches_torch_conversion():
    """torch's float32 -> bfloat16 cast rounds to nearest even: a library
    routine the definition reduces to."""
    import torch
    rng = np.random.default_rng(7)
    x = (rng.standard_normal(400_000) * np.exp(rng.uniform(-85, 85, 400_000))).astype(np.float32)
    bits = rng.integers(0, 2 ** 32, 400_000, dtype=np.uint64).astype(np.uint32).view(np.float32)
    x = np.concatenate([x, bits[np.isfinite(bits)], np.float32([0.0, -0.0, 1e-45, -1e-45, 1.17549435e-38])])
    got = e4m3.bf16_round(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


def test_bf16_round_special_values():
    f = lambda v: float(e4m3.bf16_round(np.float32(v)))
    assert f(1 + 2 ** -8) == 1.0                      # tie -> even (mantissa 0)
    assert f(1 + 3 * 2 ** -8) == 1 + 2 ** -6          # tie -> even (mantissa 2)
    assert f(1 + 2 ** -8 + 2 ** -20) == 1 + 2 ** -7   # above the tie
    assert f(-(1 + 2 ** -8)) == -1.0
    assert f(3.0) == 3.0 and f(0.0) == 0.0
    assert np.signbit(e4m3.bf16_round(np.float32(-0.0)))
    # power-of-two scaling commutes with the rounding (normal range)
    v = np.random.default_rng(1).standard_normal(1000).astype(np.float32)
    for k in (-20, -3, 5, 40):
        sc = np.float32(2.0 ** k)
        assert np.array_equal(e4m3.bf16_round(v * sc), e4m3.bf16_round(v) * sc)


@pytest.mark.parametrize("rule", [e4m3.RULE_FP32_AMAX, e4m3.RULE_POW2_CEIL, e4m3.RULE_POW2_OCP])
def test_blocks2d_one_row_is_the_row_quantizer(rule):
    x = np.random.default_rng(2).standard_normal((37, 256)).astype(np.float32)
    a = e4m3.quantize_blocks2d(x, 1, 32, rule)
    b = e4m3.quantize_rows(x, 32, rule)
    for u, v in zip(a, b):
        assert np.array_equal(np.asarray(u), np.asarray(v))


@pytest.mark.parametrize("rule", [e4m3.RULE_FP32_AMAX, e4m3.RULE_POW2_CEIL, e4m3.RULE_POW2_OCP])
def test_blocks2d_scale_is_the_block_max_and_codes_follow(rule):
    """One scale per (4 rows x 16) block from the maximum over the whole
    block; every code is the brute-force nearest code of fl32(x / s); a short
    last row block."""
    rng = np.random.default_rng(3)
    x = (rng.standard_normal((10, 48)) * np.exp(rng.uniform(-3, 3, (10, 1)))).astype(np.float32)
    codes, stored, s, deq = e4m3.quantize_blocks2d(x, 4, 16, rule)
    for rb in range(3):
        rows = slice(4 * rb, min(10, 4 * rb + 4))
        for kb in range(3):
            blk = x[rows, 16 * kb:16 * kb + 16]
            amax = np.float32(np.max(np.abs(blk)))
            sb, stb = e4m3.block_scales(np.array([amax]), rule)
            assert np.all(s[rows, kb] == sb[0])
            assert np.all(stored[rows, kb] == stb[0])
            for (i, j), v in np.ndenumerate(blk):
                q = np.float32(v / sb[0])
                assert codes[rows][i, 16 * kb + j] == e4m3.encode_bruteforce(float(q))


POW2_SWEEP_EXPONENTS = (-126, -48, -20, -9, 0, 8, 60, 119, 120, 127)


@pytest.mark.parametrize("e", POW2_SWEEP_EXPONENTS)
def test_c_codec_pow2_matches_numpy_codec(e):
    """The C twin's cast under a power-of-two scale 2^e (the sweep the device
    cast is checked against) equals the numpy codec applied to the binary32
    quotient fl32(x / 2^e): runs of consecutive bit patterns at random
    starts, and runs around every binary32 exponent boundary whose quotient
    lands near the e4m3 range (subnormal quotients, midpoints, 448, overflow
    of the quotient)."""
    lib = oracle_c_lib()
    rng = np.random.default_rng(1000 + e)
    starts = list(rng.integers(0, 2 ** 32 - 4096, size=300))
    for E in range(0, 255):                      # exponent field of x
        q = E - 127 - e                          # exponent of the quotient
        if -12 <= q <= 9 or E in (0, 1, 254):
            for sign in (0, 1):
                starts.append((sign << 31) | (E << 23) | int(rng.integers(0, 2 ** 23 - 4096)))
                starts.append((sign << 31) | (E << 23))
    n = 4096
    for st in starts:
        st = int(st)
        got = np.empty(n, dtype=np.uint8)
        lib.oracle_e4m3_sweep_pow2(st, n, e, got.ctypes.data)
        pat = (np.arange(n, dtype=np.uint64) + st).astype(np.uint32)
        x = pat.view(np.float32)
        fin = np.isfinite(x)
        with np.errstate(over="ignore"):
            quot = (x[fin].astype(np.float64) * 2.0 ** -e).astype(np.float32)
        want = e4m3.encode(quot)
        assert np.array_equal(got[fin], want), (hex(st), e)


def test_c_codec_pow2_saturates_overflowing_quotients():
    lib = oracle_c_lib()
    for e, pat in ((-126, 0x3F800000), (-48, 0x7F7FFFFF), (-9, 0x7F000000), (-1, 0x7F7FFFFF)):
        for sign in (0, 1):
            got = np.empty(1, dtype=np.uint8)
            lib.oracle_e4m3_sweep_pow2((sign << 31) | pat, 1, e, got.ctypes.data)
            assert got[0] == (0xFE if sign else 0x7E), (e, hex(pat))
