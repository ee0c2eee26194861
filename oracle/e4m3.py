"""OCP E4M3 codec and block-scale rules (oracle; test infrastructure only).

Format (the OCP 8-bit floating-point specification the paper cites for
e4m3, Section 2.2; maximum 448 as used in Appendix D and E.2): sign bit,
4 exponent bits with bias 7, 3 mantissa bits.  Exponent field 0 encodes the
subnormals m * 2^-9 (m = 0..7); fields 1..15 encode (1 + m/8) * 2^(E-7),
except that field 15 with m = 7 (codes 0x7F / 0xFF) is NaN, so the largest
finite magnitude is 1.75 * 2^8 = 448.  There is no infinity.

Quantization of one block (Appendix E.2: a block's scale is its absolute
maximum over 448 kept in fp32, the scaled block is cast to e4m3 with
round-to-nearest-even).  Readings where the paper is silent:

* the cast rounds |v| to the nearest representable magnitude, ties to the
  even mantissa code, then saturates to 448; it never yields NaN;
* the sign is kept, so a negative value that rounds to zero encodes 0x80;
* before the scale is formed the block maximum is clamped from below at
  fl32(1e-12) (the "minimum-scale clamp" of Appendix E.2 engages when a
  block's absolute maximum falls below 1e-12);
* the scaled value is the IEEE binary32 quotient fl32(x / s), then cast;
* power-of-two scale rules (the benchmark configurations ask for
  power-of-two scales): POW2_CEIL takes the smallest integer e with
  a <= 448 * 2^e (no clipping); POW2_OCP takes e = floor(log2 a) - 8 (the OCP
  microscaling rule, which clips the top of the block to 448).  Their scales
  are stored as E8M0 bytes e + 127.
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np

E4M3_MAX = 448.0
CLAMP = np.float32(1e-12)           # fl32(1e-12)

RULE_FP32_AMAX = 0
RULE_POW2_CEIL = 1
RULE_POW2_OCP = 2
RULES = {"fp32_amax": RULE_FP32_AMAX, "pow2_ceil": RULE_POW2_CEIL,
         "pow2_ocp": RULE_POW2_OCP}


# ---------------------------------------------------------------------------
# Decoding: the value of every code, exactly
# ---------------------------------------------------------------------------

def code_value_exact(code: int):
    """Exact value of an e4m3 code as a Fraction (None for NaN)."""
    s = -1 if code & 0x80 else 1
    E = (code >> 3) & 0xF
    m = code & 0x7
    if E == 15 and m == 7:
        return None
    if E == 0:
        return s * Fraction(m, 8) * Fraction(1, 2 ** 6)
    return s * (1 + Fraction(m, 8)) * (Fraction(2) ** (E - 7))


def decode_table() -> np.ndarray:
    """float64 value of all 256 codes (NaN codes map to nan)."""
    t = np.empty(256, dtype=np.float64)
    for c in range(256):
        v = code_value_exact(c)
        # Fractions carry no signed zero; code 0x80 decodes to -0.0
        t[c] = np.nan if v is None else np.copysign(float(v), -1.0 if c & 0x80 else 1.0)
    return t


DECODE = decode_table()


# ---------------------------------------------------------------------------
# Encoding, brute force (the definition, for tiny inputs)
# ---------------------------------------------------------------------------

def encode_bruteforce(v: float) -> int:
    """Nearest finite code to the real value of ``v`` by exhaustive search over
    all 254 finite codes in exact rational arithmetic.  Ties go to the code
    with the even mantissa field; a tie between +0 and -0 cannot arise because
    the sign is taken from v.  Magnitudes above 448 saturate to 448."""
    x = Fraction(float(v))
    neg = np.signbit(np.float64(v))
    best, best_d = None, None
    for c in range(128):               # magnitudes only
        cv = code_value_exact(c)
        if cv is None:
            continue
        d = abs(abs(x) - cv)
        if best is None or d < best_d or (d == best_d and (c & 1) == 0 and (best & 1) == 1):
            best, best_d = c, d
    return best | (0x80 if neg else 0)


# ---------------------------------------------------------------------------
# Encoding, vectorised (every step exact in binary64)
# ---------------------------------------------------------------------------

def encode(v) -> np.ndarray:
    """e4m3 codes of the float32 array ``v`` (round to nearest even, saturate).

    For |v| > 0 let e = max(floor(log2 |v|), -6); the representable
    magnitudes in [2^e, 2^(e+1)) (or below 2^-6 for the subnormals) are the
    multiples of q = 2^(e-3).  |v|/q is exact in binary64; numpy's rint
    rounds half to even, and the parity of that integer is the parity of
    the mantissa field.  The result is then clamped to 448.
    """
    v = np.asarray(v, dtype=np.float32)
    a = np.abs(v.astype(np.float64))
    neg = np.signbit(v)
    _, ex = np.frexp(a)                 # a = f 2^ex, f in [0.5, 1)
    e = np.maximum(ex - 1, -6)
    q = np.ldexp(1.0, e - 3)
    mag = np.rint(a / q) * q
    mag = np.minimum(mag, E4M3_MAX)
    # code of the magnitude
    _, ex2 = np.frexp(mag)
    E2 = ex2 - 1
    sub = mag < 2.0 ** -6
    man_sub = np.rint(mag / 2.0 ** -9)
    frac = np.where(sub, 0.0, mag / np.ldexp(1.0, np.where(sub, 0, E2)))
    man_norm = np.rint((frac - 1.0) * 8.0)
    exp_field = np.where(sub, 0, E2 + 7)
    man = np.where(sub, man_sub, man_norm)
    code = (exp_field.astype(np.int64) << 3) | man.astype(np.int64)
    code = code | np.where(neg, 0x80, 0)
    return code.astype(np.uint8)


def decode(codes) -> np.ndarray:
    return DECODE[np.asarray(codes, dtype=np.uint8)]


# ---------------------------------------------------------------------------
# Block scales
# ---------------------------------------------------------------------------

def pow2_ceil_exponent(a) -> np.ndarray:
    """Smallest integer e with a <= 448 * 2^e, for float32 a > 0.

    With E = floor(log2 a), 448 * 2^(E-9) = 0.875 * 2^E < a and
    448 * 2^(E-7) = 3.5 * 2^E > a, so e is E-8 or E-7; the comparison below
    is exact in binary64.
    """
    a = np.asarray(a, dtype=np.float64)
    _, ex = np.frexp(a)
    E = ex - 1
    e = E - 8
    return np.where(a <= E4M3_MAX * np.ldexp(1.0, e), e, e + 1).astype(np.int64)


def pow2_ocp_exponent(a) -> np.ndarray:
    """e = floor(log2 a) - 8 for float32 a > 0."""
    _, ex = np.frexp(np.asarray(a, dtype=np.float64))
    return (ex - 1 - 8).astype(np.int64)


def block_scales(amax, rule: int):
    """Scale of every block from its float32 absolute maximum.

    Returns (s, stored): s the float32 scale actually divided by, and the
    stored form -- float32 for FP32_AMAX, uint8 E8M0 (e + 127) otherwise.
    """
    a = np.maximum(np.asarray(amax, dtype=np.float32), CLAMP)
    if rule == RULE_FP32_AMAX:
        s = (a / np.float32(E4M3_MAX)).astype(np.float32)   # one fp32 division
        return s, s
    if rule == RULE_POW2_CEIL:
        e = pow2_ceil_exponent(a)
    elif rule == RULE_POW2_OCP:
        e = pow2_ocp_exponent(a)
    else:
        raise ValueError(f"unknown scale rule {rule}")
    s = np.ldexp(np.float32(1.0), e.astype(np.int32)).astype(np.float32)
    return s, (e + 127).astype(np.uint8)


def quantize_rows(x, bs: int, rule: int):
    """Quantize a float32 matrix whose blocks run along its last axis.

    x has shape (rows, kdim) with kdim a multiple of bs.  Returns
    (codes uint8 (rows, kdim), stored scales (rows, kdim/bs),
    float32 scales (rows, kdim/bs), dequantized float64 (rows, kdim)).
    """
    x = np.asarray(x, dtype=np.float32)
    rows, kdim = x.shape
    if kdim % bs:
        raise ValueError("block size does not divide the contracted length")
    xb = x.reshape(rows, kdim // bs, bs)
    amax = np.max(np.abs(xb), axis=2)
    s, stored = block_scales(amax, rule)
    v = (xb / s[:, :, None]).astype(np.float32)            # fl32(x / s)
    codes = encode(v).reshape(rows, kdim)
    deq = (decode(codes).reshape(rows, kdim // bs, bs)
           * s[:, :, None].astype(np.float64)).reshape(rows, kdim)
    return codes, stored, s, deq


# ---------------------------------------------------------------------------
# Deployment-granularity pieces (Appendix E, weight-scale granularity):
# bfloat16 pre-rounding of an encoded weight combination, and block scales
# shared by a run of rows as well as a run of the contracted axis.
# ---------------------------------------------------------------------------

def bf16_round(x) -> np.ndarray:
    """float32 values rounded to the nearest bfloat16 value (8 significant
    bits, the float32 exponent range), ties to the even mantissa; returned
    as float32.  For x != 0 let e = max(floor(log2 |x|), -126); the
    bfloat16 values in [2^e, 2^(e+1)) (or below 2^-126, the subnormals) are
    the multiples of q = 2^(e-7).  |x|/q is exact in binary64 and numpy's
    rint rounds half to even; a result of 2^128 overflows to infinity."""
    x = np.asarray(x, dtype=np.float32)
    a = np.abs(x.astype(np.float64))
    _, ex = np.frexp(a)
    e = np.maximum(ex - 1, -126)
    q = np.ldexp(1.0, e - 7)
    with np.errstate(over="ignore"):
        r = (np.rint(a / q) * q).astype(np.float32)
    return np.where(np.signbit(x), -r, r).astype(np.float32)


def quantize_blocks2d(x, row_block: int, bs: int, rule: int):
    """Quantize a float32 matrix with one scale per block of row_block rows x
    bs consecutive positions of the last axis (the last row block may be
    short): the block maximum is taken over the whole 2-D block.  Returns the
    same tuple as quantize_rows, the stored scales replicated over the rows of
    each block: (codes (rows, kdim), stored (rows, kdim/bs), s (rows, kdim/bs),
    dequantized float64)."""
    x = np.asarray(x, dtype=np.float32)
    rows, kdim = x.shape
    if kdim % bs:
        raise ValueError("block size does not divide the contracted length")
    nrb = -(-rows // row_block)
    amax_rows = np.max(np.abs(x.reshape(rows, kdim // bs, bs)), axis=2)   # (rows, kdim/bs)
    amax = np.empty_like(amax_rows)
    for i in range(nrb):
        sl = slice(i * row_block, min(rows, (i + 1) * row_block))
        amax[sl] = np.max(amax_rows[sl], axis=0, keepdims=True)
    s, stored = block_scales(amax, rule)
    xb = x.reshape(rows, kdim // bs, bs)
    v = (xb / s[:, :, None]).astype(np.float32)
    codes = encode(v).reshape(rows, kdim)
    deq = (decode(codes).reshape(rows, kdim // bs, bs)
           * s[:, :, None].astype(np.float64)).reshape(rows, kdim)
    return codes, stored, s, deq
