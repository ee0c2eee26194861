"""Host-side checks of the ABI's constants and of the tiled code layout.

The tiled layout FMM_LAYOUT_TILE256x64 is rebuilt here from its definition in
include/fmm8.h with plain loops; the binding's row-major reconstruction must
invert it exactly.  No GPU is needed.
"""
import os
import re

import numpy as np
import torch

import paper_2609_26077_amd as fm
from paper_2609_26077_amd.runner import (_unpack_scales128, _unpermute_scales256, _untile128x128,
                                          _untile256x64)

HEADER = os.path.join(os.path.dirname(__file__), "..", "include", "fmm8.h")


def test_header_constants_match_binding():
    text = open(HEADER).read()
    consts = dict((k, int(v)) for k, v in re.findall(r"\b(FMM_[A-Z0-9_x]+)\s*=\s*(-?\d+)", text))
    assert "FMM_LAYOUT_TILE256x64" in consts and "FMM_OK" in consts
    for name, value in consts.items():
        assert getattr(fm, name) == value, name


def _tile_by_definition(codes):
    """[b][T][rows][kdim] -> the byte image of FMM_LAYOUT_TILE256x64."""
    b, T, rows, kdim = codes.shape
    out = np.empty(codes.size, dtype=np.uint8)
    pos = 0
    for bi in range(b):
        for r in range(T):
            for tile in range(rows // 256):
                for ks in range(kdim // 64):
                    img = np.empty((256, 64), dtype=np.uint8)
                    for t in range(256):
                        src = codes[bi, r, 256 * tile + t, 64 * ks:64 * ks + 64]
                        for c in range(4):
                            s = c ^ ((t >> 2) & 3)
                            img[t, 16 * s:16 * s + 16] = src[16 * c:16 * c + 16]
                    out[pos:pos + img.size] = img.ravel()
                    pos += img.size
    return out


def test_untile_inverts_the_documented_layout():
    rng = np.random.default_rng(0)
    codes = rng.integers(0, 256, size=(2, 3, 512, 192), dtype=np.uint8)
    raw = torch.from_numpy(_tile_by_definition(codes))
    back = _untile256x64(raw, 2, 3, 512, 192).numpy()
    assert np.array_equal(back, codes)


def test_unpermute_scales_inverts_the_documented_layout():
    rng = np.random.default_rng(1)
    b, T, rows, kb = 2, 3, 512, 5
    scales = rng.integers(0, 256, size=(b, T, rows, kb), dtype=np.uint8)
    raw = np.empty(scales.size, dtype=np.uint8)
    for bi in range(b):
        for r in range(T):
            for k in range(kb):
                base = ((bi * T + r) * kb + k) * rows
                for p in range(rows):
                    tr = p % 256
                    h, i, j = tr // 128, (tr // 32) % 4, tr % 32
                    raw[base + (p - tr) + 4 * (32 * h + j) + i] = scales[bi, r, p, k]
    back = _unpermute_scales256(torch.from_numpy(raw), b, T, rows, kb).numpy()
    assert np.array_equal(back, scales)


def test_untile128_inverts_the_documented_layout():
    rng = np.random.default_rng(2)
    b, T, rows, kdim = 2, 2, 256, 384
    codes = rng.integers(0, 256, size=(b, T, rows, kdim), dtype=np.uint8)
    raw = np.empty(codes.size, dtype=np.uint8)
    pos = 0
    for bi in range(b):
        for r in range(T):
            for tile in range(rows // 128):
                for ks in range(kdim // 128):
                    img = np.empty((128, 128), dtype=np.uint8)
                    for t in range(128):
                        src = codes[bi, r, 128 * tile + t, 128 * ks:128 * ks + 128]
                        for c in range(8):
                            s = c ^ (t & 7) ^ ((t >> 3) & 1)
                            img[t, 16 * s:16 * s + 16] = src[16 * c:16 * c + 16]
                    raw[pos:pos + img.size] = img.ravel()
                    pos += img.size
    back = _untile128x128(torch.from_numpy(raw), b, T, rows, kdim).numpy()
    assert np.array_equal(back, codes)


def test_unpack_scales128_inverts_the_documented_layout():
    rng = np.random.default_rng(3)
    b, T, rows, kdim = 2, 2, 256, 384
    for block in (16, 32, 128):
        kb = kdim // block
        rec = 8 if block == 16 else 4
        scales = rng.integers(0, 256, size=(b, T, rows, kb), dtype=np.uint8)
        raw = np.empty(b * T * rows * (kdim // 128) * rec, dtype=np.uint8)
        pos = 0
        for bi in range(b):
            for r in range(T):
                for tile in range(rows // 128):
                    for ks in range(kdim // 128):
                        for t in range(128):
                            p = 128 * tile + t
                            if block == 16:
                                record = [scales[bi, r, p, 8 * ks + q] for q in (0, 2, 4, 6, 1, 3, 5, 7)]
                            elif block == 32:
                                record = [scales[bi, r, p, 4 * ks + q] for q in (0, 2, 1, 3)]
                            else:
                                record = [scales[bi, r, p, ks]] * 4
                            raw[pos:pos + rec] = record
                            pos += rec
        back = _unpack_scales128(torch.from_numpy(raw), b, T, rows, kdim, kb).numpy()
        assert np.array_equal(back, scales), block
