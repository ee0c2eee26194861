"""The device e4m3 casts against the oracle's codec over every finite float32.

All 2^32 bit patterns are generated on the device in chunks and compared byte
for byte with the plain-C oracle codec, which runs on host threads (ctypes
releases the GIL):
* fmm_e4m3_quantize, the cast the fp32 amax/448 rule applies after dividing
  by the block scale;
* fmm_e4m3_quantize_pow2 at exponents spanning the power-of-two rules' range
  and the entry point's limits, the cast every E8M0-scaled block goes through
  (the scaled convert with the clamp at 448 2^e), against the oracle's code of
  the binary32 quotient fl32(x / 2^e).
NaN and infinity inputs are undefined behaviour and are excluded.
"""
import sys
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

from tests.test_oracle_codec import POW2_SWEEP_EXPONENTS, oracle_c_lib

pytestmark = pytest.mark.gpu

CHUNK = 1 << 28


def _host_codes(lib, start, n, out, e=None):
    nthreads = 16
    per = n // nthreads

    def work(i):
        s = start + i * per
        view = out[i * per:(i + 1) * per]
        if e is None:
            lib.oracle_e4m3_sweep(s, per, view.ctypes.data)
        else:
            lib.oracle_e4m3_sweep_pow2(s, per, e, view.ctypes.data)
    with ThreadPoolExecutor(nthreads) as ex:
        list(ex.map(work, range(nthreads)))


def test_codec_all_float32_patterns():
    _sweep(None)


@pytest.mark.parametrize("e", POW2_SWEEP_EXPONENTS)
def test_pow2_codec_all_float32_patterns(e):
    _sweep(e)


def _sweep(e):
    import torch
    import paper_2609_26077_amd as fm
    lib = oracle_c_lib()
    dev = torch.device("cuda:0")
    host = np.empty(CHUNK, dtype=np.uint8)
    out = torch.empty(CHUNK, dtype=torch.uint8, device=dev)
    total_bad = 0
    for c in range(1 << 32 >> 28):
        start = c * CHUNK
        idx = torch.arange(CHUNK, dtype=torch.int64, device=dev) + start   # patterns
        x = torch.where(idx >= 2 ** 31, idx - 2 ** 32, idx).to(torch.int32).view(torch.float32)
        if e is None:
            fm.fmm_e4m3_quantize(x, out, CHUNK)
        else:
            fm.fmm_e4m3_quantize_pow2(x, out, CHUNK, e)
        got = out.cpu().numpy()
        _host_codes(lib, start, CHUNK, host, e)
        pat = np.arange(start, start + CHUNK, dtype=np.uint32)
        finite = (pat & 0x7F800000) != 0x7F800000
        bad = np.nonzero((got != host) & finite)[0]
        if bad.size:
            i = bad[0]
            print(f"e={e} chunk {c}: {bad.size} mismatches, first pattern {int(pat[i]):#010x} "
                  f"device {got[i]:#04x} oracle {host[i]:#04x}", flush=True)
        total_bad += bad.size
        print(f"codec e={e} chunk {c + 1}/16 done", flush=True)
        del idx, x
    assert total_bad == 0


def test_codec_edges_and_tails():
    """Lengths that are not a multiple of four, and n = 0."""
    import torch
    import paper_2609_26077_amd as fm
    from oracle import e4m3
    rng = np.random.default_rng(0)
    for n in (0, 1, 2, 3, 5, 7, 1025):
        v = (rng.standard_normal(n) * 300).astype(np.float32)
        x = torch.from_numpy(v).cuda()
        out = torch.full((max(n, 4),), 0xAB, dtype=torch.uint8, device="cuda:0")
        fm.fmm_e4m3_quantize(x, out, n)
        got = out.cpu().numpy()
        assert np.array_equal(got[:n], e4m3.encode(v))
        assert np.all(got[n:] == 0xAB)            # nothing written past n


def test_pow2_codec_edges_and_tails():
    """The scaled cast on lengths that are not a multiple of four and n = 0,
    and its argument checks."""
    import torch
    import paper_2609_26077_amd as fm
    from oracle import e4m3
    rng = np.random.default_rng(1)
    for e in (-20, 0, 7):
        for n in (0, 1, 2, 3, 5, 7, 1025):
            v = (rng.standard_normal(n) * 300 * 2.0 ** e).astype(np.float32)
            x = torch.from_numpy(v).cuda()
            out = torch.full((max(n, 4),), 0xAB, dtype=torch.uint8, device="cuda:0")
            fm.fmm_e4m3_quantize_pow2(x, out, n, e)
            got = out.cpu().numpy()
            assert np.array_equal(got[:n], e4m3.encode((v.astype(np.float64) * 2.0 ** -e).astype(np.float32)))
            assert np.all(got[n:] == 0xAB)
    x = torch.zeros(4, dtype=torch.float32, device="cuda:0")
    out = torch.zeros(4, dtype=torch.uint8, device="cuda:0")
    for bad_e in (-127, 128):
        with pytest.raises(fm.FmmError):
            fm.fmm_e4m3_quantize_pow2(x, out, 4, bad_e)
