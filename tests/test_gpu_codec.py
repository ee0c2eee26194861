"""The device e4m3 cast against the oracle's codec over every finite float32.

All 2^32 bit patterns are generated on the device in chunks, quantized by
fmm_e4m3_quantize (the same device routine the encoder uses after dividing by
the block scale), and compared byte for byte with the plain-C oracle codec,
which runs on host threads (ctypes releases the GIL).  NaN and infinity
inputs are undefined behaviour and are excluded.
"""
import sys
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

from tests.test_oracle_codec import oracle_c_lib

pytestmark = pytest.mark.gpu

CHUNK = 1 << 28


def _host_codes(lib, start, n, out):
    nthreads = 16
    per = n // nthreads

    def work(i):
        s = start + i * per
        view = out[i * per:(i + 1) * per]
        lib.oracle_e4m3_sweep(s, per, view.ctypes.data)
    with ThreadPoolExecutor(nthreads) as ex:
        list(ex.map(work, range(nthreads)))


def test_codec_all_float32_patterns():
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
        fm.fmm_e4m3_quantize(x, out, CHUNK)
        got = out.cpu().numpy()
        _host_codes(lib, start, CHUNK, host)
        pat = np.arange(start, start + CHUNK, dtype=np.uint32)
        finite = (pat & 0x7F800000) != 0x7F800000
        bad = np.nonzero((got != host) & finite)[0]
        if bad.size:
            i = bad[0]
            print(f"chunk {c}: {bad.size} mismatches, first pattern {int(pat[i]):#010x} "
                  f"device {got[i]:#04x} oracle {host[i]:#04x}", flush=True)
        total_bad += bad.size
        print(f"codec chunk {c + 1}/16 done", flush=True)
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
