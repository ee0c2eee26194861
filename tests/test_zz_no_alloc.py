"""The allocation-free error reduction against the one with a caller scratch.

fmm_error_stats_noalloc keeps the reduction's partials in a static device
array of the library instead of a caller workspace.  Through the C-ABI, on
two calls in a row (the second with a smaller input, so that it runs over
what the first left in the array), its sums must equal fmm_error_stats's
bit for bit (the same kernels in the same fixed order), and both must agree
with numpy's binary64 sums.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def _case(fm, torch, batch, M, N, seed):
    rng = np.random.default_rng(seed)
    C = torch.from_numpy(rng.standard_normal((batch, M, N)).astype(np.float32)).cuda()
    Cref = torch.from_numpy(rng.standard_normal((batch, M, N))).cuda()
    nbytes = fm.fmm_error_stats_scratch_size(batch, M, N)
    scratch = torch.empty(max(nbytes, 8), dtype=torch.uint8, device="cuda:0")
    want = torch.empty((batch, 2), dtype=torch.float64, device="cuda:0")
    fm.fmm_error_stats(batch, M, N, C, Cref, want, scratch, nbytes)
    got = torch.full((batch, 2), float("nan"), dtype=torch.float64, device="cuda:0")
    fm.fmm_error_stats_noalloc(batch, M, N, C, Cref, got)
    torch.cuda.synchronize()
    w, g = want.cpu().numpy(), got.cpu().numpy()
    assert np.array_equal(g.view(np.uint64), w.view(np.uint64)), (g, w)
    c64, r64 = C.cpu().numpy().astype(np.float64), Cref.cpu().numpy()
    e2 = ((c64 - r64) ** 2).reshape(batch, -1).sum(axis=1)
    r2 = (r64 ** 2).reshape(batch, -1).sum(axis=1)
    assert np.allclose(g[:, 0], e2, rtol=1e-12) and np.allclose(g[:, 1], r2, rtol=1e-12)


def test_noalloc_matches_scratch_form_twice():
    import torch
    import paper_2609_26077_amd as fm
    print("noalloc: batch 7 x 300 x 257, then batch 3 x 65 x 33", flush=True)
    _case(fm, torch, 7, 300, 257, seed=1)
    _case(fm, torch, 3, 65, 33, seed=2)


def test_noalloc_largest_batch_then_small():
    import torch
    import paper_2609_26077_amd as fm
    print("noalloc: the largest batch, 1024 x 64 x 48, then 2 x 16 x 16", flush=True)
    _case(fm, torch, fm.FMM_ERROR_STATS_NOALLOC_MAX_BATCH, 64, 48, seed=3)
    _case(fm, torch, 2, 16, 16, seed=4)


def test_noalloc_rejects_oversized_batch():
    import torch
    import paper_2609_26077_amd as fm
    n = fm.FMM_ERROR_STATS_NOALLOC_MAX_BATCH + 1
    out = torch.zeros((n, 2), dtype=torch.float64, device="cuda:0")
    C = torch.zeros((n, 1, 1), dtype=torch.float32, device="cuda:0")
    Cref = torch.zeros((n, 1, 1), dtype=torch.float64, device="cuda:0")
    with pytest.raises(fm.FmmError) as ei:
        fm.fmm_error_stats_noalloc(n, 1, 1, C, Cref, out)
    assert ei.value.status == fm.FMM_ERR_WORKSPACE
    assert "exceeds the static scratch" in str(ei.value)
