"""The torch wrappers refuse buffers the plan's kernels would index out of
bounds (wrong dtype, shape, layout or device) before any library call.  CPU
only: the plan object below has no device state, and every check fires
before the C-ABI is reached."""
import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2609_26077_amd", "libfmm8.so")
pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libfmm8.so not built")


def _fake_plan(batch, M, K, N, device):
    import torch
    from paper_2609_26077_amd.runner import FMM
    f = FMM.__new__(FMM)
    f.shape = (batch, M, K, N)
    f.device = torch.device(device)
    f.plan = None          # any call that got past the checks would fail in ctypes
    f.ws = None
    return f


def test_wrong_inputs_are_refused_before_the_library():
    import torch
    f = _fake_plan(2, 8, 16, 4, "cpu")
    A = torch.zeros((2, 8, 16), dtype=torch.float32)
    B = torch.zeros((2, 16, 4), dtype=torch.float32)
    C = torch.zeros((2, 8, 4), dtype=torch.float32)
    bad = [
        ((A.half(), B), "dtype"),
        ((A, B.double()), "dtype"),
        ((A[:, :, :8], B), "shape"),
        ((A, torch.zeros((2, 16, 5))), "shape"),
        ((torch.zeros((2, 16, 8)).transpose(1, 2), B), "contiguous"),
        ((A, B[:1]), "shape"),
        (("not a tensor", B), "torch.Tensor"),
    ]
    for (a, b), what in bad:
        for call in (lambda: f.matmul(a, b), lambda: f.encode(a, b), lambda: f.encode_noise(a, b)):
            with pytest.raises(ValueError, match=what):
                call()
    for c, what in ((C.double(), "dtype"), (C[:, :4], "shape"), (C.transpose(1, 2), "shape"),
                    (torch.zeros((2, 4, 8)).transpose(1, 2), "contiguous")):
        for call in (lambda: f.matmul(A, B, c), lambda: f.multiply(c), lambda: f.products(c),
                     lambda: f.combine(c)):
            with pytest.raises(ValueError, match=what):
                call()


def test_device_mismatch_is_refused():
    import torch
    f = _fake_plan(1, 4, 4, 4, "cuda:0")
    A = torch.zeros((1, 4, 4), dtype=torch.float32)           # host tensors
    with pytest.raises(ValueError, match="expected cuda:0"):
        f.matmul(A, A)


def test_measurement_wrappers_check_their_buffers():
    import torch
    from paper_2609_26077_amd.runner import error_stats, reference_f64
    A = torch.zeros((1, 4, 6), dtype=torch.float32)
    with pytest.raises(ValueError, match="dtype"):
        reference_f64(A, torch.zeros((1, 6, 3), dtype=torch.float64))
    with pytest.raises(ValueError, match="shape"):
        reference_f64(A, torch.zeros((1, 5, 3), dtype=torch.float32))
    C = torch.zeros((1, 4, 3), dtype=torch.float32)
    with pytest.raises(ValueError, match="dtype"):
        error_stats(C, torch.zeros((1, 4, 3), dtype=torch.float32))
    with pytest.raises(ValueError, match="shape"):
        error_stats(C, torch.zeros((1, 3, 4), dtype=torch.float64))
