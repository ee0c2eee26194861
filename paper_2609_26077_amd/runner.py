"""Convenience wrappers over the C-ABI with torch-owned device buffers.

Allocation and marshalling only: the arithmetic of every call happens in the
library's HIP kernels.
"""
from __future__ import annotations

import numpy as np
import torch

from . import (FMM_LAYOUT_TILE128x128, FMM_LAYOUT_TILE256x64, Realization, fmm_combine, fmm_encode, fmm_error_stats,
               fmm_error_stats_scratch_size, fmm_matmul, fmm_multiply, fmm_operand_views,
               fmm_plan_create, fmm_products, fmm_encode_noise, fmm_encode_noise_scratch_size,
               fmm_plan_workspace_size, fmm_realization_builtin, fmm_reference_f64, make_desc)


def _require(x, name, shape, dtype, device):
    """Raise ValueError unless x is a contiguous torch tensor of exactly this
    shape and dtype on this device: the kernels index with the plan's sizes,
    so any other buffer would be read or written out of bounds."""
    if not isinstance(x, torch.Tensor):
        raise ValueError(f"{name}: expected a torch.Tensor, got {type(x).__name__}")
    if x.dtype != dtype:
        raise ValueError(f"{name}: dtype {x.dtype}, expected {dtype}")
    if tuple(x.shape) != tuple(shape):
        raise ValueError(f"{name}: shape {tuple(x.shape)}, expected {tuple(shape)}")
    if not x.is_contiguous():
        raise ValueError(f"{name}: not contiguous")
    if x.device != device:
        raise ValueError(f"{name}: on {x.device}, expected {device}")


class FMM:
    """One planned product shape on one device, with its own workspace.
    Every call checks its tensors (float32, contiguous, on the plan's device,
    exactly the plan's shapes) before anything reaches the library."""

    def __init__(self, realization, batch, M, K, N, depth=1, block=32, rule="pow2_ceil",
                 device="cuda:0", exact_dot=False, flags=0):
        if not isinstance(realization, Realization):
            realization = fmm_realization_builtin(realization)
        self.real = realization
        self.device = torch.device(device)
        if self.device.type == "cuda" and self.device.index is None:
            self.device = torch.device("cuda", torch.cuda.current_device())
        self.shape = (int(batch), int(M), int(K), int(N))
        self.depth, self.block = int(depth), int(block)
        with torch.cuda.device(self.device):
            desc = make_desc(batch, M, K, N, depth, block, rule, exact_dot=exact_dot)
            desc.flags |= int(flags)
            self.plan = fmm_plan_create(realization, desc)
            nbytes = fmm_plan_workspace_size(self.plan)
            self.ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=self.device)
        self.scale_bytes = 4 if (rule in ("fp32_amax", 0)) else 1

    def _inputs(self, A, B):
        b, M, K, N = self.shape
        _require(A, "A", (b, M, K), torch.float32, self.device)
        _require(B, "B", (b, K, N), torch.float32, self.device)

    def _output(self, C):
        b, M, K, N = self.shape
        if C is None:
            return torch.empty((b, M, N), dtype=torch.float32, device=self.device)
        _require(C, "C", (b, M, N), torch.float32, self.device)
        return C

    def matmul(self, A, B, C=None, stream=None):
        self._inputs(A, B)
        C = self._output(C)
        fmm_matmul(self.plan, A, B, C, self.ws, stream)
        return C

    def encode(self, A, B, stream=None):
        self._inputs(A, B)
        fmm_encode(self.plan, A, B, self.ws, stream)

    def multiply(self, C=None, stream=None):
        C = self._output(C)
        fmm_multiply(self.plan, self.ws, C, stream)
        return C

    def products(self, C=None, stream=None):
        """First half of multiply (the sub-products); returns C, which it may or may not have written."""
        C = self._output(C)
        fmm_products(self.plan, self.ws, C, stream)
        return C

    def combine(self, C, stream=None):
        """Second half of multiply (the rest of the W-combine); writes C."""
        C = self._output(C)
        fmm_combine(self.plan, self.ws, C, stream)
        return C

    def encode_noise(self, A, B, stream=None):
        """Operand-side rounding energy of the encoding in the workspace (call
        after encode with the same A, B): numpy [batch][2 sides][T][2] of
        (sum (xhat - x)^2, sum x^2) per batch element, side and term."""
        self._inputs(A, B)
        batch, T = self.shape[0], None
        from . import fmm_realization_terms
        _, T = fmm_realization_terms(self.real, self.depth)
        out = torch.empty((batch, 2, T, 2), dtype=torch.float64, device=self.device)
        nbytes = fmm_encode_noise_scratch_size(self.plan)
        scratch = torch.empty(max(nbytes, 8), dtype=torch.uint8, device=self.device)
        fmm_encode_noise(self.plan, A, B, self.ws, out, scratch, nbytes, stream)
        return out.cpu().numpy()

    def cross_terms(self, A, B, stream=None):
        """The cross-term diagnostic of the encoding in the workspace (call
        after encode with the same A, B; depth 1): numpy [batch][2] of
        (|L|^2, diag) per batch element (include/fmm8.h, fmm_cross_terms)."""
        self._inputs(A, B)
        from . import fmm_cross_terms, fmm_cross_terms_scratch_size
        out = torch.empty((self.shape[0], 2), dtype=torch.float64, device=self.device)
        nbytes = fmm_cross_terms_scratch_size(self.plan)
        scratch = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=self.device)
        fmm_cross_terms(self.plan, A, B, self.ws, out, scratch, nbytes, stream)
        return out.cpu().numpy()

    def operands(self):
        """(a_codes, a_scales, b_codes, b_scales) as [batch][terms][rows][kdim]
        and [batch][terms][rows][kblocks] tensors: views of the workspace, or
        row-major copies where the plan keeps them in the tiled layout."""
        a, b = fmm_operand_views(self.plan, self.ws)
        base = self.ws.data_ptr()
        out = []
        for v in (a, b):
            nc = v.batch * v.terms * v.rows * v.kdim
            ns = v.batch * v.terms * v.rows * v.kblocks
            c0 = v.codes - base
            s0 = v.scales - base
            raw = self.ws[c0:c0 + nc]
            if v.code_layout == FMM_LAYOUT_TILE256x64:
                codes = _untile256x64(raw, v.batch, v.terms, v.rows, v.kdim)
                if v.scale_bytes == 4:
                    scales = (self.ws[s0:s0 + 4 * ns].view(torch.float32)
                              .view(v.batch, v.terms, v.kblocks, v.rows).permute(0, 1, 3, 2).contiguous())
                else:
                    scales = _unpermute_scales256(self.ws[s0:s0 + ns], v.batch, v.terms, v.rows, v.kblocks)
            elif v.code_layout == FMM_LAYOUT_TILE128x128:
                codes = _untile128x128(raw, v.batch, v.terms, v.rows, v.kdim)
                nrec = v.batch * v.terms * v.rows * (v.kdim // 128) * (8 if v.kblocks == v.kdim // 16 else 4)
                scales = _unpack_scales128(self.ws[s0:s0 + nrec], v.batch, v.terms, v.rows, v.kdim,
                                           v.kblocks)
            else:
                codes = raw.view(v.batch, v.terms, v.rows, v.kdim)
                sraw = self.ws[s0:s0 + ns * v.scale_bytes]
                if v.scale_bytes == 4:
                    scales = sraw.view(torch.float32).view(v.batch, v.terms, v.rows, v.kblocks)
                else:
                    scales = sraw.view(v.batch, v.terms, v.rows, v.kblocks)
            out += [codes, scales]
        return tuple(out)


def _untile256x64(raw, batch, terms, rows, kdim):
    """Row-major copy of codes in FMM_LAYOUT_TILE256x64 (see include/fmm8.h)."""
    t = raw.view(batch, terms, rows // 256, kdim // 64, 256, 4, 16)
    row = torch.arange(256, device=raw.device)[:, None]
    chunk = torch.arange(4, device=raw.device)[None, :]
    t = t[:, :, :, :, row, chunk ^ ((row >> 2) & 3), :]      # logical chunk c of tile row
    return t.permute(0, 1, 2, 4, 3, 5, 6).reshape(batch, terms, rows, kdim)


def _untile128x128(raw, batch, terms, rows, kdim):
    """Row-major copy of codes in FMM_LAYOUT_TILE128x128 (see include/fmm8.h)."""
    t = raw.view(batch, terms, rows // 128, kdim // 128, 128, 8, 16)
    row = torch.arange(128, device=raw.device)[:, None]
    chunk = torch.arange(8, device=raw.device)[None, :]
    t = t[:, :, :, :, row, chunk ^ (row & 7) ^ ((row >> 3) & 1), :]
    return t.permute(0, 1, 2, 4, 3, 5, 6).reshape(batch, terms, rows, kdim)


def _unpack_scales128(raw, batch, terms, rows, kdim, kblocks):
    """[batch][terms][rows][kblocks] copy of E8M0 scales in FMM_LAYOUT_TILE128x128."""
    if kblocks == kdim // 16:                  # block 16: record order is blocks 0, 2, 4, 6, 1, 3, 5, 7
        t = raw.view(batch, terms, rows // 128, kdim // 128, 128, 8)
        t = t[..., torch.tensor([0, 4, 1, 5, 2, 6, 3, 7], device=raw.device)]
    else:
        t = raw.view(batch, terms, rows // 128, kdim // 128, 128, 4)
        if kblocks == kdim // 32:              # block 32: record order is blocks 0, 2, 1, 3
            t = t[..., torch.tensor([0, 2, 1, 3], device=raw.device)]
        else:                                  # block 128: the byte repeated
            t = t[..., :1]
    return t.permute(0, 1, 2, 4, 3, 5).reshape(batch, terms, rows, kblocks)


def _unpermute_scales256(raw, batch, terms, rows, kblocks):
    """[batch][terms][rows][kblocks] copy of scales in FMM_LAYOUT_TILE256x64."""
    t = raw.view(batch, terms, kblocks, rows // 256, 256)
    r = torch.arange(256, device=raw.device)
    stored = (((r >> 7) * 32 + (r & 31)) * 4 + ((r >> 5) & 3))     # where tile row r sits
    t = t[..., stored]
    return t.reshape(batch, terms, kblocks, rows).permute(0, 1, 3, 2).contiguous()


def reference_f64(A, B, stream=None):
    b, M, K = A.shape
    N = B.shape[2]
    _require(A, "A", (b, M, K), torch.float32, A.device)
    _require(B, "B", (b, K, N), torch.float32, A.device)
    Cref = torch.empty((b, M, N), dtype=torch.float64, device=A.device)
    fmm_reference_f64(b, M, K, N, A, B, Cref, stream)
    return Cref


def error_stats(C, Cref, stream=None):
    """(err2, ref2) per product as numpy float64 arrays (one host sync)."""
    b, M, N = C.shape
    _require(C, "C", (b, M, N), torch.float32, C.device)
    _require(Cref, "Cref", (b, M, N), torch.float64, C.device)
    nbytes = fmm_error_stats_scratch_size(b, M, N)
    scratch = torch.empty(max(nbytes, 8), dtype=torch.uint8, device=C.device)
    out = torch.empty((b, 2), dtype=torch.float64, device=C.device)
    fmm_error_stats(b, M, N, C, Cref, out, scratch, nbytes, stream)
    o = out.cpu().numpy()
    return o[:, 0].copy(), o[:, 1].copy()
