"""Python binding of libfmm8 (the C-ABI declared in include/fmm8.h).

Argument marshalling only: every function below has the name of the C entry
point it calls and forwards plain pointers and sizes.  Device memory and
streams come from PyTorch (``torch.Tensor.data_ptr()``,
``torch.cuda.Stream.cuda_stream``); every computation runs in the library's
HIP kernels.  Importing this module loads the library and fails loudly if it
has not been built (run ``python paper_2609_26077_amd/_build.py``).
"""
from __future__ import annotations

import ctypes
import os
import sys

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfmm8.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is missing: the HIP library has not been built "
        f"(python {os.path.join(_HERE, '_build.py')})")

# The library's device calls take torch's device pointers and streams, so
# it must bind to the HIP runtime torch uses.  torch ships its own
# libamdhip64; importing torch first maps that runtime, and the library's
# libamdhip64.so.7 dependency then resolves to it (loaded the other way
# round, the process would hold two runtimes and the library could not see
# torch's allocations, or the device at all).
try:
    import torch as _torch  # noqa: F401
except ImportError:         # host-only use of the realization calls
    _torch = None

_lib = ctypes.CDLL(LIB_PATH)

# ---- constants (mirror include/fmm8.h) -------------------------------------
FMM_OK = 0
FMM_ERR_ARG = -1
FMM_ERR_SHAPE = -2
FMM_ERR_UNSUPPORTED = -3
FMM_ERR_NOT_EXACT = -4
FMM_ERR_SINGULAR = -5
FMM_ERR_HIP = -6
FMM_ERR_DEVICE = -7
FMM_ERR_WORKSPACE = -8
FMM_ERR_NOMEM = -9

FMM_CUBIC8 = 0
FMM_STRASSEN = 1
FMM_WINOGRAD = 2
FMM_TSTAR = 3
BUILTINS = {"cubic8": FMM_CUBIC8, "strassen": FMM_STRASSEN, "winograd": FMM_WINOGRAD,
            "tstar": FMM_TSTAR}

FMM_FLAG_EXACT_DOT = 1
FMM_FLAG_B_BLOCK128 = 2
FMM_FLAG_B_BF16 = 4
FMM_FLAG_LARGE_TILE = 8
FMM_LAYOUT_ROWS = 0
FMM_LAYOUT_TILE256x64 = 1
FMM_LAYOUT_TILE128x128 = 2

FMM_RULE_FP32_AMAX = 0
FMM_RULE_POW2_CEIL = 1
FMM_RULE_POW2_OCP = 2
RULES = {"fp32_amax": FMM_RULE_FP32_AMAX, "pow2_ceil": FMM_RULE_POW2_CEIL,
         "pow2_ocp": FMM_RULE_POW2_OCP}

_vp = ctypes.c_void_p
_i64 = ctypes.c_int64
_dp = ctypes.POINTER(ctypes.c_double)
_fp = ctypes.POINTER(ctypes.c_float)


class fmm_plan_desc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int64), ("M", ctypes.c_int64), ("K", ctypes.c_int64),
                ("N", ctypes.c_int64), ("depth", ctypes.c_int32), ("block", ctypes.c_int32),
                ("rule", ctypes.c_int32), ("flags", ctypes.c_int32)]


class fmm_view(ctypes.Structure):
    _fields_ = [("codes", ctypes.c_void_p), ("scales", ctypes.c_void_p),
                ("batch", ctypes.c_int64), ("terms", ctypes.c_int64), ("rows", ctypes.c_int64),
                ("kdim", ctypes.c_int64), ("kblocks", ctypes.c_int64),
                ("scale_bytes", ctypes.c_int32), ("code_layout", ctypes.c_int32)]


_SIGS = {
    "fmm_realization_builtin": (ctypes.c_int, [ctypes.c_int, ctypes.POINTER(_vp)]),
    "fmm_realization_create": (ctypes.c_int, [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                              _dp, _dp, _dp, ctypes.c_double, ctypes.POINTER(_vp)]),
    "fmm_realization_transform": (ctypes.c_int, [_vp, _dp, _dp, _dp, ctypes.POINTER(_vp)]),
    "fmm_realization_rebalance": (ctypes.c_int, [_vp, ctypes.POINTER(_vp)]),
    "fmm_realization_optimize": (ctypes.c_int, [_vp, ctypes.c_int, _dp, ctypes.c_int, ctypes.c_double,
                                                ctypes.c_double, ctypes.POINTER(_vp), _dp, _dp]),
    "fmm_realization_phi_gradient": (ctypes.c_int, [_vp, _dp, _dp, _dp]),
    "fmm_realization_metrics": (ctypes.c_int, [_vp, ctypes.c_int, _dp, _dp, _dp]),
    "fmm_realization_terms": (ctypes.c_int, [_vp, ctypes.c_int, ctypes.POINTER(_i64),
                                             ctypes.POINTER(_i64)]),
    "fmm_realization_shape": (ctypes.c_int, [_vp, ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_int),
                                             ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_int)]),
    "fmm_realization_coefficients": (ctypes.c_int, [_vp, _dp, _dp, _dp]),
    "fmm_realization_tables": (ctypes.c_int, [_vp, ctypes.c_int, _fp, _fp, _fp]),
    "fmm_realization_destroy": (None, [_vp]),
    "fmm_plan_create": (ctypes.c_int, [_vp, ctypes.POINTER(fmm_plan_desc), ctypes.POINTER(_vp)]),
    "fmm_plan_workspace_size": (ctypes.c_int, [_vp, ctypes.POINTER(ctypes.c_size_t)]),
    "fmm_encode": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp]),
    "fmm_operand_views": (ctypes.c_int, [_vp, _vp, ctypes.POINTER(fmm_view),
                                         ctypes.POINTER(fmm_view)]),
    "fmm_multiply": (ctypes.c_int, [_vp, _vp, _vp, _vp]),
    "fmm_products": (ctypes.c_int, [_vp, _vp, _vp, _vp]),
    "fmm_combine": (ctypes.c_int, [_vp, _vp, _vp, _vp]),
    "fmm_matmul": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp, _vp]),
    "fmm_plan_destroy": (None, [_vp]),
    "fmm_reference_f64": (ctypes.c_int, [_i64, _i64, _i64, _i64, _vp, _vp, _vp, _vp]),
    "fmm_error_stats_scratch_size": (ctypes.c_int, [_i64, _i64, _i64,
                                                    ctypes.POINTER(ctypes.c_size_t)]),
    "fmm_error_stats": (ctypes.c_int, [_i64, _i64, _i64, _vp, _vp, _vp, _vp, ctypes.c_size_t,
                                       _vp]),
    "fmm_error_stats_noalloc": (ctypes.c_int, [_i64, _i64, _i64, _vp, _vp, _vp, _vp]),
    "fmm_cross_terms_scratch_size": (ctypes.c_int, [_vp, ctypes.POINTER(ctypes.c_size_t)]),
    "fmm_cross_terms": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]),
    "fmm_e4m3_quantize": (ctypes.c_int, [_vp, _vp, _i64, _vp]),
    "fmm_e4m3_quantize_pow2": (ctypes.c_int, [_vp, _vp, _i64, ctypes.c_int32, _vp]),
    "fmm_encode_noise_scratch_size": (ctypes.c_int, [_vp, ctypes.POINTER(ctypes.c_size_t)]),
    "fmm_encode_noise": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]),
    "fmm_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "fmm_last_error_detail": (ctypes.c_char_p, []),
    "fmm_device_check": (ctypes.c_int, [ctypes.c_int]),
}

for _name, (_res, _args) in _SIGS.items():
    _f = getattr(_lib, _name)
    _f.restype = _res
    _f.argtypes = _args

EXPORTS = tuple(_SIGS)


class FmmError(RuntimeError):
    def __init__(self, status: int, call: str):
        detail = _lib.fmm_last_error_detail().decode()
        msg = f"{call}: {_lib.fmm_status_string(status).decode()} ({status})"
        if status in (FMM_ERR_HIP, FMM_ERR_WORKSPACE) and detail:
            msg += f": {detail}"
        super().__init__(msg)
        self.status = status


def _check(status: int, call: str) -> None:
    if status != FMM_OK:
        raise FmmError(status, call)


def _ptr(x):
    """Device pointer of a torch tensor (or an int address, or None)."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


# ---------------------------------------------------------------------------
# Realizations: the C calls, plus a small owning handle
# ---------------------------------------------------------------------------

class Realization:
    """Owns an fmm_real handle."""

    # bound here, not looked up at collection time: module globals may already
    # be gone while the interpreter shuts down, when handles are left to the OS
    _destroy = _lib.fmm_realization_destroy
    _finalizing = sys.is_finalizing

    def __init__(self, handle: int):
        self.handle = handle

    def __del__(self):
        h, self.handle = getattr(self, "handle", None), None
        if h and not self._finalizing():
            self._destroy(h)


def fmm_realization_builtin(which) -> Realization:
    if isinstance(which, str):
        which = BUILTINS[which]
    h = _vp()
    _check(_lib.fmm_realization_builtin(int(which), ctypes.byref(h)), "fmm_realization_builtin")
    return Realization(h.value)


def _darr(a, n):
    import numpy as np
    a = np.ascontiguousarray(a, dtype=np.float64).reshape(-1)
    if a.size != n:
        raise ValueError(f"expected {n} doubles, got {a.size}")
    return a, a.ctypes.data_as(_dp)


def fmm_realization_create(U, V, w, tol: float = 1e-9, shape=(2, 2, 2)) -> Realization:
    """A realization of <m,k,n;R> from R x mk, R x kn, R x nm coefficient
    arrays; shape = (m, k, n).  Shapes other than (2, 2, 2) run at depth 1
    on the large-tile plans only."""
    import numpy as np
    m, k, n = (int(x) for x in shape)
    R = int(np.asarray(U).shape[0])
    Ua, Up = _darr(U, m * k * R)
    Va, Vp = _darr(V, k * n * R)
    Wa, Wp = _darr(w, n * m * R)
    h = _vp()
    _check(_lib.fmm_realization_create(m, k, n, R, Up, Vp, Wp, float(tol), ctypes.byref(h)),
           "fmm_realization_create")
    return Realization(h.value)


def _orbit_sizes(d: Realization):
    (m, k, n), _ = fmm_realization_shape(d)
    return m * m, k * k, n * n


def fmm_realization_transform(d: Realization, X, Y, Z) -> Realization:
    """D . (X, Y, Z): 2 x 2 factors at <2,2,2>; m x m, k x k, n x n for another shape."""
    sx, sy, sz = _orbit_sizes(d)
    Xa, Xp = _darr(X, sx)
    Ya, Yp = _darr(Y, sy)
    Za, Zp = _darr(Z, sz)
    h = _vp()
    _check(_lib.fmm_realization_transform(d.handle, Xp, Yp, Zp, ctypes.byref(h)),
           "fmm_realization_transform")
    return Realization(h.value)


def fmm_realization_optimize(d: Realization, starts=None, max_iter: int = 1000, gtol: float = 1e-10,
                             tol: float = 1e-9):
    """Re-basing: (realization of least Phi, its Phi, per-start terminal Phi).
    starts: None or an (n, P) array of (X, Y, Z) triples, row-major each
    (P = 12 at <2,2,2>, m^2 + k^2 + n^2 for another shape); the identity
    start is always run first."""
    import numpy as np
    P = sum(_orbit_sizes(d))
    if starts is None:
        n, sp = 0, None
    else:
        sa = np.ascontiguousarray(starts, dtype=np.float64).reshape(-1, P)
        n, sp = sa.shape[0], sa.ctypes.data_as(_dp)
    start_phi = np.empty(n + 1, dtype=np.float64)
    phi = ctypes.c_double()
    h = _vp()
    _check(_lib.fmm_realization_optimize(d.handle, n, sp, int(max_iter), float(gtol), float(tol),
                                         ctypes.byref(h), ctypes.byref(phi),
                                         start_phi.ctypes.data_as(_dp)), "fmm_realization_optimize")
    return Realization(h.value), phi.value, start_phi


def fmm_realization_phi_gradient(d: Realization, g):
    """(Phi(D . g), gradient over the P entries of g = (X, Y, Z); P = 12 at
    <2,2,2>, m^2 + k^2 + n^2 for another shape)."""
    import numpy as np
    P = sum(_orbit_sizes(d))
    ga, gp = _darr(g, P)
    grad = np.empty(P, dtype=np.float64)
    phi = ctypes.c_double()
    _check(_lib.fmm_realization_phi_gradient(d.handle, gp, ctypes.byref(phi), grad.ctypes.data_as(_dp)),
           "fmm_realization_phi_gradient")
    return phi.value, grad


def fmm_realization_rebalance(d: Realization) -> Realization:
    h = _vp()
    _check(_lib.fmm_realization_rebalance(d.handle, ctypes.byref(h)), "fmm_realization_rebalance")
    return Realization(h.value)


def fmm_realization_metrics(d: Realization, depth: int = 1):
    phi, gam, res = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    _check(_lib.fmm_realization_metrics(d.handle, depth, ctypes.byref(phi), ctypes.byref(gam),
                                        ctypes.byref(res)), "fmm_realization_metrics")
    return {"phi": phi.value, "gamma": gam.value, "brent_residual": res.value}


def fmm_realization_terms(d: Realization, depth: int = 1):
    R, T = _i64(), _i64()
    _check(_lib.fmm_realization_terms(d.handle, depth, ctypes.byref(R), ctypes.byref(T)),
           "fmm_realization_terms")
    return R.value, T.value


def fmm_realization_shape(d: Realization):
    """((m, k, n), R)."""
    m, k, n, R = (ctypes.c_int() for _ in range(4))
    _check(_lib.fmm_realization_shape(d.handle, ctypes.byref(m), ctypes.byref(k), ctypes.byref(n),
                                      ctypes.byref(R)), "fmm_realization_shape")
    return (m.value, k.value, n.value), R.value


def fmm_realization_coefficients(d: Realization):
    import numpy as np
    (m, k, n), R = fmm_realization_shape(d)
    U, V, W = np.zeros((R, m * k)), np.zeros((R, k * n)), np.zeros((R, n * m))
    _check(_lib.fmm_realization_coefficients(d.handle, U.ctypes.data_as(_dp),
                                             V.ctypes.data_as(_dp), W.ctypes.data_as(_dp)),
           "fmm_realization_coefficients")
    return U, V, W


def fmm_realization_tables(d: Realization, depth: int = 1):
    import numpy as np
    _, T = fmm_realization_terms(d, depth)
    (m, k, n), _ = fmm_realization_shape(d)
    if (m, k, n) == (2, 2, 2):
        U, V, W = (np.zeros((T, 4 ** depth), dtype=np.float32) for _ in range(3))
    else:
        U, V, W = (np.zeros((T, c), dtype=np.float32) for c in (m * k, k * n, n * m))
    _check(_lib.fmm_realization_tables(d.handle, depth, U.ctypes.data_as(_fp),
                                       V.ctypes.data_as(_fp), W.ctypes.data_as(_fp)),
           "fmm_realization_tables")
    return U, V, W


# ---------------------------------------------------------------------------
# Plans and device calls
# ---------------------------------------------------------------------------

class Plan:
    """Owns an fmm_plan handle and remembers its descriptor."""

    _destroy = _lib.fmm_plan_destroy
    _finalizing = sys.is_finalizing

    def __init__(self, handle: int, desc: fmm_plan_desc):
        self.handle = handle
        self.desc = desc

    def __del__(self):
        h, self.handle = getattr(self, "handle", None), None
        if h and not self._finalizing():
            self._destroy(h)


def make_desc(batch, M, K, N, depth=1, block=32, rule="pow2_ceil", exact_dot=False,
              flags=None) -> fmm_plan_desc:
    if isinstance(rule, str):
        rule = RULES[rule]
    if flags is None:
        flags = FMM_FLAG_EXACT_DOT if exact_dot else 0
    return fmm_plan_desc(int(batch), int(M), int(K), int(N), int(depth), int(block), int(rule),
                         int(flags))


def fmm_encode_noise_scratch_size(p: Plan) -> int:
    n = ctypes.c_size_t()
    _check(_lib.fmm_encode_noise_scratch_size(p.handle, ctypes.byref(n)), "fmm_encode_noise_scratch_size")
    return n.value


def fmm_encode_noise(p: Plan, A, B, ws, out, scratch, scratch_bytes: int, stream=None):
    _check(_lib.fmm_encode_noise(p.handle, _ptr(A), _ptr(B), _ptr(ws), _ptr(out), _ptr(scratch),
                                 int(scratch_bytes), _stream(stream)), "fmm_encode_noise")


def fmm_cross_terms_scratch_size(p: Plan) -> int:
    n = ctypes.c_size_t()
    _check(_lib.fmm_cross_terms_scratch_size(p.handle, ctypes.byref(n)), "fmm_cross_terms_scratch_size")
    return n.value


def fmm_cross_terms(p: Plan, A, B, ws, out, scratch, scratch_bytes: int, stream=None):
    _check(_lib.fmm_cross_terms(p.handle, _ptr(A), _ptr(B), _ptr(ws), _ptr(out), _ptr(scratch),
                                int(scratch_bytes), _stream(stream)), "fmm_cross_terms")


def fmm_plan_create(d: Realization, desc: fmm_plan_desc) -> Plan:
    h = _vp()
    _check(_lib.fmm_plan_create(d.handle, ctypes.byref(desc), ctypes.byref(h)), "fmm_plan_create")
    return Plan(h.value, desc)


def fmm_plan_create_status(d: Realization, desc: fmm_plan_desc) -> int:
    """The raw status of fmm_plan_create (the plan, if any, is released)."""
    h = _vp()
    st = _lib.fmm_plan_create(d.handle, ctypes.byref(desc), ctypes.byref(h))
    if h.value:
        _lib.fmm_plan_destroy(h.value)
    return st


def fmm_plan_workspace_size(p: Plan) -> int:
    n = ctypes.c_size_t()
    _check(_lib.fmm_plan_workspace_size(p.handle, ctypes.byref(n)), "fmm_plan_workspace_size")
    return n.value


def fmm_encode(p: Plan, A, B, ws, stream=None) -> None:
    _check(_lib.fmm_encode(p.handle, _ptr(A), _ptr(B), _ptr(ws), _stream(stream)), "fmm_encode")


def fmm_operand_views(p: Plan, ws):
    a, b = fmm_view(), fmm_view()
    _check(_lib.fmm_operand_views(p.handle, _ptr(ws), ctypes.byref(a), ctypes.byref(b)),
           "fmm_operand_views")
    return a, b


def fmm_multiply(p: Plan, ws, C, stream=None) -> None:
    _check(_lib.fmm_multiply(p.handle, _ptr(ws), _ptr(C), _stream(stream)), "fmm_multiply")


def fmm_products(p: Plan, ws, C, stream=None) -> None:
    _check(_lib.fmm_products(p.handle, _ptr(ws), _ptr(C), _stream(stream)), "fmm_products")


def fmm_combine(p: Plan, ws, C, stream=None) -> None:
    _check(_lib.fmm_combine(p.handle, _ptr(ws), _ptr(C), _stream(stream)), "fmm_combine")


def fmm_matmul(p: Plan, A, B, C, ws, stream=None) -> None:
    _check(_lib.fmm_matmul(p.handle, _ptr(A), _ptr(B), _ptr(C), _ptr(ws), _stream(stream)),
           "fmm_matmul")


def fmm_reference_f64(batch, M, K, N, A, B, Cref, stream=None) -> None:
    _check(_lib.fmm_reference_f64(batch, M, K, N, _ptr(A), _ptr(B), _ptr(Cref), _stream(stream)),
           "fmm_reference_f64")


def fmm_error_stats_scratch_size(batch, M, N) -> int:
    n = ctypes.c_size_t()
    _check(_lib.fmm_error_stats_scratch_size(batch, M, N, ctypes.byref(n)),
           "fmm_error_stats_scratch_size")
    return n.value


def fmm_error_stats(batch, M, N, C, Cref, out, scratch, scratch_bytes, stream=None) -> None:
    _check(_lib.fmm_error_stats(batch, M, N, _ptr(C), _ptr(Cref), _ptr(out), _ptr(scratch),
                                int(scratch_bytes), _stream(stream)), "fmm_error_stats")


FMM_ERROR_STATS_NOALLOC_MAX_BATCH = 1024


def fmm_error_stats_noalloc(batch, M, N, C, Cref, out, stream=None) -> None:
    _check(_lib.fmm_error_stats_noalloc(batch, M, N, _ptr(C), _ptr(Cref), _ptr(out), _stream(stream)),
           "fmm_error_stats_noalloc")


def fmm_e4m3_quantize(x, out, n, stream=None) -> None:
    _check(_lib.fmm_e4m3_quantize(_ptr(x), _ptr(out), int(n), _stream(stream)), "fmm_e4m3_quantize")


def fmm_e4m3_quantize_pow2(x, out, n, e, stream=None) -> None:
    _check(_lib.fmm_e4m3_quantize_pow2(_ptr(x), _ptr(out), int(n), int(e), _stream(stream)),
           "fmm_e4m3_quantize_pow2")


def fmm_status_string(status: int) -> str:
    return _lib.fmm_status_string(status).decode()


def fmm_device_check(device: int = 0) -> int:
    return _lib.fmm_device_check(device)
