"""Thin Python binding of the C ABI in include/lp.h.

Each function has the name of the C entry point it calls and only marshals
arguments: it checks that tensors live on the GPU, are contiguous, have the
problem dtype and at least the element count the C call will touch, then passes
``data_ptr()`` values and the current HIP stream. Every step of the computation
runs in the HIP library; there is no fallback. If the library is missing, every
call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Tuple

# the in-tree build; LP_LIBRARY names another build of the same library (e.g. to
# compare kernel variants under the same tests)
LIB_PATH = os.environ.get("LP_LIBRARY") or os.path.join(os.path.dirname(os.path.abspath(__file__)), "liblp.so")

LP_ABI_VERSION = 4
LP_OK, LP_EINVAL, LP_EUNSUPPORTED, LP_EWORKSPACE, LP_EHIP, LP_ENONFINITE = range(6)
LP_F32, LP_F64 = 0, 1
LP_DENSE, LP_CONV3X3 = 0, 1
LP_TANH, LP_RELU, LP_SMOOTHRELU, LP_IDENTITY = 0, 1, 2, 3
LP_RELAX_F, LP_RELAX_FCF, LP_RELAX_FCFCF = 0, 1, 2
LP_CYCLE_V, LP_CYCLE_F = 0, 1
LP_STATE, LP_ADJOINT = 0, 1
LP_OPEN_IDENTITY, LP_OPEN_DENSE_ACT, LP_OPEN_CONV_ACT = 0, 1, 2
LP_STORE_ALL, LP_STORE_CPOINTS = 0, 1

ACT = {"tanh": LP_TANH, "relu": LP_RELU, "smoothrelu": LP_SMOOTHRELU, "identity": LP_IDENTITY}
LAYER = {"dense": LP_DENSE, "conv3x3": LP_CONV3X3}
RELAX = {"F": LP_RELAX_F, "FCF": LP_RELAX_FCF, "FCFCF": LP_RELAX_FCFCF}
CYCLE = {"V": LP_CYCLE_V, "F": LP_CYCLE_F}
OPENING = {"identity": LP_OPEN_IDENTITY, "dense_act": LP_OPEN_DENSE_ACT, "conv_act": LP_OPEN_CONV_ACT}

# Every symbol the header declares (checked by the CPU test suite).
EXPORTS = (
    "lp_abi_version", "lp_status_string", "lp_last_error", "lp_workspace_bytes",
    "lp_dsig_bytes", "lp_serial_forward", "lp_serial_adjoint", "lp_mgrit_forward", "lp_mgrit_adjoint",
    "lp_gradient", "lp_gradient_cpoints", "lp_residual_norm", "lp_residual_norm_noalloc", "lp_check_finite", "lp_open_forward", "lp_open_grad",
    "lp_loss_terminal", "lp_sgd_update", "lp_vec_axpby", "lp_vec_dot", "lp_accuracy",
    "lp_trace_enable", "lp_trace_read",
)


class LpProblem(ctypes.Structure):
    _fields_ = [("abi_version", ctypes.c_int32), ("dtype", ctypes.c_int32), ("layer", ctypes.c_int32),
                ("act", ctypes.c_int32), ("N", ctypes.c_int32), ("B", ctypes.c_int32),
                ("C", ctypes.c_int32), ("H", ctypes.c_int32), ("W", ctypes.c_int32),
                ("h", ctypes.c_double)]

    @property
    def q(self) -> int:
        return self.C * self.H * self.W


class LpMgrit(ctypes.Structure):
    _fields_ = [("cf", ctypes.c_int32), ("max_levels", ctypes.c_int32), ("min_coarse", ctypes.c_int32),
                ("relax", ctypes.c_int32), ("max_iter", ctypes.c_int32), ("warm_start", ctypes.c_int32),
                ("rtol", ctypes.c_double), ("stag", ctypes.c_double), ("cycle", ctypes.c_int32),
                ("storage", ctypes.c_int32)]


class LpError(RuntimeError):
    def __init__(self, status: int, call: str, detail: str):
        super().__init__(f"{call}: status {status} ({detail})")
        self.status = status


_lib: Optional[ctypes.CDLL] = None

_P = ctypes.POINTER(LpProblem)
_M = ctypes.POINTER(LpMgrit)
_v = ctypes.c_void_p
_i32 = ctypes.c_int32
_sz = ctypes.c_size_t
_dp = ctypes.POINTER(ctypes.c_double)
_ip = ctypes.POINTER(ctypes.c_int32)

_SIGS = {
    "lp_abi_version": ([], _i32),
    "lp_status_string": ([_i32], ctypes.c_char_p),
    "lp_last_error": ([], ctypes.c_char_p),
    "lp_workspace_bytes": ([_P, _M], _sz),
    "lp_dsig_bytes": ([_P], _sz),
    "lp_serial_forward": ([_P, _v, _v, _v, _v, _v], _i32),
    "lp_serial_adjoint": ([_P, _v, _v, _v, _v, _v, _v], _i32),
    "lp_mgrit_forward": ([_P, _M, _v, _v, _v, _v, _v, _sz, _dp, _ip, _v], _i32),
    "lp_mgrit_adjoint": ([_P, _M, _v, _v, _v, _v, _v, _v, _sz, _dp, _ip, _v], _i32),
    "lp_gradient": ([_P, _v, _v, _v, _v, _v, _v, _v, _v, _sz, _v], _i32),
    "lp_gradient_cpoints": ([_P, _i32, _v, _v, _v, _v, _v, _v, _v, _sz, _v], _i32),
    "lp_residual_norm": ([_P, _i32, _v, _v, _v, _v, _v, _sz, _dp, _v], _i32),
    "lp_residual_norm_noalloc": ([_P, _i32, _v, _v, _v, _v, _dp, _v], _i32),
    "lp_check_finite": ([_v], _i32),
    "lp_open_forward": ([_P, _i32, _i32, _v, _v, _v, _v], _i32),
    "lp_open_grad": ([_P, _i32, _i32, _v, _v, _v, _v, _v], _i32),
    "lp_loss_terminal": ([_P, _i32, _v, _v, _v, _v, _v, _v, _v, _v, _v, _sz, _v], _i32),
    "lp_sgd_update": ([_i32, _sz, ctypes.c_double, _v, _v, _v], _i32),
    "lp_vec_axpby": ([_i32, _sz, ctypes.c_double, _v, ctypes.c_double, _v, _v], _i32),
    "lp_vec_dot": ([_i32, _sz, _v, _v, _v, _v], _i32),
    "lp_accuracy": ([_P, _i32, _v, _v, _v, _v, _v, _v, _sz, _v], _i32),
    "lp_trace_enable": ([ctypes.c_uint32], _i32),
    "lp_trace_read": ([_i32, _i32, _ip, _dp], _i32),
}


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load liblp.so (once). Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it with paper_1812_04352_amd.build.build()")
        lib = ctypes.CDLL(path)
        for name, (args, res) in _SIGS.items():
            f = getattr(lib, name)
            f.argtypes = args
            f.restype = res
        if lib.lp_abi_version() != LP_ABI_VERSION:
            raise RuntimeError("liblp.so ABI version mismatch")
        _lib = lib
    return _lib


def _check(rc: int, call: str) -> None:
    if rc != LP_OK:
        lib = load()
        raise LpError(rc, call, lib.lp_last_error().decode())


def problem(dtype: str, layer: str, act: str, N: int, B: int, C: int, H: int = 1, W: int = 1,
            h: float = 1.0) -> LpProblem:
    return LpProblem(LP_ABI_VERSION, LP_F32 if dtype == "f32" else LP_F64, LAYER[layer], ACT[act],
                     N, B, C, H, W, h)


def mgrit(cf: int = 4, max_levels: int = 2, min_coarse: int = 1, relax: str = "FCF", max_iter: int = 1,
          warm_start: bool = False, rtol: float = 0.0, stag: float = 0.0, cycle: str = "V",
          storage: str = "all") -> LpMgrit:
    """storage: "all" (every layer of U stored) or "cpoints" (U holds the fine C-points only)."""
    return LpMgrit(cf, max_levels, min_coarse, RELAX[relax], max_iter, int(bool(warm_start)), rtol, stag,
                   CYCLE[cycle], {"all": LP_STORE_ALL, "cpoints": LP_STORE_CPOINTS}[storage])


def traj_rows(p: "LpProblem", mg: Optional[LpMgrit] = None) -> int:
    """Rows of the primal trajectory U under the schedule's storage: N + 1, or
    N / cf + 1 C-points."""
    if mg is not None and mg.storage == LP_STORE_CPOINTS:
        return p.N // mg.cf + 1
    return p.N + 1


# ---------------------------------------------------------------- tensor marshalling

def _stream():
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _elem_dtype(p: LpProblem):
    import torch
    return torch.float32 if p.dtype == LP_F32 else torch.float64


def _arr(t, numel: int, name: str, dtype=None):
    """Device pointer of a contiguous GPU tensor holding at least numel elements."""
    if t is None:
        raise ValueError(f"{name} is required")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if t.numel() < numel:
        raise ValueError(f"{name} has {t.numel()} elements, needs {numel}")
    return ctypes.c_void_p(t.data_ptr())


def _weights(p: LpProblem, K, b):
    dt = _elem_dtype(p)
    nk = p.N * (p.C * p.C if p.layer == LP_DENSE else p.C * p.C * 9)
    return _arr(K, nk, "K", dt), _arr(b, p.N * p.C, "b", dt)


def _ws(ws, need: int):
    if need == 0:
        return ctypes.c_void_p(ws.data_ptr() if ws is not None else 0), (ws.numel() if ws is not None else 0)
    if ws is None:
        raise ValueError(f"a workspace of {need} bytes is required")
    nbytes = ws.numel() * ws.element_size()
    if not ws.is_cuda or not ws.is_contiguous():
        raise ValueError("workspace must be a contiguous GPU tensor")
    return ctypes.c_void_p(ws.data_ptr()), nbytes


def lp_workspace_bytes(p: LpProblem, mg: Optional[LpMgrit] = None) -> int:
    n = load().lp_workspace_bytes(ctypes.byref(p), ctypes.byref(mg) if mg is not None else None)
    if n == 0:
        raise LpError(LP_EINVAL, "lp_workspace_bytes", load().lp_last_error().decode())
    return int(n)


def alloc_workspace(p: LpProblem, mg: Optional[LpMgrit] = None, device="cuda"):
    import torch
    return torch.empty(lp_workspace_bytes(p, mg), dtype=torch.uint8, device=device)


def lp_dsig_bytes(p: LpProblem) -> int:
    return int(load().lp_dsig_bytes(ctypes.byref(p)))


def alloc_dsig(p: LpProblem, device="cuda"):
    """A buffer for the sigma' record of p (may be empty: the identity has none)."""
    import torch
    return torch.empty(max(1, lp_dsig_bytes(p)), dtype=torch.uint8, device=device)


def _dsig(p: LpProblem, dsig):
    """Device pointer of a sigma' record buffer (any dtype, counted in bytes), or NULL."""
    if dsig is None:
        return None
    if not dsig.is_cuda or not dsig.is_contiguous():
        raise ValueError("dsig must be a contiguous GPU tensor")
    need = lp_dsig_bytes(p)
    if dsig.numel() * dsig.element_size() < need:
        raise ValueError(f"dsig holds {dsig.numel() * dsig.element_size()} bytes, needs {need}")
    return ctypes.c_void_p(dsig.data_ptr())


def lp_serial_forward(p: LpProblem, K, b, U, dsig=None) -> None:
    Kp, bp = _weights(p, K, b)
    _check(load().lp_serial_forward(ctypes.byref(p), Kp, bp, _arr(U, (p.N + 1) * p.B * p.q, "U", _elem_dtype(p)),
                                    _dsig(p, dsig), _stream()), "lp_serial_forward")


def lp_serial_adjoint(p: LpProblem, K, b, U, Lam, dsig=None) -> None:
    Kp, bp = _weights(p, K, b)
    n = (p.N + 1) * p.B * p.q
    _check(load().lp_serial_adjoint(ctypes.byref(p), Kp, bp, _arr(U, n, "U", _elem_dtype(p)), _dsig(p, dsig),
                                    _arr(Lam, n, "Lam", _elem_dtype(p)), _stream()), "lp_serial_adjoint")


def lp_mgrit_forward(p: LpProblem, mg: LpMgrit, K, b, U, ws, history: bool = True,
                     dsig=None) -> Tuple[int, list]:
    """history=False passes no residual history: without a stopping rule the
    call then returns without waiting for the stream (the list is empty).
    dsig: a buffer (alloc_dsig) that receives the iterate's sigma' record."""
    Kp, bp = _weights(p, K, b)
    hist = (ctypes.c_double * max(1, mg.max_iter))() if history else None
    it = ctypes.c_int32(0)
    wp, wn = _ws(ws, 1)
    _check(load().lp_mgrit_forward(ctypes.byref(p), ctypes.byref(mg), Kp, bp,
                                   _arr(U, traj_rows(p, mg) * p.B * p.q, "U", _elem_dtype(p)), _dsig(p, dsig), wp, wn,
                                   hist, ctypes.byref(it), _stream()), "lp_mgrit_forward")
    return it.value, list(hist[:it.value]) if history else []


def lp_mgrit_adjoint(p: LpProblem, mg: LpMgrit, K, b, U, Lam, ws, history: bool = True,
                     dsig=None) -> Tuple[int, list]:
    """history as for lp_mgrit_forward; dsig: the sigma' record of U (or None)."""
    Kp, bp = _weights(p, K, b)
    n = (p.N + 1) * p.B * p.q
    hist = (ctypes.c_double * max(1, mg.max_iter))() if history else None
    it = ctypes.c_int32(0)
    wp, wn = _ws(ws, 1)
    _check(load().lp_mgrit_adjoint(ctypes.byref(p), ctypes.byref(mg), Kp, bp,
                                   _arr(U, traj_rows(p, mg) * p.B * p.q, "U", _elem_dtype(p)),
                                   _dsig(p, dsig), _arr(Lam, n, "Lam", _elem_dtype(p)), wp, wn, hist,
                                   ctypes.byref(it), _stream()), "lp_mgrit_adjoint")
    return it.value, list(hist[:it.value]) if history else []


def lp_gradient(p: LpProblem, K, b, U, Lam, dK, db, ws, dsig=None) -> None:
    Kp, bp = _weights(p, K, b)
    dKp, dbp = _weights(p, dK, db)
    n = (p.N + 1) * p.B * p.q
    wp, wn = _ws(ws, 1)
    _check(load().lp_gradient(ctypes.byref(p), Kp, bp, _arr(U, n, "U", _elem_dtype(p)), _dsig(p, dsig),
                              _arr(Lam, n, "Lam", _elem_dtype(p)), dKp, dbp, wp, wn, _stream()), "lp_gradient")


def lp_gradient_cpoints(p: LpProblem, cf: int, K, b, Uc, Lam, dK, db, ws) -> None:
    """lp_gradient from the C-point trajectory Uc [N/cf + 1][B][q]."""
    Kp, bp = _weights(p, K, b)
    dKp, dbp = _weights(p, dK, db)
    wp, wn = _ws(ws, 1)
    _check(load().lp_gradient_cpoints(ctypes.byref(p), cf, Kp, bp,
                                      _arr(Uc, (p.N // cf + 1) * p.B * p.q, "Uc", _elem_dtype(p)),
                                      _arr(Lam, (p.N + 1) * p.B * p.q, "Lam", _elem_dtype(p)), dKp, dbp, wp, wn,
                                      _stream()), "lp_gradient_cpoints")


def lp_residual_norm(p: LpProblem, which: int, K, b, U, Lam, ws) -> float:
    Kp, bp = _weights(p, K, b)
    n = (p.N + 1) * p.B * p.q
    out = ctypes.c_double(0.0)
    lam = _arr(Lam, n, "Lam", _elem_dtype(p)) if which == LP_ADJOINT else None
    wp, wn = _ws(ws, 1)
    _check(load().lp_residual_norm(ctypes.byref(p), which, Kp, bp, _arr(U, n, "U", _elem_dtype(p)), lam, wp, wn,
                                   ctypes.byref(out), _stream()), "lp_residual_norm")
    return out.value


def lp_residual_norm_noalloc(p: LpProblem, which: int, K, b, U, Lam) -> float:
    """lp_residual_norm on the library's static scratch (no workspace)."""
    Kp, bp = _weights(p, K, b)
    n = (p.N + 1) * p.B * p.q
    out = ctypes.c_double(0.0)
    lam = _arr(Lam, n, "Lam", _elem_dtype(p)) if which == LP_ADJOINT else None
    _check(load().lp_residual_norm_noalloc(ctypes.byref(p), which, Kp, bp, _arr(U, n, "U", _elem_dtype(p)), lam,
                                           ctypes.byref(out), _stream()), "lp_residual_norm_noalloc")
    return out.value


def lp_check_finite() -> None:
    """Raise LpError(LP_ENONFINITE) if a residual norm computed on the current
    device since the last check was NaN or Inf (waits for the current stream)."""
    _check(load().lp_check_finite(_stream()), "lp_check_finite")


def lp_open_forward(p: LpProblem, opening: int, nf: int, y, L_in, u0) -> None:
    dt = _elem_dtype(p)
    if opening == LP_OPEN_IDENTITY:
        yp, Lp = _arr(y, p.B * p.q, "y", dt), None
    elif opening == LP_OPEN_DENSE_ACT:
        yp, Lp = _arr(y, p.B * nf, "y", dt), _arr(L_in, p.q * nf, "L_in", dt)
    else:
        yp, Lp = _arr(y, p.B * p.H * p.W, "y", dt), _arr(L_in, p.C * 9, "L_in", dt)
    _check(load().lp_open_forward(ctypes.byref(p), opening, nf, yp, Lp, _arr(u0, p.B * p.q, "u0", dt), _stream()),
           "lp_open_forward")


def lp_open_grad(p: LpProblem, opening: int, nf: int, y, L_in, lam0, dL_in) -> None:
    dt = _elem_dtype(p)
    if opening == LP_OPEN_DENSE_ACT:
        yp, nL = _arr(y, p.B * nf, "y", dt), p.q * nf
    else:
        yp, nL = _arr(y, p.B * p.H * p.W, "y", dt), p.C * 9
    _check(load().lp_open_grad(ctypes.byref(p), opening, nf, yp, _arr(L_in, nL, "L_in", dt),
                               _arr(lam0, p.B * p.q, "lam0", dt), _arr(dL_in, nL, "dL_in", dt), _stream()),
           "lp_open_grad")


def lp_loss_terminal(p: LpProblem, nc: int, uN, W, mu, c, J, lamN, dW, dmu, ws) -> None:
    import torch
    dt = _elem_dtype(p)
    wp, wn = _ws(ws, 1)
    _check(load().lp_loss_terminal(ctypes.byref(p), nc, _arr(uN, p.B * p.q, "uN", dt), _arr(W, nc * p.q, "W", dt),
                                   _arr(mu, nc, "mu", dt), _arr(c, p.B * nc, "c", dt),
                                   _arr(J, 1, "J", torch.float64), _arr(lamN, p.B * p.q, "lamN", dt),
                                   _arr(dW, nc * p.q, "dW", dt), _arr(dmu, nc, "dmu", dt), wp, wn, _stream()),
           "lp_loss_terminal")


def lp_trace_enable(kind_mask: int) -> None:
    _check(load().lp_trace_enable(kind_mask), "lp_trace_enable")


def lp_trace_read(kind: int, level: int = -1) -> Tuple[int, float]:
    n = ctypes.c_int32(0)
    ms = ctypes.c_double(0.0)
    _check(load().lp_trace_read(kind, level, ctypes.byref(n), ctypes.byref(ms)), "lp_trace_read")
    return n.value, ms.value


def lp_sgd_update(x, g, lr: float) -> None:
    import torch
    if x.dtype not in (torch.float32, torch.float64) or g.dtype != x.dtype:
        raise ValueError("x and g must share dtype float32 or float64")
    n = x.numel()
    dtype = LP_F32 if x.dtype == torch.float32 else LP_F64
    _check(load().lp_sgd_update(dtype, n, lr, _arr(g, n, "g"), _arr(x, n, "x"), _stream()), "lp_sgd_update")


LP_DOT_PARTIALS = 256


def _vec_dtype(*ts):
    import torch
    dt = ts[0].dtype
    if dt not in (torch.float32, torch.float64) or any(t.dtype != dt for t in ts):
        raise ValueError("vectors must share dtype float32 or float64")
    return LP_F32 if dt == torch.float32 else LP_F64


def lp_vec_axpby(y, x, a: float, b: float) -> None:
    """y <- a x + b y over all elements (b = 0: y <- a x)."""
    n = y.numel()
    if x.numel() != n:
        raise ValueError("x and y differ in size")
    _check(load().lp_vec_axpby(_vec_dtype(x, y), n, a, _arr(x, n, "x"), b, _arr(y, n, "y"), _stream()),
           "lp_vec_axpby")


def lp_vec_dot(x, y, out) -> None:
    """out[0] <- x . y in fp64 (out: a device float64 tensor of 1 + LP_DOT_PARTIALS
    elements; the value is left on the device)."""
    import torch
    n = x.numel()
    if y.numel() != n:
        raise ValueError("x and y differ in size")
    _check(load().lp_vec_dot(_vec_dtype(x, y), n, _arr(x, n, "x"), _arr(y, n, "y"),
                             _arr(out, 1 + LP_DOT_PARTIALS, "out", torch.float64), _stream()), "lp_vec_dot")


def lp_accuracy(p: LpProblem, nc: int, uN, W, mu, c, acc, ws) -> None:
    """acc[0] <- fraction of examples whose predicted class is their one-hot class."""
    import torch
    dt = _elem_dtype(p)
    wp, wn = _ws(ws, 1)
    _check(load().lp_accuracy(ctypes.byref(p), nc, _arr(uN, p.B * p.q, "uN", dt), _arr(W, nc * p.q, "W", dt),
                              _arr(mu, nc, "mu", dt), _arr(c, p.B * nc, "c", dt), _arr(acc, 1, "acc", torch.float64),
                              wp, wn, _stream()), "lp_accuracy")
