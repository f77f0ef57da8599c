"""ctypes binding of liboptima.so: argument marshalling only.

Every function has the name of the C entry point it wraps, takes torch tensors
(device memory) and passes their data pointers and the current HIP stream
through. No computation of the method happens here. The library must exist:
importing this module without it raises, there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, fields

import torch

# OPTIMA_LIBRARY names another build of the same library (the host-sanitized
# build that the ABI tests run against); by default the in-tree library.
_LIB_PATH = os.environ.get("OPTIMA_LIBRARY") or os.path.join(
    os.path.dirname(os.path.abspath(__file__)), "liboptima.so")

OPTIMA_OK = 0
OPTIMA_E_INVAL = -1
OPTIMA_E_HIP = -2
OPTIMA_E_NONFINITE = -3
OPTIMA_E_WORKSPACE = -4
OPTIMA_E_UNSUPPORTED = -5
DTYPE_F32 = 0
DTYPE_BF16 = 1
DTYPE_F64 = 2
METHOD_RAPDHG = 0
METHOD_CG = 1
PREC_FP32 = 0
PREC_BF16X3 = 1


class OptimaError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{message} (status {status})")
        self.status = status


if not os.path.exists(_LIB_PATH):
    raise ImportError(
        f"{_LIB_PATH} is missing: build it with `python paper_2512_13886_amd/build.py`")
_lib = ctypes.CDLL(_LIB_PATH)

_i64, _i32, _sz, _vp, _f32 = ctypes.c_int64, ctypes.c_int, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_float


class _Opts(ctypes.Structure):
    _fields_ = [("max_iters", ctypes.c_int64), ("check_every", ctypes.c_int32),
                ("fixed_iters", ctypes.c_int32), ("eps_rel", ctypes.c_float),
                ("eps_abs", ctypes.c_float), ("beta_sufficient", ctypes.c_float),
                ("beta_necessary", ctypes.c_float), ("beta_artificial", ctypes.c_float),
                ("step_safety", ctypes.c_float), ("restarts", ctypes.c_int32),
                ("precision", ctypes.c_int32), ("method", ctypes.c_int32),
                ("col_scale", ctypes.c_void_p), ("sparse", ctypes.c_int32),
                ("cooperative", ctypes.c_int32)]


class _Stats(ctypes.Structure):
    _fields_ = [("iters", _vp), ("restarts", _vp), ("converged", _vp),
                ("f_initial", _vp), ("f_final", _vp), ("kkt_final", _vp)]


class _Info(ctypes.Structure):
    _fields_ = [("iterations", ctypes.c_int64), ("gemm_calls", ctypes.c_int64),
                ("row_products", ctypes.c_int64), ("checks", ctypes.c_int64),
                ("timed_launches", ctypes.c_int64), ("timed_row_products", ctypes.c_int64),
                ("timed_product_ms", ctypes.c_double), ("sparse_products", ctypes.c_int64),
                ("few_launches", ctypes.c_int64), ("few_row_products", ctypes.c_int64),
                ("few_product_ms", ctypes.c_double), ("persistent_launches", ctypes.c_int64)]


def _sig(name, res, args):
    f = getattr(_lib, name)
    f.restype = res
    f.argtypes = args
    return f


_status_string = _sig("optima_status_string", ctypes.c_char_p, [_i32])
_abi_version = _sig("optima_abi_version", _i32, [])
# The structs above mirror include/optima.h at this ABI version.
ABI_VERSION = 11
if _abi_version() != ABI_VERSION:
    raise ImportError(f"{_LIB_PATH} has ABI version {_abi_version()}, the binding expects "
                      f"{ABI_VERSION}: rebuild the library")
_hess_ws = _sig("optima_hessian_workspace_bytes", _sz, [_i64, _i64, _i32])
_hess_acc = _sig("optima_hessian_accumulate", _i32,
                 [_vp, _i32, _i64, _i64, _vp, _i32, _vp, _sz, _vp])
_damp = _sig("optima_hessian_damp", _i32, [_vp, _i64, _f32, _vp, _vp])
_jacobi = _sig("optima_hessian_jacobi", _i32, [_vp, _i64, _vp, _vp])
_spec_ws = _sig("optima_spectral_norm_workspace_bytes", _sz, [_i64, _i32])
_spec = _sig("optima_spectral_norm", _i32,
             [_vp, _i64, _vp, _i32, _i32, _f32, _vp, _sz, _vp, _vp, _vp])
_spec_na = _sig("optima_spectral_norm_noalloc", _i32,
                [_vp, _i64, _vp, _i32, _i32, _f32, _vp, _vp, _vp])
_lz_ws = _sig("optima_spectral_lanczos_workspace_bytes", _sz, [_i64, _i32])
_lz = _sig("optima_spectral_lanczos", _i32,
           [_vp, _i64, _vp, _i32, _f32, _vp, _sz, _vp, _vp, _vp])
_mask = _sig("optima_wanda_mask", _i32,
             [_vp, _i64, _i64, _vp, _i32, _i64, _i32, ctypes.c_double, _vp, _vp])
_fwd_ws = _sig("optima_linear_forward_workspace_bytes", _sz, [_i64, _i64, _i64])
_fwd = _sig("optima_linear_forward", _i32,
            [_vp, _i64, _i64, _vp, _i64, _i32, _vp, _i32, _vp, _vp, _vp, _sz, _vp])
_opts_default = _sig("optima_solver_opts_default", None, [ctypes.POINTER(_Opts)])
_qp_ws = _sig("optima_qp_workspace_bytes", _sz, [_i64, _i64])
_qp_solve = _sig("optima_qp_solve_batched", _i32,
                 [_vp, _i64, _vp, _vp, _vp, _i64, ctypes.POINTER(_Opts), _vp, _sz, _vp,
                  ctypes.POINTER(_Stats), ctypes.POINTER(_Info), _vp])


def library_path() -> str:
    return _LIB_PATH


def optima_status_string(status: int) -> str:
    return _status_string(int(status)).decode()


def optima_abi_version() -> int:
    return int(_abi_version())


def _check(status: int):
    if status != OPTIMA_OK:
        raise OptimaError(status, optima_status_string(status))


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _need_cuda(name, t, dtype=None):
    if t is None:
        raise ValueError(f"{name} is required")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")


def _workspace(nbytes: int, ws, device, stream=None):
    """The caller's workspace, or a new one allocated on the stream the call
    runs on. torch's caching allocator ties a block to the stream it was
    allocated on, so the block freed when the call returns is handed only to
    later work on that stream, which runs after the library's kernels."""
    if ws is not None:
        _need_cuda("ws", ws)
        return ws, ws.numel() * ws.element_size()
    n = max(int(nbytes), 1)
    if stream is None:
        return torch.empty(n, dtype=torch.uint8, device=device), int(nbytes)
    with torch.cuda.stream(stream):
        return torch.empty(n, dtype=torch.uint8, device=device), int(nbytes)


@dataclass
class SolverOpts:
    """Mirror of optima_solver_opts; defaults come from the library."""
    max_iters: int = 0
    check_every: int = 0
    fixed_iters: int = 0
    eps_rel: float = 0.0
    eps_abs: float = 0.0
    beta_sufficient: float = 0.0
    beta_necessary: float = 0.0
    beta_artificial: float = 0.0
    step_safety: float = 0.0
    restarts: int = 0
    precision: int = 0
    method: int = 0
    col_scale: "torch.Tensor | None" = None  # [d] float32 device scaling D, or None
    sparse: int = 0
    cooperative: int = 0

    @classmethod
    def default(cls, **overrides) -> "SolverOpts":
        c = _Opts()
        _opts_default(ctypes.byref(c))
        o = cls(**{f.name: getattr(c, f.name) for f in fields(cls)})
        for k, v in overrides.items():
            if not hasattr(o, k):
                raise AttributeError(k)
            setattr(o, k, v)
        return o

    def _c(self) -> _Opts:
        vals = {f.name: getattr(self, f.name) for f in fields(self)}
        scale = vals.pop("col_scale")
        c = _Opts(**vals)
        c.col_scale = None if scale is None else scale.data_ptr()
        return c


def optima_hessian_workspace_bytes(n_tok: int, d: int, dtype: int) -> int:
    return int(_hess_ws(n_tok, d, dtype))


def optima_hessian_accumulate(X: torch.Tensor, H: torch.Tensor, accumulate: bool = False,
                              ws: torch.Tensor | None = None, stream=None) -> None:
    """H (+)= X^T X for X [n_tok, d] (float32 or bfloat16), H [d, d] float32."""
    _need_cuda("X", X)
    _need_cuda("H", H, torch.float32)
    if X.dim() != 2 or H.shape != (X.shape[1], X.shape[1]):
        raise ValueError("X must be [n_tok, d] and H [d, d]")
    dtype = {torch.float32: DTYPE_F32, torch.bfloat16: DTYPE_BF16}.get(X.dtype)
    if dtype is None:
        raise ValueError("X must be float32 or bfloat16")
    n_tok, d = X.shape
    ws, nbytes = _workspace(optima_hessian_workspace_bytes(n_tok, d, dtype), ws, X.device,
                           stream)
    _check(_hess_acc(_ptr(X), dtype, n_tok, d, _ptr(H), int(bool(accumulate)), _ptr(ws),
                     nbytes, _stream(stream)))


def optima_hessian_damp(H: torch.Tensor, rel_damp: float, lambda_out: torch.Tensor,
                        stream=None) -> None:
    _need_cuda("H", H, torch.float32)
    _need_cuda("lambda_out", lambda_out, torch.float32)
    _check(_damp(_ptr(H), H.shape[0], float(rel_damp), _ptr(lambda_out), _stream(stream)))


SPECTRAL_MAX_BLOCK = 16


def optima_hessian_jacobi(H: torch.Tensor, scale_out: torch.Tensor, stream=None) -> None:
    """H <- D H D in place with D = diag(H)^(-1/2); scale_out [d] receives D."""
    _need_cuda("H", H, torch.float32)
    _need_cuda("scale_out", scale_out, torch.float32)
    if H.dim() != 2 or H.shape[0] != H.shape[1] or scale_out.numel() != H.shape[0]:
        raise ValueError("H must be [d, d] and scale_out [d]")
    _check(_jacobi(_ptr(H), H.shape[0], _ptr(scale_out), _stream(stream)))


def optima_spectral_norm_workspace_bytes(d: int, block: int = 1) -> int:
    return int(_spec_ws(d, block))


def optima_spectral_norm(H: torch.Tensor, V0: torch.Tensor, lambda_max: torch.Tensor,
                         max_iters: int = 1000, tol: float = 1e-6,
                         ws: torch.Tensor | None = None, iters: torch.Tensor | None = None,
                         stream=None) -> None:
    """lambda_max(H). V0 is one start vector [d] (power iteration) or a block
    of start vectors [block, d] (subspace iteration with Rayleigh-Ritz)."""
    _need_cuda("H", H, torch.float32)
    _need_cuda("V0", V0, torch.float32)
    _need_cuda("lambda_max", lambda_max, torch.float32)
    if iters is not None:
        _need_cuda("iters", iters, torch.int32)
    d = H.shape[0]
    if V0.dim() == 1:
        block = 1
    elif V0.dim() == 2:
        block = V0.shape[0]
    else:
        raise ValueError("V0 must be [d] or [block, d]")
    if V0.shape[-1] != d:
        raise ValueError("V0 vectors must have length d")
    ws, nbytes = _workspace(optima_spectral_norm_workspace_bytes(d, block), ws, H.device,
                           stream)
    _check(_spec(_ptr(H), d, _ptr(V0), int(block), int(max_iters), float(tol), _ptr(ws), nbytes,
                 _ptr(lambda_max), _ptr(iters), _stream(stream)))


SPECTRAL_NOALLOC_MAX_DIM = 16384


def optima_spectral_norm_noalloc(H: torch.Tensor, V0: torch.Tensor, lambda_max: torch.Tensor,
                                 max_iters: int = 1000, tol: float = 1e-6,
                                 iters: torch.Tensor | None = None, stream=None) -> None:
    """optima_spectral_norm with the library's fixed per-device work array
    instead of a workspace: nothing is allocated (d <= SPECTRAL_NOALLOC_MAX_DIM;
    calls that overlap on one device race on that array)."""
    _need_cuda("H", H, torch.float32)
    _need_cuda("V0", V0, torch.float32)
    _need_cuda("lambda_max", lambda_max, torch.float32)
    if iters is not None:
        _need_cuda("iters", iters, torch.int32)
    d = H.shape[0]
    if V0.dim() not in (1, 2) or V0.shape[-1] != d:
        raise ValueError("V0 must be [d] or [block, d]")
    block = 1 if V0.dim() == 1 else V0.shape[0]
    _check(_spec_na(_ptr(H), d, _ptr(V0), int(block), int(max_iters), float(tol),
                    _ptr(lambda_max), _ptr(iters), _stream(stream)))


LANCZOS_MAX_STEPS = 256


def optima_spectral_lanczos_workspace_bytes(d: int, max_steps: int = LANCZOS_MAX_STEPS) -> int:
    return int(_lz_ws(d, max_steps))


def optima_spectral_lanczos(H: torch.Tensor, v0: torch.Tensor, lambda_max: torch.Tensor,
                            max_steps: int = LANCZOS_MAX_STEPS, tol: float = 1e-7,
                            ws: torch.Tensor | None = None, steps: torch.Tensor | None = None,
                            stream=None) -> None:
    """lambda_max(H) by the Lanczos process started from v0 [d]."""
    _need_cuda("H", H, torch.float32)
    _need_cuda("v0", v0, torch.float32)
    _need_cuda("lambda_max", lambda_max, torch.float32)
    if steps is not None:
        _need_cuda("steps", steps, torch.int32)
    d = H.shape[0]
    if v0.dim() != 1 or v0.shape[0] != d:
        raise ValueError("v0 must be [d]")
    ws, nbytes = _workspace(optima_spectral_lanczos_workspace_bytes(d, max_steps), ws, H.device,
                           stream)
    _check(_lz(_ptr(H), d, _ptr(v0), int(max_steps), float(tol), _ptr(ws), nbytes,
               _ptr(lambda_max), _ptr(steps), _stream(stream)))


ACT_NONE = 0
ACT_SILU = 1


def optima_linear_forward_workspace_bytes(n_tok: int, d_in: int, d_out: int) -> int:
    return int(_fwd_ws(n_tok, d_in, d_out))


def optima_linear_forward(X: torch.Tensor, W: torch.Tensor, Y: torch.Tensor | None = None,
                          act: int = ACT_NONE, Y_ref: torch.Tensor | None = None,
                          err_out: torch.Tensor | None = None, ws: torch.Tensor | None = None,
                          stream=None) -> None:
    """Y = act(X W^T) for X [n_tok, d_in] bfloat16 and W [d_out, d_in] float32
    (rounded to bf16 on the device); Y bfloat16 or float32 [n_tok, d_out].
    With Y_ref (float32 [n_tok, d_out]) err_out (float64 [1]) receives the sum
    of (X W^T - Y_ref)^2."""
    _need_cuda("X", X, torch.bfloat16)
    _need_cuda("W", W, torch.float32)
    if X.dim() != 2 or W.dim() != 2 or W.shape[1] != X.shape[1]:
        raise ValueError("X must be [n_tok, d_in] and W [d_out, d_in]")
    n_tok, d_in = X.shape
    d_out = W.shape[0]
    y_dtype = -1
    if Y is not None:
        _need_cuda("Y", Y)
        y_dtype = {torch.bfloat16: DTYPE_BF16, torch.float32: DTYPE_F32}.get(Y.dtype, -1)
        if y_dtype < 0 or Y.shape != (n_tok, d_out):
            raise ValueError("Y must be bfloat16 or float32 [n_tok, d_out]")
    if Y_ref is not None:
        _need_cuda("Y_ref", Y_ref, torch.float32)
        if Y_ref.shape != (n_tok, d_out):
            raise ValueError("Y_ref must be [n_tok, d_out]")
    if (Y_ref is None) != (err_out is None):
        raise ValueError("Y_ref and err_out go together")
    if err_out is not None:
        _need_cuda("err_out", err_out, torch.float64)
    ws, nbytes = _workspace(optima_linear_forward_workspace_bytes(n_tok, d_in, d_out), ws,
                            W.device, stream)
    empty = n_tok == 0  # an empty tensor may report a null address
    _check(_fwd(None if empty else _ptr(X), n_tok, d_in, _ptr(W), d_out, int(act),
                None if empty else _ptr(Y), y_dtype, None if empty else _ptr(Y_ref),
                _ptr(err_out), _ptr(ws), nbytes, _stream(stream)))


MASK_UNSTRUCTURED = 0
MASK_2TO4 = 1


def optima_wanda_mask(W0: torch.Tensor, col_sq: torch.Tensor, mask: torch.Tensor,
                      pattern: int = MASK_UNSTRUCTURED, sparsity: float = 0.5,
                      col_sq_stride: int = 1, stream=None) -> None:
    """Wanda mask of W0 [n_cols, d] into mask [n_cols, d] (uint8, 1 keeps).

    col_sq holds the squared input norms, element i at flat index
    i * col_sq_stride (float32 or float64); the undamped Hessian H [d, d] with
    col_sq_stride = d + 1 passes its diagonal."""
    _need_cuda("W0", W0, torch.float32)
    _need_cuda("col_sq", col_sq)
    _need_cuda("mask", mask, torch.uint8)
    if W0.dim() != 2 or mask.shape != W0.shape:
        raise ValueError("W0 and mask must be [n_cols, d]")
    n, d = W0.shape
    dt = {torch.float32: DTYPE_F32, torch.float64: DTYPE_F64}.get(col_sq.dtype)
    if dt is None:
        raise ValueError("col_sq must be float32 or float64")
    if d > 0 and (d - 1) * int(col_sq_stride) + 1 > col_sq.numel():
        raise ValueError("col_sq too short for d and the stride")
    _check(_mask(_ptr(W0), n, d, _ptr(col_sq), dt, int(col_sq_stride), int(pattern),
                 float(sparsity), _ptr(mask), _stream(stream)))


def optima_qp_workspace_bytes(d: int, n_cols: int) -> int:
    return int(_qp_ws(d, n_cols))


def optima_qp_solve_batched(H: torch.Tensor, lambda_max: torch.Tensor | None, W0: torch.Tensor,
                            mask: torch.Tensor, W_out: torch.Tensor,
                            opts: SolverOpts | None = None, ws: torch.Tensor | None = None,
                            stats: dict | None = None, stream=None) -> dict:
    """Solves every row QP of W0 under `mask`; returns the run totals.

    lambda_max may be None with opts.method == METHOD_CG. stats: optional dict
    of device tensors with keys among iters (int32), restarts (int32),
    converged (uint8), f_initial, f_final, kkt_final (float32).
    """
    _need_cuda("H", H, torch.float32)
    if lambda_max is not None:
        _need_cuda("lambda_max", lambda_max, torch.float32)
    _need_cuda("W0", W0, torch.float32)
    _need_cuda("mask", mask, torch.uint8)
    _need_cuda("W_out", W_out, torch.float32)
    n_cols, d = W0.shape
    if H.shape != (d, d) or mask.shape != W0.shape or W_out.shape != W0.shape:
        raise ValueError("shape mismatch between H, W0, mask and W_out")
    opts = opts or SolverOpts.default()
    if opts.col_scale is not None:
        _need_cuda("opts.col_scale", opts.col_scale, torch.float32)
        if opts.col_scale.numel() != d:
            raise ValueError("opts.col_scale must have d entries")
    ws, nbytes = _workspace(optima_qp_workspace_bytes(d, n_cols), ws, W0.device, stream)
    st = _Stats()
    kinds = {"iters": torch.int32, "restarts": torch.int32, "converged": torch.uint8,
             "f_initial": torch.float32, "f_final": torch.float32, "kkt_final": torch.float32}
    for key, t in (stats or {}).items():
        if key not in kinds:
            raise KeyError(key)
        _need_cuda(key, t, kinds[key])
        if t.numel() != n_cols:
            raise ValueError(f"stats[{key}] must have n_cols entries")
        setattr(st, key, t.data_ptr())
    info = _Info()
    c_opts = opts._c()
    _check(_qp_solve(_ptr(H), d, _ptr(lambda_max), _ptr(W0), _ptr(mask), n_cols,
                     ctypes.byref(c_opts), _ptr(ws), nbytes, _ptr(W_out), ctypes.byref(st),
                     ctypes.byref(info), _stream(stream)))
    return {f[0]: getattr(info, f[0]) for f in _Info._fields_}
