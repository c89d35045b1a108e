"""Python binding of libdyad, the Dyad layer (arXiv 2312.06881) for MI355X.

Argument marshalling only: every step of the computation runs in the HIP
kernels of ``libdyad.so``; PyTorch supplies device memory and the stream.

Two levels:
  * ``dyad_forward``, ``dyad_backward_dx``, ``dyad_backward_dw``,
    ``dyad_dw_workspace_bytes``, ``dyad_strerror``: the C-ABI of
    ``include/dyad.h`` with the same names and arguments (pointers as ints);
    they return the status code.
  * ``forward``, ``backward_dx``, ``backward_dw``: tensor-level helpers that
    allocate outputs with torch on the inputs' device, call the C-ABI on
    torch's current stream, and raise ``DyadError`` on a non-zero status.

There is no CPU fallback: if ``libdyad.so`` is missing or fails to load, every
call raises.
"""
from __future__ import annotations

import ctypes
import os

import torch  # loaded first: libdyad binds to the HIP runtime torch has loaded

__all__ = [
    "IT", "OT", "DT", "F32", "BF16", "ACT_NONE", "ACT_GELU", "DyadError",
    "dyad_forward", "dyad_forward_noalloc", "dyad_forward_ex", "dyad_backward_dx", "dyad_backward_dw",
    "dyad_backward_dw_ex", "dyad_dw_workspace_bytes", "dyad_dw_workspace_bytes_ex",
    "dyad_strerror", "forward", "backward_dx", "backward_dw", "lib_path",
]

IT, OT, DT = 0, 1, 2
F32, BF16 = 0, 1
ACT_NONE, ACT_GELU = 0, 1
VARIANTS = {"IT": IT, "OT": OT, "DT": DT}
ACTS = {"none": ACT_NONE, "gelu": ACT_GELU}
STATUS = {0: "DYAD_OK", -1: "DYAD_ERR_INVALID_ARG", -2: "DYAD_ERR_SHAPE", -3: "DYAD_ERR_ALIGN",
          -4: "DYAD_ERR_DTYPE", -5: "DYAD_ERR_WORKSPACE", -6: "DYAD_ERR_LAUNCH"}

_PKG = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_PKG, "libdyad.so")
_lib = None

_i64 = ctypes.c_int64
_vp = ctypes.c_void_p
_int = ctypes.c_int


class DyadError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


def lib_path() -> str:
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(f"libdyad.so is not built ({_LIB_PATH}); run "
                           "`python -m paper_2312_06881_amd.build`")
    lib = ctypes.CDLL(_LIB_PATH)
    lib.dyad_forward.restype = _int
    lib.dyad_forward.argtypes = [_int, _i64, _i64, _i64, _i64, _int, _vp, _vp, _vp, _vp, _int,
                                 _vp, _vp, _vp]
    lib.dyad_forward_noalloc.restype = _int
    lib.dyad_forward_noalloc.argtypes = lib.dyad_forward.argtypes
    lib.dyad_backward_dx.restype = _int
    lib.dyad_backward_dx.argtypes = [_int, _i64, _i64, _i64, _i64, _int, _vp, _vp, _vp, _int,
                                     _vp, _vp, _vp]
    lib.dyad_backward_dw.restype = _int
    lib.dyad_backward_dw.argtypes = [_int, _i64, _i64, _i64, _i64, _int, _vp, _vp, _vp, _vp, _vp,
                                     _vp, ctypes.c_size_t, _vp]
    lib.dyad_dw_workspace_bytes.restype = ctypes.c_size_t
    lib.dyad_dw_workspace_bytes.argtypes = [_int, _i64, _i64, _i64, _i64, _int]
    lib.dyad_forward_ex.restype = _int
    lib.dyad_forward_ex.argtypes = [_int, _i64, _i64, _i64, _i64, _int, _int, _vp, _vp, _vp, _vp, _int,
                                    _vp, _vp, _vp]
    lib.dyad_backward_dw_ex.restype = _int
    lib.dyad_backward_dw_ex.argtypes = [_int, _i64, _i64, _i64, _i64, _int, _int, _vp, _vp, _vp, _vp, _vp,
                                        _vp, ctypes.c_size_t, _vp]
    lib.dyad_dw_workspace_bytes_ex.restype = ctypes.c_size_t
    lib.dyad_dw_workspace_bytes_ex.argtypes = [_int, _i64, _i64, _i64, _i64, _int, _int]
    lib.dyad_strerror.restype = ctypes.c_char_p
    lib.dyad_strerror.argtypes = [_int]
    _lib = lib
    return lib


# ---- C-ABI, same names and argument order as include/dyad.h -----------------

def dyad_forward(variant, n_in, n_out, n_dyad, M, dtype, X, W1, W2, bias, act, Y, H, stream) -> int:
    return _load().dyad_forward(variant, n_in, n_out, n_dyad, M, dtype, X, W1, W2, bias, act, Y, H,
                                stream)


def dyad_forward_noalloc(variant, n_in, n_out, n_dyad, M, dtype, X, W1, W2, bias, act, Y, H,
                         stream) -> int:
    return _load().dyad_forward_noalloc(variant, n_in, n_out, n_dyad, M, dtype, X, W1, W2, bias, act,
                                        Y, H, stream)


def dyad_forward_ex(variant, n_in, n_out, n_dyad, M, dtype, act_in, X, W1, W2, bias, act, Y, H,
                    stream) -> int:
    return _load().dyad_forward_ex(variant, n_in, n_out, n_dyad, M, dtype, act_in, X, W1, W2, bias, act,
                                   Y, H, stream)


def dyad_backward_dx(variant, n_in, n_out, n_dyad, M, dtype, dZ, W1, W2, act_in, H_in, dX,
                     stream) -> int:
    return _load().dyad_backward_dx(variant, n_in, n_out, n_dyad, M, dtype, dZ, W1, W2, act_in,
                                    H_in, dX, stream)


def dyad_backward_dw(variant, n_in, n_out, n_dyad, M, dtype, dZ, X, dW1, dW2, dbias, workspace,
                     workspace_bytes, stream) -> int:
    return _load().dyad_backward_dw(variant, n_in, n_out, n_dyad, M, dtype, dZ, X, dW1, dW2, dbias,
                                    workspace, workspace_bytes, stream)


def dyad_dw_workspace_bytes(variant, n_in, n_out, n_dyad, M, dtype) -> int:
    return _load().dyad_dw_workspace_bytes(variant, n_in, n_out, n_dyad, M, dtype)


def dyad_backward_dw_ex(variant, n_in, n_out, n_dyad, M, dtype, act_in, dZ, X, dW1, dW2, dbias, workspace,
                        workspace_bytes, stream) -> int:
    return _load().dyad_backward_dw_ex(variant, n_in, n_out, n_dyad, M, dtype, act_in, dZ, X, dW1, dW2,
                                       dbias, workspace, workspace_bytes, stream)


def dyad_dw_workspace_bytes_ex(variant, n_in, n_out, n_dyad, M, dtype, act_in) -> int:
    return _load().dyad_dw_workspace_bytes_ex(variant, n_in, n_out, n_dyad, M, dtype, act_in)


def dyad_strerror(status: int) -> str:
    return _load().dyad_strerror(status).decode()


# ---- tensor helpers ----------------------------------------------------------

_DT = {torch.float32: F32, torch.bfloat16: BF16}


def _variant(v) -> int:
    return VARIANTS[v] if isinstance(v, str) else int(v)


def _act(a) -> int:
    return ACTS[a] if isinstance(a, str) else int(a)


def _dtype(*ts) -> int:
    dts = {t.dtype for t in ts if t is not None}
    if len(dts) != 1 or next(iter(dts)) not in _DT:
        raise TypeError(f"tensors must share one dtype of float32/bfloat16, got {dts}")
    return _DT[next(iter(dts))]


def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("libdyad takes device tensors")
    if not t.is_contiguous():
        raise ValueError("libdyad takes contiguous tensors")
    return t.data_ptr() or None


def _stream(t):
    return torch.cuda.current_stream(t.device).cuda_stream


def _check(rc: int):
    if rc != 0:
        raise DyadError(rc, dyad_strerror(rc))


def _width(n, D, b, what):
    """A layer width: n if given (it must need exactly b blocks of D), else D * b."""
    if n is None:
        return D * b
    if not (D * (b - 1) < n <= D * b):
        raise ValueError(f"{what}={n} does not fit weight blocks of {b} (n_dyad {D})")
    return n


def forward(x, w1, w2, bias=None, variant="IT", act="none", stash_h=False, n_out=None, act_in="none"):
    """y = W x + b per token (optionally GELU); returns y, or (y, h) with the pre-activation h.

    Weights are [n_dyad, bo, bi]; x is [M, n_in] with n_in padded up to n_dyad * bi.  n_out
    defaults to n_dyad * bo (or bias's length); a smaller n_out needing the same bo blocks is
    a zero-padded layer.  act_in="gelu": the layer's input is GELU(x), x being the previous
    layer's pre-activation, applied inside the kernel (dyad_forward_ex)."""
    D, bo, bi = w1.shape
    M, n_in = x.shape
    _width(n_in, D, bi, "n_in")
    n_out = _width(n_out if n_out is not None or bias is None else bias.shape[0], D, bo, "n_out")
    a = _act(act)
    y = torch.empty((M, n_out), dtype=x.dtype, device=x.device)
    h = torch.empty_like(y) if (stash_h and a == ACT_GELU) else None
    ai = _act(act_in)
    if ai == ACT_NONE:
        _check(dyad_forward(_variant(variant), n_in, n_out, D, M, _dtype(x, w1, w2, bias), _ptr(x),
                            _ptr(w1), _ptr(w2), _ptr(bias), a, _ptr(y), _ptr(h), _stream(x)))
    else:
        _check(dyad_forward_ex(_variant(variant), n_in, n_out, D, M, _dtype(x, w1, w2, bias), ai, _ptr(x),
                               _ptr(w1), _ptr(w2), _ptr(bias), a, _ptr(y), _ptr(h), _stream(x)))
    return (y, h) if stash_h else y


def backward_dx(dz, w1, w2, variant="IT", act_in="none", h_in=None, n_in=None):
    """dX = W^T dz per token, times GELU'(h_in) when act_in is "gelu".  n_in defaults to
    h_in's width, else n_dyad * bi."""
    D, bo, bi = w1.shape
    M, n_out = dz.shape
    _width(n_out, D, bo, "n_out")
    n_in = _width(n_in if n_in is not None or h_in is None else h_in.shape[1], D, bi, "n_in")
    dx = torch.empty((M, n_in), dtype=dz.dtype, device=dz.device)
    _check(dyad_backward_dx(_variant(variant), n_in, n_out, D, M, _dtype(dz, w1, w2, h_in),
                            _ptr(dz), _ptr(w1), _ptr(w2), _act(act_in), _ptr(h_in), _ptr(dx),
                            _stream(dz)))
    return dx


def backward_dw(dz, x, n_dyad, variant="IT", want_db=True, workspace=None, act_in="none"):
    """(dW1, dW2, db) of one layer; db is None unless want_db.  act_in="gelu": the layer's
    input is GELU(x), formed inside the kernel (dyad_backward_dw_ex)."""
    M, n_out = dz.shape
    n_in = x.shape[1]
    D = n_dyad
    dt = _dtype(dz, x)
    shp = (D, -(-n_out // D), -(-n_in // D))   # widths zero-padded up to n_dyad blocks
    dw1 = torch.empty(shp, dtype=dz.dtype, device=dz.device)
    dw2 = torch.empty(shp, dtype=dz.dtype, device=dz.device)
    db = torch.empty((n_out,), dtype=dz.dtype, device=dz.device) if want_db else None
    v = _variant(variant)
    ai = _act(act_in)
    need = dyad_dw_workspace_bytes_ex(v, n_in, n_out, D, M, dt, ai)
    if workspace is None and need:
        workspace = torch.empty((need,), dtype=torch.uint8, device=dz.device)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(dyad_backward_dw_ex(v, n_in, n_out, D, M, dt, ai, _ptr(dz), _ptr(x), _ptr(dw1), _ptr(dw2),
                               _ptr(db), _ptr(workspace), ws_bytes, _stream(dz)))
    return dw1, dw2, db
