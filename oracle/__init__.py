"""CPU oracle for the Dyad layer (arXiv 2312.06881) -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path (the ``libdyad`` C-ABI
and its Python binding) never touches it, and it shares no code with them.

The arithmetic lives in ``dyad_oracle.c`` (plain fp64 loops, one loop nest per
weight component, following Sec. 2.2 Eq. 1-10 and Sec. 2.4 Eq. 11-16 of the
paper); this module only marshals numpy float64 arrays into it.

Parity is pinned by the ``-m "not gpu"`` tests against things other than the
oracle itself: a dense weight built from the permutation matrix of Eq. 5,
a gather / batched-product / scatter form built from the index definitions, the
n_dyad=1 collapse to a dense layer, the parameter counts the paper prints,
finite differences for the backward pass, and ``math.erf`` for GELU.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

IT, OT, DT = 0, 1, 2
VARIANTS = {"IT": IT, "OT": OT, "DT": DT}
ACT_NONE, ACT_GELU = 0, 1

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdyad_oracle.so")
SOURCE = os.path.join(_HERE, "dyad_oracle.c")

_lib = None

_D = ctypes.POINTER(ctypes.c_double)
_I64 = ctypes.c_int64


def build_command(out: str = LIB_PATH) -> list[str]:
    """gcc command that builds the oracle library (plain C, fp64, OpenMP)."""
    return ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
            "-o", out, SOURCE, "-lm"]


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"oracle library missing: {LIB_PATH} (run __graft_entry__.build())")
    lib = ctypes.CDLL(LIB_PATH)
    lib.oracle_gelu.restype = ctypes.c_double
    lib.oracle_gelu.argtypes = [ctypes.c_double]
    lib.oracle_gelu_grad.restype = ctypes.c_double
    lib.oracle_gelu_grad.argtypes = [ctypes.c_double]
    lib.oracle_threads.restype = ctypes.c_int
    lib.oracle_gelu_vec.restype = None
    lib.oracle_gelu_vec.argtypes = [_I64, _D, _D]
    lib.oracle_forward.restype = None
    lib.oracle_forward.argtypes = [ctypes.c_int, _I64, _I64, _I64, _I64,
                                   _D, _D, _D, _D, ctypes.c_int, _D, _D]
    lib.oracle_backward_dx.restype = None
    lib.oracle_backward_dx.argtypes = [ctypes.c_int, _I64, _I64, _I64, _I64,
                                       _D, _D, _D, ctypes.c_int, _D, _D]
    lib.oracle_backward_dw.restype = None
    lib.oracle_backward_dw.argtypes = [ctypes.c_int, _I64, _I64, _I64, _I64,
                                       _D, _D, _D, _D, _D]
    lib.oracle_bias_grad.restype = None
    lib.oracle_bias_grad.argtypes = [_I64, _I64, _D, _D]
    lib.oracle_backward_dw_entries.restype = None
    lib.oracle_backward_dw_entries.argtypes = [
        ctypes.c_int, _I64, _I64, _I64, _I64, _D, _D, _I64,
        ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int64),
        ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int64), _D]
    _lib = lib
    return lib


def _f64(a, shape=None):
    a = np.ascontiguousarray(np.asarray(a, dtype=np.float64))
    if shape is not None and a.shape != tuple(shape):
        raise ValueError(f"expected shape {tuple(shape)}, got {a.shape}")
    return a


def _ptr(a):
    return None if a is None else a.ctypes.data_as(_D)


def _variant(v) -> int:
    return VARIANTS[v] if isinstance(v, str) else int(v)


def _check_shape(n_in, n_out, D):
    if D <= 0 or n_in <= 0 or n_out <= 0:
        raise ValueError(f"n_in={n_in}, n_out={n_out}, n_dyad={D} must be positive")


def block_sizes(n_in, n_out, D):
    """(bi, bo): per-block sizes, each width zero-padded up to a multiple of D
    (appendix, caveat on rectangular W)."""
    return -(-n_in // D), -(-n_out // D)


def gelu(x: float) -> float:
    return _load().oracle_gelu(float(x))


def gelu_grad(x: float) -> float:
    return _load().oracle_gelu_grad(float(x))


def gelu_array(x):
    """GELU(x) = x Phi(x) elementwise, fp64, any shape."""
    lib = _load()
    x = _f64(x)
    out = np.empty_like(x)
    lib.oracle_gelu_vec(x.size, _ptr(x), _ptr(out))
    return out


def threads() -> int:
    """OpenMP threads the oracle's parallel loops use."""
    return _load().oracle_threads()


def forward(variant, n_in, n_out, D, X, W1, W2, bias=None, act=ACT_NONE, want_h=False):
    """Y = W X + b per token (optionally GELU); returns Y or (Y, H)."""
    lib = _load()
    _check_shape(n_in, n_out, D)
    X = _f64(X)
    M = X.shape[0]
    X = _f64(X, (M, n_in))
    bi, bo = block_sizes(n_in, n_out, D)
    W1 = _f64(W1, (D, bo, bi))
    W2 = _f64(W2, (D, bo, bi))
    b = None if bias is None else _f64(bias, (n_out,))
    Y = np.empty((M, n_out), np.float64)
    H = np.empty((M, n_out), np.float64) if (want_h and act == ACT_GELU) else None
    lib.oracle_forward(_variant(variant), n_in, n_out, D, M, _ptr(X), _ptr(W1), _ptr(W2),
                       _ptr(b), int(act), _ptr(Y), _ptr(H))
    return (Y, H) if want_h else Y


def backward_dx(variant, n_in, n_out, D, dZ, W1, W2, act_in=ACT_NONE, H_in=None):
    """dX = W^T dZ per token, times GELU'(H_in) when act_in is GELU."""
    lib = _load()
    _check_shape(n_in, n_out, D)
    dZ = _f64(dZ)
    M = dZ.shape[0]
    dZ = _f64(dZ, (M, n_out))
    bi, bo = block_sizes(n_in, n_out, D)
    W1 = _f64(W1, (D, bo, bi))
    W2 = _f64(W2, (D, bo, bi))
    h = None
    if act_in == ACT_GELU:
        if H_in is None:
            raise ValueError("H_in is required when act_in is GELU")
        h = _f64(H_in, (M, n_in))
    dX = np.empty((M, n_in), np.float64)
    lib.oracle_backward_dx(_variant(variant), n_in, n_out, D, M, _ptr(dZ), _ptr(W1), _ptr(W2),
                           int(act_in), _ptr(h), _ptr(dX))
    return dX


def backward_dw(variant, n_in, n_out, D, dZ, X, want_db=True):
    """(dW1, dW2, db) summed over all tokens; db is None unless want_db."""
    lib = _load()
    _check_shape(n_in, n_out, D)
    dZ = _f64(dZ)
    M = dZ.shape[0]
    dZ = _f64(dZ, (M, n_out))
    X = _f64(X, (M, n_in))
    bi, bo = block_sizes(n_in, n_out, D)
    shp = (D, bo, bi)
    dW1 = np.empty(shp, np.float64)
    dW2 = np.empty(shp, np.float64)
    db = np.empty((n_out,), np.float64) if want_db else None
    lib.oracle_backward_dw(_variant(variant), n_in, n_out, D, M, _ptr(dZ), _ptr(X),
                           _ptr(dW1), _ptr(dW2), _ptr(db))
    return dW1, dW2, db


def bias_grad(dZ):
    """db = sum over tokens of dZ."""
    lib = _load()
    dZ = _f64(dZ)
    M, n_out = dZ.shape
    db = np.empty((n_out,), np.float64)
    lib.oracle_bias_grad(n_out, M, _ptr(dZ), _ptr(db))
    return db


def backward_dw_entries(variant, n_in, n_out, D, dZ, X, comp, i, j, k):
    """Selected entries dW_comp[i][j][k] (arrays of equal length), each a full sum over tokens."""
    lib = _load()
    _check_shape(n_in, n_out, D)
    dZ = _f64(dZ)
    M = dZ.shape[0]
    dZ = _f64(dZ, (M, n_out))
    X = _f64(X, (M, n_in))
    comp = np.ascontiguousarray(comp, dtype=np.int32)
    i = np.ascontiguousarray(i, dtype=np.int64)
    j = np.ascontiguousarray(j, dtype=np.int64)
    k = np.ascontiguousarray(k, dtype=np.int64)
    n = comp.shape[0]
    if not (i.shape[0] == j.shape[0] == k.shape[0] == n):
        raise ValueError("entry index arrays differ in length")
    bi, bo = block_sizes(n_in, n_out, D)
    if n and (comp.min() < 1 or comp.max() > 2 or i.min() < 0 or i.max() >= D or
              j.min() < 0 or j.max() >= bo or k.min() < 0 or k.max() >= bi):
        raise ValueError("entry index out of range")
    out = np.empty((n,), np.float64)
    lib.oracle_backward_dw_entries(
        _variant(variant), n_in, n_out, D, M, _ptr(dZ), _ptr(X), n,
        comp.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
        i.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
        j.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
        k.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), _ptr(out))
    return out
