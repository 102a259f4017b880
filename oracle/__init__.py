"""SparseProp CPU oracle (test infrastructure only).

Thin ctypes wrapper around ``sparseprop_oracle.c``: a plain fp64-accumulating
implementation of the sparse linear and convolution passes of SparseProp
(Nikdan et al., ICML 2023, Sec. 3.2 Eq. 1-2 and Sec. 3.3 Eq. 3-5), plus its
own encoders for the two sparse formats and the transposed views.

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the HIP path.
Every value function returns ``(value, abssum)`` in float64, where
``abssum`` is the sum of the absolute values of the terms of each output.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "sparseprop_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (OpenMP, no FMA contraction, no fast-math)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.run(
            ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
             "-Wall", "-shared", "-fPIC", _SRC, "-o", tmp, "-lm"],
            check=True)
        os.replace(tmp, _LIB)
    return _LIB


class ConvShape(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int64), ("IC", ctypes.c_int64),
                ("H", ctypes.c_int64), ("W", ctypes.c_int64),
                ("OC", ctypes.c_int64), ("KH", ctypes.c_int32),
                ("KW", ctypes.c_int32), ("stride_h", ctypes.c_int32),
                ("stride_w", ctypes.c_int32), ("pad_h", ctypes.c_int32),
                ("pad_w", ctypes.c_int32)]


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        _lib = ctypes.CDLL(_LIB)
        _lib.orc_linear_encode.restype = ctypes.c_int64
        _lib.orc_conv_encode.restype = ctypes.c_int64
        _lib.orc_conv_out_hw.restype = ctypes.c_int
        _lib.orc_num_threads.restype = ctypes.c_int
    return _lib


def _p(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def num_threads() -> int:
    return int(_load().orc_num_threads())


# ----------------------------------------------------------------- linear

def linear_encode(mask, W):
    """CSR of the pattern ``mask`` (out x in) with values from ``W``."""
    mask = _c(mask, np.uint8)
    W = _c(W, np.float32)
    out_f, in_f = mask.shape
    nnz_cap = int(np.count_nonzero(mask))
    row_ptr = np.zeros(out_f + 1, np.int32)
    col_idx = np.zeros(max(nnz_cap, 1), np.int32)
    vals = np.zeros(max(nnz_cap, 1), np.float32)
    n = _load().orc_linear_encode(ctypes.c_int64(out_f), ctypes.c_int64(in_f),
                                  _p(mask), _p(W), _p(row_ptr), _p(col_idx),
                                  _p(vals))
    return row_ptr, col_idx[:n].copy(), vals[:n].copy()


def linear_transpose(in_f, out_f, row_ptr, col_idx):
    row_ptr = _c(row_ptr, np.int32)
    col_idx = _c(col_idx, np.int32)
    nnz = int(row_ptr[-1])
    t_col_ptr = np.zeros(in_f + 1, np.int32)
    t_row_idx = np.zeros(max(nnz, 1), np.int32)
    t_perm = np.zeros(max(nnz, 1), np.int32)
    _load().orc_linear_transpose(ctypes.c_int64(in_f), ctypes.c_int64(out_f),
                                 _p(row_ptr), _p(col_idx), _p(t_col_ptr),
                                 _p(t_row_idx), _p(t_perm))
    return t_col_ptr, t_row_idx[:nnz].copy(), t_perm[:nnz].copy()


def linear_fwd(X, row_ptr, col_idx, vals, out_f):
    X = _c(X, np.float32)
    B, in_f = X.shape
    Y = np.zeros((B, out_f), np.float64)
    A = np.zeros((B, out_f), np.float64)
    _load().orc_linear_fwd(_p(X), ctypes.c_int64(B), ctypes.c_int64(in_f),
                           ctypes.c_int64(out_f), _p(_c(row_ptr, np.int32)),
                           _p(_c(col_idx, np.int32)), _p(_c(vals, np.float32)),
                           _p(Y), _p(A))
    return Y, A


def linear_bwd_input(dY, row_ptr, col_idx, vals, in_f):
    dY = _c(dY, np.float32)
    B, out_f = dY.shape
    dX = np.zeros((B, in_f), np.float64)
    A = np.zeros((B, in_f), np.float64)
    _load().orc_linear_bwd_input(_p(dY), ctypes.c_int64(B), ctypes.c_int64(in_f),
                                 ctypes.c_int64(out_f), _p(_c(row_ptr, np.int32)),
                                 _p(_c(col_idx, np.int32)),
                                 _p(_c(vals, np.float32)), _p(dX), _p(A))
    return dX, A


def linear_bwd_weight(dY, X, row_ptr, col_idx):
    dY = _c(dY, np.float32)
    X = _c(X, np.float32)
    B, out_f = dY.shape
    in_f = X.shape[1]
    nnz = int(row_ptr[-1])
    dW = np.zeros(max(nnz, 1), np.float64)
    A = np.zeros(max(nnz, 1), np.float64)
    _load().orc_linear_bwd_weight(_p(dY), _p(X), ctypes.c_int64(B),
                                  ctypes.c_int64(in_f), ctypes.c_int64(out_f),
                                  _p(_c(row_ptr, np.int32)),
                                  _p(_c(col_idx, np.int32)), _p(dW), _p(A))
    return dW[:nnz], A[:nnz]


# ------------------------------------------------------------------- conv

def conv_shape(B, IC, H, W, OC, KH, KW, stride=(1, 1), pad=(0, 0)) -> ConvShape:
    return ConvShape(B, IC, H, W, OC, KH, KW, stride[0], stride[1], pad[0], pad[1])


def conv_out_hw(s: ConvShape):
    oh = ctypes.c_int64()
    ow = ctypes.c_int64()
    rc = _load().orc_conv_out_hw(ctypes.byref(s), ctypes.byref(oh), ctypes.byref(ow))
    if rc:
        raise ValueError("invalid convolution shape")
    return int(oh.value), int(ow.value)


def conv_encode(mask, W):
    """Five-array format of a dense [OC][IC][KH][KW] pattern/values."""
    mask = _c(mask, np.uint8)
    W = _c(W, np.float32)
    OC, IC, KH, KW = mask.shape
    nnz_cap = max(int(np.count_nonzero(mask)), 1)
    w_oc = np.zeros(OC + 1, np.int32)
    w_ic = np.zeros(OC * (IC + 1), np.int16)
    w_x = np.zeros(nnz_cap, np.uint8)
    w_y = np.zeros(nnz_cap, np.uint8)
    w_vals = np.zeros(nnz_cap, np.float32)
    n = _load().orc_conv_encode(ctypes.c_int64(OC), ctypes.c_int64(IC),
                                ctypes.c_int32(KH), ctypes.c_int32(KW),
                                _p(mask), _p(W), _p(w_oc), _p(w_ic), _p(w_x),
                                _p(w_y), _p(w_vals))
    if n < 0:
        raise ValueError("an output channel holds more than 32767 entries")
    return w_oc, w_ic, w_x[:n].copy(), w_y[:n].copy(), w_vals[:n].copy()


def conv_transpose(OC, IC, w_oc, w_ic):
    w_oc = _c(w_oc, np.int32)
    w_ic = _c(w_ic, np.int16)
    nnz = int(w_oc[-1])
    t_ic_ptr = np.zeros(IC + 1, np.int32)
    t_oc = np.zeros(max(nnz, 1), np.int32)
    t_perm = np.zeros(max(nnz, 1), np.int32)
    _load().orc_conv_transpose(ctypes.c_int64(OC), ctypes.c_int64(IC), _p(w_oc),
                               _p(w_ic), _p(t_ic_ptr), _p(t_oc), _p(t_perm))
    return t_ic_ptr, t_oc[:nnz].copy(), t_perm[:nnz].copy()


def conv_fwd(X, s: ConvShape, w_oc, w_ic, w_x, w_y, w_vals):
    X = _c(X, np.float32)
    OH, OW = conv_out_hw(s)
    Y = np.zeros((s.B, s.OC, OH, OW), np.float64)
    A = np.zeros_like(Y)
    _load().orc_conv_fwd(_p(X), ctypes.byref(s), _p(_c(w_oc, np.int32)),
                         _p(_c(w_ic, np.int16)), _p(_c(w_x, np.uint8)),
                         _p(_c(w_y, np.uint8)), _p(_c(w_vals, np.float32)),
                         _p(Y), _p(A))
    return Y, A


def conv_bwd_input(dY, s: ConvShape, w_oc, w_ic, w_x, w_y, w_vals):
    dY = _c(dY, np.float32)
    dX = np.zeros((s.B, s.IC, s.H, s.W), np.float64)
    A = np.zeros_like(dX)
    _load().orc_conv_bwd_input(_p(dY), ctypes.byref(s), _p(_c(w_oc, np.int32)),
                               _p(_c(w_ic, np.int16)), _p(_c(w_x, np.uint8)),
                               _p(_c(w_y, np.uint8)), _p(_c(w_vals, np.float32)),
                               _p(dX), _p(A))
    return dX, A


def conv_bwd_weight(dY, X, s: ConvShape, w_oc, w_ic, w_x, w_y):
    dY = _c(dY, np.float32)
    X = _c(X, np.float32)
    nnz = int(np.asarray(w_oc)[-1])
    dW = np.zeros(max(nnz, 1), np.float64)
    A = np.zeros(max(nnz, 1), np.float64)
    _load().orc_conv_bwd_weight(_p(dY), _p(X), ctypes.byref(s),
                                _p(_c(w_oc, np.int32)), _p(_c(w_ic, np.int16)),
                                _p(_c(w_x, np.uint8)), _p(_c(w_y, np.uint8)),
                                _p(dW), _p(A))
    return dW[:nnz], A[:nnz]
