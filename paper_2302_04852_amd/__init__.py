"""Python binding of libsparseprop.so (SparseProp sparse forward/backward
passes on MI355X / gfx950).

Thin ctypes layer: every function has the name of the C entry point it calls
(see include/sparseprop.h), takes torch device tensors for device buffers
and Python ints for sizes, passes the current HIP stream, and raises
``SparsePropError`` on a non-zero status.  It performs no computation of
its own; the library must be built (``paper_2302_04852_amd.build.build()``)
and importing this package fails loudly when it is not.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# SPARSEPROP_LIB selects another build of the same library (e.g. a variant
# compiled with different tuning flags); the default is the in-tree build.
LIB_PATH = os.environ.get("SPARSEPROP_LIB") or os.path.join(_HERE, "libsparseprop.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(LIB_PATH + " is not built: run paper_2302_04852_amd.build.build() "
                      "(or __graft_entry__.build()) first; there is no fallback implementation")
_lib = ctypes.CDLL(LIB_PATH)

SP_OK, SP_ERR_INVALID_ARG, SP_ERR_UNSUPPORTED, SP_ERR_HIP, SP_ERR_WORKSPACE = 0, 1, 2, 3, 4
SP_VARIANT_SPARSE, SP_VARIANT_DENSE = 0, 1
SP_SELECT_ALWAYS_TIME = 1


class SparsePropError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__("%s failed: %s (status %d)" % (fn, sp_status_string(status), status))


class ConvShape(ctypes.Structure):
    """Mirror of sp_conv_shape."""
    _fields_ = [("B", ctypes.c_int64), ("IC", ctypes.c_int64), ("H", ctypes.c_int64),
                ("W", ctypes.c_int64), ("OC", ctypes.c_int64), ("KH", ctypes.c_int32),
                ("KW", ctypes.c_int32), ("stride_h", ctypes.c_int32), ("stride_w", ctypes.c_int32),
                ("pad_h", ctypes.c_int32), ("pad_w", ctypes.c_int32)]


def conv_shape(B, IC, H, W, OC, KH, KW, stride=(1, 1), pad=(0, 0)) -> ConvShape:
    return ConvShape(B, IC, H, W, OC, KH, KW, stride[0], stride[1], pad[0], pad[1])


_I64 = ctypes.c_int64
_I32 = ctypes.c_int32
_P = ctypes.c_void_p
_SZ = ctypes.c_size_t

_SIGS = {
    "sp_linear_encode_rows": [_I64, _I64, _P, _P, _P],
    "sp_linear_encode_fill": [_I64, _I64, _P, _P, _P, _P, _P, _P],
    "sp_linear_transpose_ws": [_I64, _I64, _I64, ctypes.POINTER(_SZ)],
    "sp_linear_transpose": [_I64, _I64, _P, _P, _I64, _P, _P, _P, _P, _SZ, _P],
    "sp_linear_plan_bytes": [_I64, _I64, _I64, ctypes.POINTER(_SZ)],
    "sp_linear_plan": [_I64, _I64, _P, _P, _I64, _P, _SZ, _P],
    "sp_linear_plan_csc": [_P, _I64, _I64, _I64, _P, _P, _P, _P],
    "sp_linear_fwd": [_P, _I64, _I64, _I64, _P, _I64, _P, _P, _P],
    "sp_linear_bwd_input": [_P, _I64, _I64, _I64, _P, _I64, _P, _P, _P],
    "sp_linear_bwd_weight_ws": [_I64, _I64, _I64, _I64, ctypes.POINTER(_SZ)],
    "sp_linear_bwd_weight": [_P, _P, _I64, _I64, _I64, _I64, _P, _P, _P, _SZ, _P],
    "sp_linear_bwd": [_P, _P, _I64, _I64, _I64, _P, _I64, _P, _P, _P, _P, _SZ, _P],
    "sp_linear_validate": [_I64, _I64, _P, _P, _I64],
    "sp_linear_densify": [_I64, _I64, _P, _P, _P, _I64, _P, _P],
    "sp_linear_dense_ws": [_I64, _I64, _I64, ctypes.POINTER(_SZ)],
    "sp_linear_dense_fwd": [_P, _I64, _I64, _I64, _P, _P, _P, _SZ, _P],
    "sp_linear_dense_bwd_input": [_P, _I64, _I64, _I64, _P, _P, _P, _SZ, _P],
    "sp_linear_dense_bwd_weight": [_P, _P, _I64, _I64, _I64, _P, _P, _I64, _P, _P, _SZ, _P],
    "sp_linear_select_ws": [_I64, _I64, _I64, _I64, ctypes.POINTER(_SZ)],
    "sp_linear_select": [_P, _P, _I64, _I64, _I64, _P, _P, _P, _I64, _P, _P, _P, _P, _P, _SZ, _I32, _I32,
                         ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_float), _P],
    "sp_conv_out_hw": [ctypes.POINTER(ConvShape), ctypes.POINTER(_I64), ctypes.POINTER(_I64)],
    "sp_conv_encode_rows": [_I64, _I64, _I32, _I32, _P, _P, _P, _P],
    "sp_conv_encode_fill": [_I64, _I64, _I32, _I32, _P, _P, _P, _P, _P, _P, _P, _P],
    "sp_conv_transpose": [_I64, _I64, _P, _P, _I64, _P, _P, _P, _P],
    "sp_conv_plan_bytes": [ctypes.POINTER(ConvShape), _I64, ctypes.POINTER(_SZ)],
    "sp_conv_plan": [ctypes.POINTER(ConvShape), _P, _P, _P, _P, _I64, _P, _SZ, _P],
    "sp_conv_fwd": [_P, ctypes.POINTER(ConvShape), _P, _I64, _P, _P, _P],
    "sp_conv_bwd_input": [_P, ctypes.POINTER(ConvShape), _P, _I64, _P, _P, _P],
    "sp_conv_bwd_weight_ws": [ctypes.POINTER(ConvShape), _I64, ctypes.POINTER(_SZ)],
    "sp_conv_bwd_weight": [_P, _P, ctypes.POINTER(ConvShape), _I64, _P, _P, _P, _SZ, _P],
    "sp_conv_bwd": [_P, _P, ctypes.POINTER(ConvShape), _P, _I64, _P, _P, _P, _P, _SZ, _P],
    "sp_conv_validate": [_I64, _I64, _I32, _I32, _P, _P, _P, _P, _I64],
    "sp_conv_densify": [ctypes.POINTER(ConvShape), _P, _P, _P, _P, _P, _I64, _P, _P],
    "sp_conv_dense_ws": [ctypes.POINTER(ConvShape), ctypes.POINTER(_SZ)],
    "sp_conv_dense_fwd": [_P, ctypes.POINTER(ConvShape), _P, _P, _P, _SZ, _P],
    "sp_conv_dense_bwd_input": [_P, ctypes.POINTER(ConvShape), _P, _P, _P, _SZ, _P],
    "sp_conv_dense_bwd_weight": [_P, _P, ctypes.POINTER(ConvShape), _P, _P, _P, _P, _I64, _P, _P, _SZ, _P],
    "sp_conv_select_ws": [ctypes.POINTER(ConvShape), _I64, ctypes.POINTER(_SZ)],
    "sp_conv_select": [_P, _P, ctypes.POINTER(ConvShape), _P, _P, _P, _P, _P, _I64, _P, _P, _P, _P, _P, _SZ, _I32,
                       _I32, ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_float), _P],
}

EXPORTED = sorted(_SIGS) + ["sp_status_string", "sp_version"]

for _name, _args in _SIGS.items():
    if hasattr(_lib, _name):
        _f = getattr(_lib, _name)
        _f.argtypes = _args
        _f.restype = ctypes.c_int
_lib.sp_status_string.restype = ctypes.c_char_p
_lib.sp_status_string.argtypes = [ctypes.c_int]
_lib.sp_version.restype = ctypes.c_char_p


def sp_status_string(status: int) -> str:
    return _lib.sp_status_string(int(status)).decode()


def sp_version() -> str:
    return _lib.sp_version().decode()


def _call(name, *args):
    st = getattr(_lib, name)(*args)
    if st != SP_OK:
        raise SparsePropError(name, st)


def _ptr(t):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError("expected a torch tensor")
    if t.numel() and not t.is_cuda:
        raise ValueError("device tensor required (got a CPU tensor)")
    if not t.is_contiguous():
        raise ValueError("contiguous tensor required")
    return _P(t.data_ptr()) if t.numel() else None


def _host_ptr(a):
    """numpy array -> pointer (host-side validation entry points)."""
    return a.ctypes.data_as(_P)


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return _P(stream.cuda_stream)


def _ws(name, *args):
    out = _SZ()
    _call(name, *args, ctypes.byref(out))
    return int(out.value)


# ---------------------------------------------------------------- linear

def sp_linear_encode_rows(out_f, in_f, mask, row_ptr, stream=None):
    _call("sp_linear_encode_rows", out_f, in_f, _ptr(mask), _ptr(row_ptr), _stream(stream))


def sp_linear_encode_fill(out_f, in_f, mask, W, row_ptr, col_idx, vals, stream=None):
    _call("sp_linear_encode_fill", out_f, in_f, _ptr(mask), _ptr(W), _ptr(row_ptr), _ptr(col_idx),
          _ptr(vals), _stream(stream))


def sp_linear_transpose_ws(in_f, out_f, nnz):
    return _ws("sp_linear_transpose_ws", in_f, out_f, nnz)


def sp_linear_transpose(in_f, out_f, row_ptr, col_idx, nnz, t_col_ptr, t_row_idx, t_perm, scratch,
                        stream=None):
    _call("sp_linear_transpose", in_f, out_f, _ptr(row_ptr), _ptr(col_idx), nnz, _ptr(t_col_ptr),
          _ptr(t_row_idx), _ptr(t_perm), _ptr(scratch), scratch.numel() * scratch.element_size(),
          _stream(stream))


def sp_linear_plan_bytes(in_f, out_f, nnz):
    return _ws("sp_linear_plan_bytes", in_f, out_f, nnz)


def sp_linear_plan(in_f, out_f, row_ptr, col_idx, nnz, plan, stream=None):
    _call("sp_linear_plan", in_f, out_f, _ptr(row_ptr), _ptr(col_idx), nnz, _ptr(plan),
          plan.numel() * plan.element_size(), _stream(stream))


def sp_linear_plan_csc(plan, in_f, out_f, nnz, t_col_ptr, t_row_idx, t_perm, stream=None):
    _call("sp_linear_plan_csc", _ptr(plan), in_f, out_f, nnz, _ptr(t_col_ptr), _ptr(t_row_idx),
          _ptr(t_perm), _stream(stream))


def sp_linear_fwd(X, B, in_f, out_f, vals, nnz, plan, Y, stream=None):
    _call("sp_linear_fwd", _ptr(X), B, in_f, out_f, _ptr(vals), nnz, _ptr(plan), _ptr(Y), _stream(stream))


def sp_linear_bwd_input(dY, B, in_f, out_f, vals, nnz, plan, dX, stream=None):
    _call("sp_linear_bwd_input", _ptr(dY), B, in_f, out_f, _ptr(vals), nnz, _ptr(plan), _ptr(dX),
          _stream(stream))


def sp_linear_bwd_weight_ws(B, in_f, out_f, nnz):
    return _ws("sp_linear_bwd_weight_ws", B, in_f, out_f, nnz)


def sp_linear_bwd_weight(dY, X, B, in_f, out_f, nnz, plan, dW, workspace, stream=None):
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _call("sp_linear_bwd_weight", _ptr(dY), _ptr(X), B, in_f, out_f, nnz, _ptr(plan), _ptr(dW),
          _ptr(workspace), nbytes, _stream(stream))


def sp_linear_bwd(dY, X, B, in_f, out_f, vals, nnz, plan, dX, dW, workspace, stream=None):
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _call("sp_linear_bwd", _ptr(dY), _ptr(X), B, in_f, out_f, _ptr(vals), nnz, _ptr(plan), _ptr(dX), _ptr(dW),
          _ptr(workspace), nbytes, _stream(stream))


def _nbytes(t):
    return 0 if t is None else t.numel() * t.element_size()


def sp_linear_densify(out_f, in_f, row_ptr, col_idx, vals, nnz, Wd, stream=None):
    _call("sp_linear_densify", out_f, in_f, _ptr(row_ptr), _ptr(col_idx), _ptr(vals), nnz, _ptr(Wd),
          _stream(stream))


def sp_linear_dense_ws(B, in_f, out_f):
    return _ws("sp_linear_dense_ws", B, in_f, out_f)


def sp_linear_dense_fwd(X, B, in_f, out_f, Wd, Y, workspace, stream=None):
    _call("sp_linear_dense_fwd", _ptr(X), B, in_f, out_f, _ptr(Wd), _ptr(Y), _ptr(workspace), _nbytes(workspace),
          _stream(stream))


def sp_linear_dense_bwd_input(dY, B, in_f, out_f, Wd, dX, workspace, stream=None):
    _call("sp_linear_dense_bwd_input", _ptr(dY), B, in_f, out_f, _ptr(Wd), _ptr(dX), _ptr(workspace),
          _nbytes(workspace), _stream(stream))


def sp_linear_dense_bwd_weight(dY, X, B, in_f, out_f, row_ptr, col_idx, nnz, dW, workspace, stream=None):
    _call("sp_linear_dense_bwd_weight", _ptr(dY), _ptr(X), B, in_f, out_f, _ptr(row_ptr), _ptr(col_idx), nnz,
          _ptr(dW), _ptr(workspace), _nbytes(workspace), _stream(stream))


def sp_linear_select_ws(B, in_f, out_f, nnz):
    return _ws("sp_linear_select_ws", B, in_f, out_f, nnz)


def sp_linear_select(X, dY, B, in_f, out_f, row_ptr, col_idx, vals, nnz, plan, Y, dX, dW, workspace, reps=3,
                     flags=0, stream=None):
    """Returns (variant, [ms_sparse, ms_dense]); waits for the stream."""
    variant = ctypes.c_int(-1)
    ms = (ctypes.c_float * 2)()
    _call("sp_linear_select", _ptr(X), _ptr(dY), B, in_f, out_f, _ptr(row_ptr), _ptr(col_idx), _ptr(vals), nnz,
          _ptr(plan), _ptr(Y), _ptr(dX), _ptr(dW), _ptr(workspace), _nbytes(workspace), reps, flags,
          ctypes.byref(variant), ms, _stream(stream))
    return int(variant.value), [float(ms[0]), float(ms[1])]


def sp_linear_validate(in_f, out_f, row_ptr, col_idx, nnz):
    """Host arrays (numpy int32)."""
    _call("sp_linear_validate", in_f, out_f, _host_ptr(row_ptr), _host_ptr(col_idx), nnz)


# ------------------------------------------------------------------ conv

def sp_conv_out_hw(shape: ConvShape):
    oh, ow = _I64(), _I64()
    _call("sp_conv_out_hw", ctypes.byref(shape), ctypes.byref(oh), ctypes.byref(ow))
    return int(oh.value), int(ow.value)


def sp_conv_encode_rows(OC, IC, KH, KW, mask, w_oc, w_ic, stream=None):
    _call("sp_conv_encode_rows", OC, IC, KH, KW, _ptr(mask), _ptr(w_oc), _ptr(w_ic), _stream(stream))


def sp_conv_encode_fill(OC, IC, KH, KW, mask, W, w_oc, w_ic, w_x, w_y, w_vals, stream=None):
    _call("sp_conv_encode_fill", OC, IC, KH, KW, _ptr(mask), _ptr(W), _ptr(w_oc), _ptr(w_ic), _ptr(w_x),
          _ptr(w_y), _ptr(w_vals), _stream(stream))


def sp_conv_transpose(OC, IC, w_oc, w_ic, nnz, t_ic_ptr, t_oc, t_perm, stream=None):
    _call("sp_conv_transpose", OC, IC, _ptr(w_oc), _ptr(w_ic), nnz, _ptr(t_ic_ptr), _ptr(t_oc),
          _ptr(t_perm), _stream(stream))


def sp_conv_plan_bytes(shape: ConvShape, nnz):
    return _ws("sp_conv_plan_bytes", ctypes.byref(shape), nnz)


def sp_conv_plan(shape: ConvShape, w_oc, w_ic, w_x, w_y, nnz, plan, stream=None):
    _call("sp_conv_plan", ctypes.byref(shape), _ptr(w_oc), _ptr(w_ic), _ptr(w_x), _ptr(w_y), nnz,
          _ptr(plan), plan.numel() * plan.element_size(), _stream(stream))


def sp_conv_fwd(X, shape: ConvShape, w_vals, nnz, plan, Y, stream=None):
    _call("sp_conv_fwd", _ptr(X), ctypes.byref(shape), _ptr(w_vals), nnz, _ptr(plan), _ptr(Y),
          _stream(stream))


def sp_conv_bwd_input(dY, shape: ConvShape, w_vals, nnz, plan, dX, stream=None):
    _call("sp_conv_bwd_input", _ptr(dY), ctypes.byref(shape), _ptr(w_vals), nnz, _ptr(plan), _ptr(dX),
          _stream(stream))


def sp_conv_bwd_weight_ws(shape: ConvShape, nnz):
    return _ws("sp_conv_bwd_weight_ws", ctypes.byref(shape), nnz)


def sp_conv_bwd_weight(dY, X, shape: ConvShape, nnz, plan, dW, workspace, stream=None):
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _call("sp_conv_bwd_weight", _ptr(dY), _ptr(X), ctypes.byref(shape), nnz, _ptr(plan), _ptr(dW),
          _ptr(workspace), nbytes, _stream(stream))


def sp_conv_bwd(dY, X, shape: ConvShape, w_vals, nnz, plan, dX, dW, workspace, stream=None):
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _call("sp_conv_bwd", _ptr(dY), _ptr(X), ctypes.byref(shape), _ptr(w_vals), nnz, _ptr(plan), _ptr(dX), _ptr(dW),
          _ptr(workspace), nbytes, _stream(stream))


def sp_conv_validate(OC, IC, KH, KW, w_oc, w_ic, w_x, w_y, nnz):
    """Host arrays (numpy)."""
    _call("sp_conv_validate", OC, IC, KH, KW, _host_ptr(w_oc), _host_ptr(w_ic), _host_ptr(w_x),
          _host_ptr(w_y), nnz)


def sp_conv_densify(shape: ConvShape, w_oc, w_ic, w_x, w_y, w_vals, nnz, Wd, stream=None):
    _call("sp_conv_densify", ctypes.byref(shape), _ptr(w_oc), _ptr(w_ic), _ptr(w_x), _ptr(w_y), _ptr(w_vals), nnz,
          _ptr(Wd), _stream(stream))


def sp_conv_dense_ws(shape: ConvShape):
    return _ws("sp_conv_dense_ws", ctypes.byref(shape))


def sp_conv_dense_fwd(X, shape: ConvShape, Wd, Y, workspace, stream=None):
    _call("sp_conv_dense_fwd", _ptr(X), ctypes.byref(shape), _ptr(Wd), _ptr(Y), _ptr(workspace), _nbytes(workspace),
          _stream(stream))


def sp_conv_dense_bwd_input(dY, shape: ConvShape, Wd, dX, workspace, stream=None):
    _call("sp_conv_dense_bwd_input", _ptr(dY), ctypes.byref(shape), _ptr(Wd), _ptr(dX), _ptr(workspace),
          _nbytes(workspace), _stream(stream))


def sp_conv_dense_bwd_weight(dY, X, shape: ConvShape, w_oc, w_ic, w_x, w_y, nnz, dW, workspace, stream=None):
    _call("sp_conv_dense_bwd_weight", _ptr(dY), _ptr(X), ctypes.byref(shape), _ptr(w_oc), _ptr(w_ic), _ptr(w_x),
          _ptr(w_y), nnz, _ptr(dW), _ptr(workspace), _nbytes(workspace), _stream(stream))


def sp_conv_select_ws(shape: ConvShape, nnz):
    return _ws("sp_conv_select_ws", ctypes.byref(shape), nnz)


def sp_conv_select(X, dY, shape: ConvShape, w_oc, w_ic, w_x, w_y, w_vals, nnz, plan, Y, dX, dW, workspace, reps=3,
                   flags=0, stream=None):
    """Returns (variant, [ms_sparse, ms_dense]); waits for the stream."""
    variant = ctypes.c_int(-1)
    ms = (ctypes.c_float * 2)()
    _call("sp_conv_select", _ptr(X), _ptr(dY), ctypes.byref(shape), _ptr(w_oc), _ptr(w_ic), _ptr(w_x), _ptr(w_y),
          _ptr(w_vals), nnz, _ptr(plan), _ptr(Y), _ptr(dX), _ptr(dW), _ptr(workspace), _nbytes(workspace), reps,
          flags, ctypes.byref(variant), ms, _stream(stream))
    return int(variant.value), [float(ms[0]), float(ms[1])]
