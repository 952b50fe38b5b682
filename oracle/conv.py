"""ctypes front end of the C convolution oracle (TEST INFRASTRUCTURE ONLY).

Layouts are channels-last: X [N,H,W,C], dY [N,P,Q,K], W [K,R,S,C].  Inputs
are converted to float64 copies of the stored values; outputs are float64.
The C library is compiled from ``conv_oracle.c`` next to this file with gcc.
"""
import ctypes
import os
import subprocess
import threading

import numpy as np

from .oracle import CFLAGS

_HERE = os.path.dirname(os.path.abspath(__file__))
CONV_ORACLE_SRC = os.path.join(_HERE, "conv_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libconv_oracle.so")
_lock = threading.Lock()
_lib = None


def build_conv_oracle(src=CONV_ORACLE_SRC, out=_LIB_PATH):
    tmp = out + ".tmp%d" % os.getpid()
    subprocess.run(["gcc", *CFLAGS, src, "-o", tmp, "-lm"], check=True)
    os.replace(tmp, out)
    return out


def _bind(lib):
    dp = ctypes.POINTER(ctypes.c_double)
    lp = ctypes.POINTER(ctypes.c_int64)
    ip = ctypes.POINTER(ctypes.c_int)
    ci = ctypes.c_int
    shape = [ci] * 11
    lib.oracle_conv_out_size.argtypes = [ci] * 8 + [ip, ip]
    lib.oracle_conv_out_size.restype = ci
    for name in ("oracle_conv2d_fwd", "oracle_conv2d_bwd_data", "oracle_conv2d_bwd_filter"):
        getattr(lib, name).argtypes = [dp, dp, *shape, dp]
        getattr(lib, name).restype = ci
    for name in ("oracle_conv2d_fwd_at", "oracle_conv2d_bwd_data_at",
                 "oracle_conv2d_bwd_filter_at"):
        getattr(lib, name).argtypes = [dp, dp, *shape, lp, ci, dp]
        getattr(lib, name).restype = ci
    return lib


def load_conv_oracle(path=None):
    """Load (building first if absent or stale) the convolution oracle."""
    global _lib
    with _lock:
        if path is not None:
            return _bind(ctypes.CDLL(path))
        if _lib is None:
            if not os.path.exists(_LIB_PATH) or (
                    os.path.getmtime(_LIB_PATH) < os.path.getmtime(CONV_ORACLE_SRC)):
                build_conv_oracle()
            _lib = _bind(ctypes.CDLL(_LIB_PATH))
        return _lib


def _f64(x):
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _p(a, ctype=ctypes.c_double):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def conv_out_size(H, W, R, S, stride=(1, 1), pad=(0, 0)):
    """(P, Q) of a convolution (no dilation)."""
    P = (H + 2 * pad[0] - R) // stride[0] + 1
    Q = (W + 2 * pad[1] - S) // stride[1] + 1
    return P, Q


def _dims(X_shape, W_shape, stride, pad):
    N, H, W, C = X_shape
    K, R, S, C2 = W_shape
    if C2 != C:
        raise ValueError("channel mismatch: X has %d, the filter %d" % (C, C2))
    return (N, H, W, C, K, R, S, int(stride[0]), int(stride[1]), int(pad[0]), int(pad[1]))


def oracle_conv2d_fwd(X, Wt, stride=(1, 1), pad=(0, 0), lib=None):
    """Y [N,P,Q,K] = conv(X [N,H,W,C], W [K,R,S,C]) in float64."""
    lib = lib or load_conv_oracle()
    X, Wt = _f64(X), _f64(Wt)
    dims = _dims(X.shape, Wt.shape, stride, pad)
    P, Q = conv_out_size(dims[1], dims[2], dims[5], dims[6], stride, pad)
    Y = np.full((dims[0], P, Q, dims[4]), np.nan)
    if lib.oracle_conv2d_fwd(_p(X), _p(Wt), *dims, _p(Y)) != 0:
        raise ValueError("invalid convolution shape")
    return Y


def oracle_conv2d_bwd_data(dY, Wt, X_shape, stride=(1, 1), pad=(0, 0), lib=None):
    """dX [N,H,W,C] from dY [N,P,Q,K] and W [K,R,S,C] in float64."""
    lib = lib or load_conv_oracle()
    dY, Wt = _f64(dY), _f64(Wt)
    dims = _dims(X_shape, Wt.shape, stride, pad)
    _check_dy(dY, dims, stride, pad)
    dX = np.full(tuple(X_shape), np.nan)
    if lib.oracle_conv2d_bwd_data(_p(dY), _p(Wt), *dims, _p(dX)) != 0:
        raise ValueError("invalid convolution shape")
    return dX


def oracle_conv2d_bwd_filter(X, dY, W_shape, stride=(1, 1), pad=(0, 0), lib=None):
    """dW [K,R,S,C] from X [N,H,W,C] and dY [N,P,Q,K] in float64."""
    lib = lib or load_conv_oracle()
    X, dY = _f64(X), _f64(dY)
    dims = _dims(X.shape, W_shape, stride, pad)
    _check_dy(dY, dims, stride, pad)
    dW = np.full(tuple(W_shape), np.nan)
    if lib.oracle_conv2d_bwd_filter(_p(X), _p(dY), *dims, _p(dW)) != 0:
        raise ValueError("invalid convolution shape")
    return dW


def oracle_conv2d_fwd_at(X, Wt, flat_idx, stride=(1, 1), pad=(0, 0), lib=None):
    """Elements `flat_idx` (flat indices into Y [N,P,Q,K]) of the forward."""
    lib = lib or load_conv_oracle()
    X, Wt = _f64(X), _f64(Wt)
    dims = _dims(X.shape, Wt.shape, stride, pad)
    idx = np.ascontiguousarray(np.asarray(flat_idx, dtype=np.int64))
    out = np.full(idx.shape, np.nan)
    if lib.oracle_conv2d_fwd_at(_p(X), _p(Wt), *dims, _p(idx, ctypes.c_int64), int(idx.size),
                                _p(out)) != 0:
        raise ValueError("invalid shape or index")
    return out


def oracle_conv2d_bwd_data_at(dY, Wt, X_shape, flat_idx, stride=(1, 1), pad=(0, 0), lib=None):
    """Elements `flat_idx` (flat indices into dX [N,H,W,C]) of the data gradient."""
    lib = lib or load_conv_oracle()
    dY, Wt = _f64(dY), _f64(Wt)
    dims = _dims(X_shape, Wt.shape, stride, pad)
    _check_dy(dY, dims, stride, pad)
    idx = np.ascontiguousarray(np.asarray(flat_idx, dtype=np.int64))
    out = np.full(idx.shape, np.nan)
    if lib.oracle_conv2d_bwd_data_at(_p(dY), _p(Wt), *dims, _p(idx, ctypes.c_int64),
                                     int(idx.size), _p(out)) != 0:
        raise ValueError("invalid shape or index")
    return out


def oracle_conv2d_bwd_filter_at(X, dY, W_shape, flat_idx, stride=(1, 1), pad=(0, 0), lib=None):
    """Elements `flat_idx` (flat indices into dW [K,R,S,C]) of the filter gradient."""
    lib = lib or load_conv_oracle()
    X, dY = _f64(X), _f64(dY)
    dims = _dims(X.shape, W_shape, stride, pad)
    _check_dy(dY, dims, stride, pad)
    idx = np.ascontiguousarray(np.asarray(flat_idx, dtype=np.int64))
    out = np.full(idx.shape, np.nan)
    if lib.oracle_conv2d_bwd_filter_at(_p(X), _p(dY), *dims, _p(idx, ctypes.c_int64),
                                       int(idx.size), _p(out)) != 0:
        raise ValueError("invalid shape or index")
    return out


def _check_dy(dY, dims, stride, pad):
    N, H, W, C, K, R, S = dims[:7]
    P, Q = conv_out_size(H, W, R, S, stride, pad)
    if dY.shape != (N, P, Q, K):
        raise ValueError("dY has shape %s, expected %s" % (dY.shape, (N, P, Q, K)))
