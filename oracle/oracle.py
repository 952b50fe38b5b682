"""ctypes front end of the C attention oracle (TEST INFRASTRUCTURE ONLY).

Inputs are converted to float64 copies of the exact stored values (f32, or
bf16 widened to f32 first); outputs are float64.  The C library is compiled
from ``attn_oracle.c`` next to this file with gcc.
"""
import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
ORACLE_SRC = os.path.join(_HERE, "attn_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

CFLAGS = ["-O2", "-std=c99", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
          "-fPIC", "-shared", "-Wall", "-Wextra"]


def build_oracle(src=ORACLE_SRC, out=_LIB_PATH):
    """Compile the oracle with gcc; returns the path of the shared object."""
    tmp = out + ".tmp%d" % os.getpid()
    subprocess.run(["gcc", *CFLAGS, src, "-o", tmp, "-lm"], check=True)
    os.replace(tmp, out)
    return out


def _bind(lib):
    dp = ctypes.POINTER(ctypes.c_double)
    ip = ctypes.POINTER(ctypes.c_int)
    up = ctypes.POINTER(ctypes.c_ubyte)
    ci, cd = ctypes.c_int, ctypes.c_double
    lib.oracle_attn_fwd.argtypes = [dp, dp, dp, ip, ci, ci, ci, ci, ci, ci, cd, up, dp, dp]
    lib.oracle_attn_fwd.restype = ci
    lib.oracle_attn_bwd.argtypes = [dp, dp, dp, dp, ip, ci, ci, ci, ci, ci, ci, cd, up,
                                    dp, dp, dp, dp]
    lib.oracle_attn_bwd.restype = ci
    lib.oracle_attn_bwd_from.argtypes = [dp, dp, dp, dp, dp, dp, ip, ci, ci, ci, ci, ci, ci,
                                         cd, up, dp, dp, dp, dp]
    lib.oracle_attn_bwd_from.restype = ci
    lib.oracle_head_matrices.argtypes = [dp, dp, dp, dp, ip, ci, ci, ci, ci, ci, ci, cd,
                                         ci, ci, dp, dp, dp]
    lib.oracle_head_matrices.restype = ci
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = ci
    return lib


def load_oracle(path=None):
    """Load (building first if absent) the oracle library."""
    global _lib
    with _lock:
        if path is not None:
            return _bind(ctypes.CDLL(path))
        if _lib is None:
            if not os.path.exists(_LIB_PATH) or (
                    os.path.getmtime(_LIB_PATH) < os.path.getmtime(ORACLE_SRC)):
                build_oracle()
            _lib = _bind(ctypes.CDLL(_LIB_PATH))
        return _lib


def _f64(x):
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _ptr(a, ctype=ctypes.c_double):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _prep(Q, K, V, key_len, heads):
    """Q [B,H,Lq,d]; K, V [B,H,Lk,d] (Lq == Lk for self-attention)."""
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    if Q.ndim != 4 or K.ndim != 4 or V.shape != K.shape or \
            K.shape[:2] != Q.shape[:2] or K.shape[3] != Q.shape[3]:
        raise ValueError("Q [B,H,Lq,d], K and V [B,H,Lk,d] expected")
    B, H, Lq, d = Q.shape
    Lk = K.shape[2]
    kl = None
    if key_len is not None:
        kl = np.ascontiguousarray(np.asarray(key_len, dtype=np.int32))
        if kl.shape != (B,):
            raise ValueError("key_len must have shape [B]")
    mask = None
    if heads is not None:
        mask = np.zeros(B * H, dtype=np.uint8)
        for b, h in heads:
            mask[b * H + h] = 1
    return Q, K, V, kl, mask, (B, H, Lq, Lk, d)


def oracle_forward(Q, K, V, causal, scale, key_len=None, heads=None, lib=None):
    """O [B,H,Lq,d] and LSE [B,H,Lq] (natural log) in float64.  K and V may
    have their own length Lk (cross-attention); the causal mask is then
    bottom-right aligned (row i sees keys j <= i + Lk - Lq).

    heads: optional iterable of (b, h) to compute; other heads are NaN.
    """
    lib = lib or load_oracle()
    Q, K, V, kl, mask, (B, H, Lq, Lk, d) = _prep(Q, K, V, key_len, heads)
    O = np.full((B, H, Lq, d), np.nan)
    LSE = np.full((B, H, Lq), np.nan)
    rc = lib.oracle_attn_fwd(_ptr(Q), _ptr(K), _ptr(V),
                             None if kl is None else _ptr(kl, ctypes.c_int),
                             B, H, Lq, Lk, d, int(bool(causal)), float(scale),
                             None if mask is None else _ptr(mask, ctypes.c_ubyte),
                             _ptr(O), _ptr(LSE))
    if rc != 0:
        raise RuntimeError("oracle_attn_fwd failed")
    return O, LSE


def oracle_backward(Q, K, V, dO, causal, scale, key_len=None, heads=None, lib=None):
    """dQ [B,H,Lq,d], dK, dV [B,H,Lk,d] and D [B,H,Lq] in float64
    (recomputing O and LSE)."""
    lib = lib or load_oracle()
    Q, K, V, kl, mask, (B, H, Lq, Lk, d) = _prep(Q, K, V, key_len, heads)
    dO = _f64(dO)
    if dO.shape != Q.shape:
        raise ValueError("dO must have the shape of Q")
    dQ = np.full((B, H, Lq, d), np.nan)
    dK = np.full((B, H, Lk, d), np.nan)
    dV = np.full((B, H, Lk, d), np.nan)
    D = np.full((B, H, Lq), np.nan)
    rc = lib.oracle_attn_bwd(_ptr(Q), _ptr(K), _ptr(V), _ptr(dO),
                             None if kl is None else _ptr(kl, ctypes.c_int),
                             B, H, Lq, Lk, d, int(bool(causal)), float(scale),
                             None if mask is None else _ptr(mask, ctypes.c_ubyte),
                             _ptr(dQ), _ptr(dK), _ptr(dV), _ptr(D))
    if rc != 0:
        raise RuntimeError("oracle_attn_bwd failed")
    return dQ, dK, dV, D


def oracle_backward_from(Q, K, V, O, LSE, dO, causal, scale, key_len=None, heads=None,
                         lib=None):
    """dQ, dK, dV and D of the backward equations evaluated at the given O
    [B,H,Lq,d] and LSE [B,H,Lq] (natural log) instead of the ones the forward
    equations give for Q, K, V: P = exp(S - LSE), D = rowsum(dO * O).  This is
    what a recompute-based backward computes when it consumes the saved
    outputs of a different forward, e.g. the accelerated contract's f32
    backward after its forward on f16-rounded inputs (Sec. 4.2, table of
    arithmetic permissions)."""
    lib = lib or load_oracle()
    Q, K, V, kl, mask, (B, H, Lq, Lk, d) = _prep(Q, K, V, key_len, heads)
    O, LSE, dO = _f64(O), _f64(LSE), _f64(dO)
    if O.shape != Q.shape or dO.shape != Q.shape or LSE.shape != Q.shape[:3]:
        raise ValueError("O and dO must have the shape of Q, LSE [B,H,Lq]")
    dQ = np.full((B, H, Lq, d), np.nan)
    dK = np.full((B, H, Lk, d), np.nan)
    dV = np.full((B, H, Lk, d), np.nan)
    D = np.full((B, H, Lq), np.nan)
    rc = lib.oracle_attn_bwd_from(_ptr(Q), _ptr(K), _ptr(V), _ptr(O), _ptr(LSE), _ptr(dO),
                                  None if kl is None else _ptr(kl, ctypes.c_int),
                                  B, H, Lq, Lk, d, int(bool(causal)), float(scale),
                                  None if mask is None else _ptr(mask, ctypes.c_ubyte),
                                  _ptr(dQ), _ptr(dK), _ptr(dV), _ptr(D))
    if rc != 0:
        raise RuntimeError("oracle_attn_bwd_from failed")
    return dQ, dK, dV, D


def round_to_f16(x):
    """Values of `x` rounded to IEEE binary16 (nearest even, overflow to inf),
    returned as float64: the local input rounding of the paper's practical
    default contract, whose eligible forward matrix inputs are rounded to f16
    before an f32-accumulated product (Sec. 4.2, table of arithmetic
    permissions).  numpy's float16 conversion is the IEEE operation."""
    with np.errstate(over="ignore"):
        return np.asarray(x, dtype=np.float64).astype(np.float16).astype(np.float64)


def oracle_num_threads(lib=None):
    """Threads the oracle's parallel loops use."""
    return int((lib or load_oracle()).oracle_num_threads())


def oracle_head_matrices(Q, K, V, dO, causal, scale, b, h, key_len=None, lib=None):
    """P, dS [Lq,Lk] and Dalt [Lq] (= sum_j P_ij dP_ij) of head (b, h)."""
    lib = lib or load_oracle()
    Q, K, V, kl, _, (B, H, Lq, Lk, d) = _prep(Q, K, V, key_len, None)
    dO = _f64(dO)
    P = np.empty((Lq, Lk))
    dS = np.empty((Lq, Lk))
    Dalt = np.empty(Lq)
    rc = lib.oracle_head_matrices(_ptr(Q), _ptr(K), _ptr(V), _ptr(dO),
                                  None if kl is None else _ptr(kl, ctypes.c_int),
                                  B, H, Lq, Lk, d, int(bool(causal)), float(scale),
                                  int(b), int(h), _ptr(P), _ptr(dS), _ptr(Dalt))
    if rc != 0:
        raise RuntimeError("oracle_head_matrices failed")
    return P, dS, Dalt
