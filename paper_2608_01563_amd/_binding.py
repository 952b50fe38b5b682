"""ctypes binding of libmg.so: argument marshalling only.

Every function here checks the torch tensors it is given (device, dtype,
shape, contiguity), passes their device pointers and the current HIP stream
to the C entry point of the same name, and raises MgError on a non-MG_OK
status.  No arithmetic of the attention path happens here; if the library is
missing, load_library() raises instead of falling back to anything.
"""
import ctypes
import os
import threading

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmg.so")
HEADER_PATH = os.path.join(os.path.dirname(HERE), "include", "mg_attn.h")
CONV_HEADER_PATH = os.path.join(os.path.dirname(HERE), "include", "mg_conv.h")

STRICT_F32 = 0
FAST_BF16 = 1
ACCELERATED = 2   # f32 tensors; f16 forward matrix inputs; strict-f32 backward
CONTRACTS = {"strict_f32": STRICT_F32, "fast_bf16": FAST_BF16, "accelerated": ACCELERATED}

MG_OK = 0
STATUS_NAMES = {0: "MG_OK", 1: "MG_ERR_INVALID_ARGUMENT", 2: "MG_ERR_UNSUPPORTED",
                3: "MG_ERR_MISALIGNED", 4: "MG_ERR_WORKSPACE", 5: "MG_ERR_HIP"}

_lock = threading.Lock()
_lib = None


class MgError(RuntimeError):
    def __init__(self, status, detail):
        self.status = status
        self.detail = detail
        super().__init__("%s: %s" % (STATUS_NAMES.get(status, status), detail))


class ConvShape(ctypes.Structure):
    """mg_conv2d_shape_t of mg_conv.h."""
    _fields_ = [(n, ctypes.c_int) for n in
                ("N", "H", "W", "C", "K", "R", "S", "stride_h", "stride_w", "pad_h", "pad_w")]


def _declare(lib):
    vp, c_int, c_float, c_size = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    lib.mg_attn_fwd.argtypes = [vp, vp, vp, vp, vp, vp, c_int, c_int, c_int, c_int, c_int,
                                c_float, c_int, vp]
    lib.mg_attn_fwd.restype = c_int
    lib.mg_attn_bwd_workspace_bytes.argtypes = [c_int, c_int, c_int, c_int, c_int, c_int]
    lib.mg_attn_bwd_workspace_bytes.restype = c_size
    lib.mg_attn_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, c_int, c_int, c_int,
                                c_int, c_int, c_float, c_int, vp, c_size, vp]
    lib.mg_attn_bwd.restype = c_int
    lib.mg_attn_fwd_cross.argtypes = [vp, vp, vp, vp, vp, vp, c_int, c_int, c_int, c_int,
                                      c_int, c_int, c_float, c_int, vp]
    lib.mg_attn_fwd_cross.restype = c_int
    lib.mg_attn_bwd_cross_workspace_bytes.argtypes = [c_int, c_int, c_int, c_int, c_int, c_int,
                                                      c_int]
    lib.mg_attn_bwd_cross_workspace_bytes.restype = c_size
    lib.mg_attn_bwd_cross.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, c_int, c_int,
                                      c_int, c_int, c_int, c_int, c_float, c_int, vp, c_size, vp]
    lib.mg_attn_bwd_cross.restype = c_int
    lib.mg_attn_bwd_noalloc.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, c_int, c_int,
                                        c_int, c_int, c_int, c_int, c_float, c_int, vp]
    lib.mg_attn_bwd_noalloc.restype = c_int
    shp = ctypes.POINTER(ConvShape)
    lib.mg_conv2d_bwd_data_workspace_bytes.argtypes = [shp, c_int]
    lib.mg_conv2d_bwd_data_workspace_bytes.restype = c_size
    lib.mg_conv2d_bwd_data.argtypes = [vp, vp, vp, shp, c_int, vp, c_size, vp]
    lib.mg_conv2d_bwd_data.restype = c_int
    lib.mg_conv2d_bwd_filter_workspace_bytes.argtypes = [shp, c_int]
    lib.mg_conv2d_bwd_filter_workspace_bytes.restype = c_size
    lib.mg_conv2d_bwd_filter.argtypes = [vp, vp, vp, shp, c_int, vp, c_size, vp]
    lib.mg_conv2d_bwd_filter.restype = c_int
    lib.mg_conv2d_bwd_workspace_bytes.argtypes = [shp, c_int]
    lib.mg_conv2d_bwd_workspace_bytes.restype = c_size
    lib.mg_conv2d_bwd.argtypes = [vp, vp, vp, vp, vp, shp, c_int, vp, c_size, vp]
    lib.mg_conv2d_bwd.restype = c_int
    lib.mg_status_string.argtypes = [c_int]
    lib.mg_status_string.restype = ctypes.c_char_p
    lib.mg_last_error_detail.argtypes = []
    lib.mg_last_error_detail.restype = ctypes.c_char_p
    lib.mg_profile_enable.argtypes = [c_int]
    lib.mg_profile_enable.restype = c_int
    lib.mg_profile_collect.argtypes = [ctypes.POINTER(ctypes.c_char_p),
                                       ctypes.POINTER(ctypes.c_int64),
                                       ctypes.POINTER(ctypes.c_double), c_int]
    lib.mg_profile_collect.restype = c_int
    lib.mg_mfma_peak.argtypes = [c_int, c_int, ctypes.POINTER(ctypes.c_double), vp]
    lib.mg_mfma_peak.restype = c_int
    lib.mg_lds_probe.argtypes = [c_int, c_int, c_int, ctypes.POINTER(ctypes.c_double), vp]
    lib.mg_lds_probe.restype = c_int
    lib.mg_profile_reset.argtypes = []
    lib.mg_profile_reset.restype = None
    return lib


def load_library(path=LIB_PATH):
    """Load libmg.so (after torch, so both share one HIP runtime)."""
    global _lib
    with _lock:
        if _lib is None:
            import torch  # noqa: F401  (brings in the HIP runtime the library binds to)
            if not os.path.exists(path):
                raise RuntimeError(
                    "libmg.so is not built (%s); run `python -m "
                    "paper_2608_01563_amd.build` or __graft_entry__.build()" % path)
            _lib = _declare(ctypes.CDLL(path))
        return _lib


def _check(status):
    if status != MG_OK:
        raise MgError(status, load_library().mg_last_error_detail().decode())


def _contract_id(contract):
    if isinstance(contract, str):
        return CONTRACTS[contract]
    return int(contract)


def _stream_handle(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _alloc_stream(stream):
    """Context in which torch allocates memory for work enqueued on `stream`.

    The caching allocator ties a block to the stream current at allocation;
    a block freed by Python is handed out again only to later allocations
    on that stream, which are ordered after the kernels that use it.
    Allocating a workspace or an output on another stream than the one the
    kernels run on would let the next allocation there reuse the block while
    those kernels still write to it."""
    import contextlib
    import torch
    return contextlib.nullcontext() if stream is None else torch.cuda.stream(stream)


def _empty_bytes(nbytes, device, stream):
    import torch
    with _alloc_stream(stream):
        return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _check_tensors(contract, shape, named):
    """Each tensor in `named` must be a contiguous GPU tensor of the
    contract's dtype and of `shape`."""
    import torch
    want = torch.bfloat16 if contract == FAST_BF16 else torch.float32
    for name, t in named:
        if not t.is_cuda:
            raise ValueError("%s must be a GPU tensor" % name)
        if t.dtype != want:
            raise ValueError("%s has dtype %s, contract needs %s" % (name, t.dtype, want))
        if tuple(t.shape) != tuple(shape):
            raise ValueError("%s has shape %s, expected %s" % (name, tuple(t.shape),
                                                               tuple(shape)))
        if not t.is_contiguous():
            raise ValueError("%s must be contiguous" % name)


def _cross_shapes(Q, K):
    """(B, H, Lq, Lk, d) from Q [B,H,Lq,d] and K [B,H,Lk,d]."""
    if Q.dim() != 4 or K.dim() != 4:
        raise ValueError("Q must be [B,H,Lq,d] and K [B,H,Lk,d]")
    B, H, Lq, d = Q.shape
    if tuple(K.shape) != (B, H, K.shape[2], d):
        raise ValueError("K has shape %s, expected [%d,%d,Lk,%d]" % (tuple(K.shape), B, H, d))
    return B, H, Lq, K.shape[2], d


def _check_lse(LSE, shape):
    import torch
    if not LSE.is_cuda or LSE.dtype != torch.float32 or tuple(LSE.shape) != tuple(shape[:3]) \
            or not LSE.is_contiguous():
        raise ValueError("LSE must be a contiguous float32 GPU tensor of shape %s"
                         % (tuple(shape[:3]),))


def _check_key_len(key_len, B):
    import torch
    if key_len is None:
        return
    if not key_len.is_cuda or key_len.dtype != torch.int32 or tuple(key_len.shape) != (B,) \
            or not key_len.is_contiguous():
        raise ValueError("key_len must be a contiguous int32 GPU tensor of shape [%d]" % B)


def mg_attn_fwd(Q, K, V, O, LSE, key_len=None, *, causal, scale, contract=STRICT_F32,
                stream=None):
    """Forward pass into caller-provided O [B,H,L,d] and LSE [B,H,L]."""
    lib = load_library()
    c = _contract_id(contract)
    if Q.dim() != 4:
        raise ValueError("Q must be [B,H,L,d]")
    B, H, L, d = Q.shape
    _check_tensors(c, Q.shape, (("Q", Q), ("K", K), ("V", V), ("O", O)))
    _check_lse(LSE, Q.shape)
    _check_key_len(key_len, B)
    _check(lib.mg_attn_fwd(_ptr(Q), _ptr(K), _ptr(V), _ptr(O), _ptr(LSE), _ptr(key_len),
                           B, H, L, d, int(bool(causal)), float(scale), c,
                           _stream_handle(stream)))


def mg_attn_bwd_workspace_bytes(B, H, L, d, causal, contract=STRICT_F32):
    return int(load_library().mg_attn_bwd_workspace_bytes(B, H, L, d, int(bool(causal)),
                                                          _contract_id(contract)))


def mg_attn_bwd(Q, K, V, O, LSE, dO, dQ, dK, dV, key_len=None, *, causal, scale,
                contract=STRICT_F32, workspace=None, stream=None):
    """Backward pass into caller-provided dQ, dK, dV.  `workspace` is a GPU
    tensor of at least mg_attn_bwd_workspace_bytes(...) bytes; when None, one
    is allocated here with torch (the library itself never allocates)."""
    lib = load_library()
    c = _contract_id(contract)
    if Q.dim() != 4:
        raise ValueError("Q must be [B,H,L,d]")
    B, H, L, d = Q.shape
    _check_tensors(c, Q.shape, (("Q", Q), ("K", K), ("V", V), ("O", O), ("dO", dO),
                                ("dQ", dQ), ("dK", dK), ("dV", dV)))
    _check_lse(LSE, Q.shape)
    _check_key_len(key_len, B)
    need = mg_attn_bwd_workspace_bytes(B, H, L, d, causal, c)
    if workspace is None:
        workspace = _empty_bytes(need, Q.device, stream)
    nbytes = workspace.numel() * workspace.element_size()
    _check(lib.mg_attn_bwd(_ptr(Q), _ptr(K), _ptr(V), _ptr(O), _ptr(LSE), _ptr(dO), _ptr(dQ),
                           _ptr(dK), _ptr(dV), _ptr(key_len), B, H, L, d, int(bool(causal)),
                           float(scale), c, _ptr(workspace), nbytes, _stream_handle(stream)))


def mg_attn_fwd_cross(Q, K, V, O, LSE, key_len=None, *, causal, scale, contract=STRICT_F32,
                      stream=None):
    """Cross-attention forward: Q, O [B,H,Lq,d]; K, V [B,H,Lk,d]; LSE
    [B,H,Lq]; the causal mask is bottom-right aligned (row i sees keys
    j <= i + Lk - Lq)."""
    lib = load_library()
    c = _contract_id(contract)
    B, H, Lq, Lk, d = _cross_shapes(Q, K)
    _check_tensors(c, Q.shape, (("Q", Q), ("O", O)))
    _check_tensors(c, K.shape, (("K", K), ("V", V)))
    _check_lse(LSE, Q.shape)
    _check_key_len(key_len, B)
    _check(lib.mg_attn_fwd_cross(_ptr(Q), _ptr(K), _ptr(V), _ptr(O), _ptr(LSE), _ptr(key_len),
                                 B, H, Lq, Lk, d, int(bool(causal)), float(scale), c,
                                 _stream_handle(stream)))


def mg_attn_bwd_cross_workspace_bytes(B, H, Lq, Lk, d, causal, contract=STRICT_F32):
    return int(load_library().mg_attn_bwd_cross_workspace_bytes(
        B, H, Lq, Lk, d, int(bool(causal)), _contract_id(contract)))


def mg_attn_bwd_cross(Q, K, V, O, LSE, dO, dQ, dK, dV, key_len=None, *, causal, scale,
                      contract=STRICT_F32, workspace=None, stream=None):
    """Cross-attention backward: Q, O, dO, dQ [B,H,Lq,d]; K, V, dK, dV
    [B,H,Lk,d].  `workspace` as for mg_attn_bwd (sized by
    mg_attn_bwd_cross_workspace_bytes)."""
    lib = load_library()
    c = _contract_id(contract)
    B, H, Lq, Lk, d = _cross_shapes(Q, K)
    _check_tensors(c, Q.shape, (("Q", Q), ("O", O), ("dO", dO), ("dQ", dQ)))
    _check_tensors(c, K.shape, (("K", K), ("V", V), ("dK", dK), ("dV", dV)))
    _check_lse(LSE, Q.shape)
    _check_key_len(key_len, B)
    need = mg_attn_bwd_cross_workspace_bytes(B, H, Lq, Lk, d, causal, c)
    if workspace is None:
        workspace = _empty_bytes(need, Q.device, stream)
    nbytes = workspace.numel() * workspace.element_size()
    _check(lib.mg_attn_bwd_cross(_ptr(Q), _ptr(K), _ptr(V), _ptr(O), _ptr(LSE), _ptr(dO),
                                 _ptr(dQ), _ptr(dK), _ptr(dV), _ptr(key_len), B, H, Lq, Lk, d,
                                 int(bool(causal)), float(scale), c, _ptr(workspace), nbytes,
                                 _stream_handle(stream)))


def mg_attn_bwd_noalloc(Q, K, V, O, LSE, dO, dQ, dK, dV, key_len=None, *, causal, scale,
                        contract=STRICT_F32, stream=None):
    """mg_attn_bwd_cross with the library's static scratch array as its
    workspace: nothing is allocated, here or in the library."""
    lib = load_library()
    c = _contract_id(contract)
    B, H, Lq, Lk, d = _cross_shapes(Q, K)
    _check_tensors(c, Q.shape, (("Q", Q), ("O", O), ("dO", dO), ("dQ", dQ)))
    _check_tensors(c, K.shape, (("K", K), ("V", V), ("dK", dK), ("dV", dV)))
    _check_lse(LSE, Q.shape)
    _check_key_len(key_len, B)
    _check(lib.mg_attn_bwd_noalloc(_ptr(Q), _ptr(K), _ptr(V), _ptr(O), _ptr(LSE), _ptr(dO),
                                   _ptr(dQ), _ptr(dK), _ptr(dV), _ptr(key_len), B, H, Lq, Lk,
                                   d, int(bool(causal)), float(scale), c,
                                   _stream_handle(stream)))


def conv_shape(X_shape, W_shape, stride=(1, 1), pad=(0, 0)):
    """ConvShape from X [N,H,W,C], W [K,R,S,C], stride and padding (h, w)."""
    N, H, Wd, C = (int(v) for v in X_shape)
    K, R, S, C2 = (int(v) for v in W_shape)
    if C2 != C:
        raise ValueError("X has %d channels, the filter %d" % (C, C2))
    return ConvShape(N, H, Wd, C, K, R, S, int(stride[0]), int(stride[1]), int(pad[0]),
                     int(pad[1]))


def conv_out_hw(shape):
    return ((shape.H + 2 * shape.pad_h - shape.R) // shape.stride_h + 1,
            (shape.W + 2 * shape.pad_w - shape.S) // shape.stride_w + 1)


def _check_f32(named):
    import torch
    for name, t, want in named:
        if not t.is_cuda or t.dtype != torch.float32 or not t.is_contiguous():
            raise ValueError("%s must be a contiguous float32 GPU tensor" % name)
        if tuple(t.shape) != tuple(want):
            raise ValueError("%s has shape %s, expected %s" % (name, tuple(t.shape), tuple(want)))


def mg_conv2d_bwd_data_workspace_bytes(X_shape, W_shape, stride=(1, 1), pad=(0, 0),
                                       contract=STRICT_F32):
    shape = conv_shape(X_shape, W_shape, stride, pad)
    return int(load_library().mg_conv2d_bwd_data_workspace_bytes(ctypes.byref(shape),
                                                                 _contract_id(contract)))


def mg_conv2d_bwd_data(dY, W, dX, *, stride=(1, 1), pad=(0, 0), contract=STRICT_F32,
                       workspace=None, stream=None):
    """Data gradient into caller-provided dX [N,H,W,C] (channels-last).
    `workspace` as for mg_attn_bwd (allocated here with torch when None and
    needed)."""
    lib = load_library()
    shape = conv_shape(dX.shape, W.shape, stride, pad)
    P, Q = conv_out_hw(shape)
    _check_f32((("dY", dY, (shape.N, P, Q, shape.K)), ("W", W, tuple(W.shape)),
                ("dX", dX, tuple(dX.shape))))
    need = mg_conv2d_bwd_data_workspace_bytes(dX.shape, W.shape, stride, pad, contract)
    if workspace is None and need > 0:
        workspace = _empty_bytes(need, dX.device, stream)
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib.mg_conv2d_bwd_data(_ptr(dY), _ptr(W), _ptr(dX), ctypes.byref(shape),
                                  _contract_id(contract), _ptr(workspace), nbytes,
                                  _stream_handle(stream)))


def mg_conv2d_bwd_filter_workspace_bytes(X_shape, W_shape, stride=(1, 1), pad=(0, 0),
                                         contract=STRICT_F32):
    shape = conv_shape(X_shape, W_shape, stride, pad)
    return int(load_library().mg_conv2d_bwd_filter_workspace_bytes(ctypes.byref(shape),
                                                                   _contract_id(contract)))


def mg_conv2d_bwd_filter(X, dY, dW, *, stride=(1, 1), pad=(0, 0), contract=STRICT_F32,
                         workspace=None, stream=None):
    """Filter gradient into caller-provided dW [K,R,S,C].  `workspace` as for
    mg_attn_bwd (allocated here with torch when None and needed)."""
    lib = load_library()
    shape = conv_shape(X.shape, dW.shape, stride, pad)
    P, Q = conv_out_hw(shape)
    _check_f32((("X", X, tuple(X.shape)), ("dY", dY, (shape.N, P, Q, shape.K)),
                ("dW", dW, tuple(dW.shape))))
    need = mg_conv2d_bwd_filter_workspace_bytes(X.shape, dW.shape, stride, pad, contract)
    if workspace is None and need > 0:
        workspace = _empty_bytes(need, X.device, stream)
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib.mg_conv2d_bwd_filter(_ptr(X), _ptr(dY), _ptr(dW), ctypes.byref(shape),
                                    _contract_id(contract), _ptr(workspace), nbytes,
                                    _stream_handle(stream)))


def mg_conv2d_bwd_workspace_bytes(X_shape, W_shape, stride=(1, 1), pad=(0, 0),
                                  contract=STRICT_F32):
    shape = conv_shape(X_shape, W_shape, stride, pad)
    return int(load_library().mg_conv2d_bwd_workspace_bytes(ctypes.byref(shape),
                                                            _contract_id(contract)))


def mg_conv2d_bwd(X, W, dY, dX, dW, *, stride=(1, 1), pad=(0, 0), contract=STRICT_F32,
                  workspace=None, stream=None):
    """Both derivatives in one call into caller-provided dX and dW."""
    lib = load_library()
    shape = conv_shape(X.shape, W.shape, stride, pad)
    P, Q = conv_out_hw(shape)
    _check_f32((("X", X, tuple(X.shape)), ("W", W, tuple(W.shape)),
                ("dY", dY, (shape.N, P, Q, shape.K)), ("dX", dX, tuple(X.shape)),
                ("dW", dW, tuple(W.shape))))
    need = mg_conv2d_bwd_workspace_bytes(X.shape, W.shape, stride, pad, contract)
    if workspace is None and need > 0:
        workspace = _empty_bytes(need, X.device, stream)
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib.mg_conv2d_bwd(_ptr(X), _ptr(W), _ptr(dY), _ptr(dX), _ptr(dW),
                             ctypes.byref(shape), _contract_id(contract), _ptr(workspace),
                             nbytes, _stream_handle(stream)))


def mg_status_string(status):
    return load_library().mg_status_string(int(status)).decode()


def mg_last_error_detail():
    return load_library().mg_last_error_detail().decode()


def mg_profile_enable(enable=True):
    _check(load_library().mg_profile_enable(int(bool(enable))))


def mg_profile_reset():
    load_library().mg_profile_reset()


MFMA_KINDS = {"f32": 0, "bf16": 1, "f16": 2}


def mg_mfma_peak(kind="f32", iters=20000, stream=None):
    """Sustained dense TFLOP/s of the device's matrix cores for `kind`
    ("f32", "bf16" or "f16"), measured by the library's probe kernel; waits
    for the probe to finish."""
    out = ctypes.c_double(0.0)
    _check(load_library().mg_mfma_peak(MFMA_KINDS[kind], int(iters), ctypes.byref(out),
                                       _stream_handle(stream)))
    return out.value


def mg_lds_probe(pattern, row_bytes, iters=4000, stream=None):
    """LDS clocks per read instruction per CU for one of the kernels' access
    patterns (0-6, see mg_attn.h) on rows of `row_bytes` bytes; waits."""
    out = ctypes.c_double(0.0)
    _check(load_library().mg_lds_probe(int(pattern), int(row_bytes), int(iters),
                                       ctypes.byref(out), _stream_handle(stream)))
    return out.value


def mg_profile_collect(max_entries=32):
    """{kernel name: (launches, total_ms)} accumulated since the last reset."""
    lib = load_library()
    names = (ctypes.c_char_p * max_entries)()
    launches = (ctypes.c_int64 * max_entries)()
    total = (ctypes.c_double * max_entries)()
    n = lib.mg_profile_collect(names, launches, total, max_entries)
    if n < 0:
        raise MgError(5, lib.mg_last_error_detail().decode())
    return {names[i].decode(): (int(launches[i]), float(total[i]))
            for i in range(min(n, max_entries))}


# ------------------------------------------------------------ conveniences --
def attention_forward(Q, K, V, *, causal, scale, key_len=None, contract=None, stream=None):
    """Allocate O and LSE with torch and run the forward; returns (O, LSE).
    K and V may have their own sequence length (cross-attention)."""
    import torch
    c = _contract_id(contract) if contract is not None else (
        FAST_BF16 if Q.dtype == torch.bfloat16 else STRICT_F32)
    with _alloc_stream(stream):
        O = torch.empty_like(Q)
        LSE = torch.empty(Q.shape[:3], dtype=torch.float32, device=Q.device)
    mg_attn_fwd_cross(Q, K, V, O, LSE, key_len, causal=causal, scale=scale, contract=c,
                      stream=stream)
    return O, LSE


def attention_backward(Q, K, V, O, LSE, dO, *, causal, scale, key_len=None, contract=None,
                       workspace=None, stream=None):
    """Allocate dQ, dK, dV with torch and run the backward; returns (dQ, dK,
    dV).  K and V may have their own sequence length (cross-attention)."""
    import torch
    c = _contract_id(contract) if contract is not None else (
        FAST_BF16 if Q.dtype == torch.bfloat16 else STRICT_F32)
    with _alloc_stream(stream):
        dQ, dK, dV = torch.empty_like(Q), torch.empty_like(K), torch.empty_like(V)
    mg_attn_bwd_cross(Q, K, V, O, LSE, dO, dQ, dK, dV, key_len, causal=causal, scale=scale,
                      contract=c, workspace=workspace, stream=stream)
    return dQ, dK, dV


def conv2d_backward(X, W, dY, *, stride=(1, 1), pad=(0, 0), contract=STRICT_F32, stream=None,
                    need_input_grad=True):
    """Allocate with torch and run both convolution derivatives; returns
    (dX or None, dW).  Layouts: X [N,H,W,C], W [K,R,S,C], dY [N,P,Q,K]."""
    import torch
    with _alloc_stream(stream):
        dW = torch.empty_like(W)
        dX = torch.empty_like(X) if need_input_grad else None
    if not need_input_grad:
        mg_conv2d_bwd_filter(X, dY, dW, stride=stride, pad=pad, contract=contract,
                             stream=stream)
        return None, dW
    mg_conv2d_bwd(X, W, dY, dX, dW, stride=stride, pad=pad, contract=contract, stream=stream)
    return dX, dW
