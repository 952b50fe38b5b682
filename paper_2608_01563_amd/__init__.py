"""MI355X (gfx950) attention forward and backward behind a C ABI.

The compute path is libmgattn.so (hand-written HIP kernels, see csrc/ and
include/mg_attn.h); this package is its ctypes binding.  PyTorch is used only
for device memory and streams.
"""
from ._binding import (  # noqa: F401
    ACCELERATED,
    FAST_BF16,
    HEADER_PATH,
    LIB_PATH,
    STRICT_F32,
    MgError,
    attention_backward,
    attention_forward,
    load_library,
    mg_attn_bwd,
    mg_attn_bwd_cross,
    mg_attn_bwd_cross_workspace_bytes,
    mg_attn_bwd_workspace_bytes,
    mg_attn_fwd,
    mg_attn_fwd_cross,
    mg_last_error_detail,
    mg_profile_collect,
    mg_profile_enable,
    mg_profile_reset,
    mg_status_string,
)
