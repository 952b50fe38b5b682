"""MI355X (gfx950) attention forward and backward, and the two derivatives
of a 2-D convolution, behind a C ABI.

The compute path is libmg.so (hand-written HIP kernels, see csrc/,
include/mg_attn.h and include/mg_conv.h); this package is its ctypes binding.  PyTorch is used only
for device memory and streams.
"""
from ._binding import (  # noqa: F401
    ACCELERATED,
    FAST_BF16,
    CONV_HEADER_PATH,
    HEADER_PATH,
    LIB_PATH,
    STRICT_F32,
    MgError,
    attention_backward,
    attention_forward,
    conv2d_backward,
    conv_shape,
    load_library,
    mg_attn_bwd,
    mg_attn_bwd_cross,
    mg_attn_bwd_cross_workspace_bytes,
    mg_attn_bwd_noalloc,
    mg_attn_bwd_workspace_bytes,
    mg_attn_fwd,
    mg_attn_fwd_cross,
    mg_conv2d_bwd,
    mg_conv2d_bwd_data,
    mg_conv2d_bwd_data_workspace_bytes,
    mg_conv2d_bwd_filter,
    mg_conv2d_bwd_filter_workspace_bytes,
    mg_conv2d_bwd_workspace_bytes,
    mg_last_error_detail,
    mg_lds_probe,
    mg_mfma_peak,
    mg_profile_collect,
    mg_profile_enable,
    mg_profile_reset,
    mg_status_string,
)
