"""CPU oracles (f64) for attention forward and backward and for the
convolution derivatives -- TEST INFRASTRUCTURE.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product library never touches it; it shares no code
with the HIP path.  The arithmetic lives in ``attn_oracle.c`` (plain C99,
double precision, no FMA contraction); this module only builds that file and
marshals numpy arrays to it.

Every function follows the textbook definition of exact attention, which the
paper's tiled forward, dQ and fused dK+dV kernels (Sec. 3.3, Sec. 7.3)
compute up to floating-point ordering.  ``conv_oracle.c`` (front end
``oracle.conv``) does the same for 2-D convolution and its data and filter
gradients, the implicit-GEMM derivative kernels of Sec. 3.3 and Sec. 7.3.
"""
from .oracle import (  # noqa: F401
    build_oracle,
    oracle_forward,
    oracle_backward,
    oracle_backward_from,
    oracle_head_matrices,
    oracle_num_threads,
    round_to_f16,
    ORACLE_SRC,
)
from .conv import (  # noqa: F401
    build_conv_oracle,
    conv_out_size,
    oracle_conv2d_fwd,
    oracle_conv2d_fwd_at,
    oracle_conv2d_bwd_data,
    oracle_conv2d_bwd_data_at,
    oracle_conv2d_bwd_filter,
    oracle_conv2d_bwd_filter_at,
    CONV_ORACLE_SRC,
)
