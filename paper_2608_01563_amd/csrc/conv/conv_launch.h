// conv_launch.h -- host-side launchers of the convolution-derivative kernels.
#pragma once

#include <hip/hip_runtime.h>

namespace mg {

// One 2-D convolution (no dilation, one group), channels-last layouts:
// X [N][H][W][C], dY [N][P][Q][K], W [K][R][S][C].
struct ConvProblem {
    int N, H, W, C, K, R, S;
    int sh, sw, ph, pw;
    int P, Q;
};

// Data gradient dX = implicit GEMM over (n, h, w) x c, summing (r, s, k).
hipError_t launch_conv_dgrad_f32(const ConvProblem &p, const float *dY, const float *Wt,
                                 float *dX, hipStream_t s);

// Filter gradient dW = implicit GEMM over k x (r, s, c), summing (n, p, q).
// When the output tiles alone leave the GPU mostly idle, the sum over
// output positions is split over conv_wgrad_splits(p) workgroups per tile;
// they write f32 partials [split][K*R*S*C] to `partials`, which
// launch_conv_wgrad_reduce_f32 adds in split order.
int conv_wgrad_splits(const ConvProblem &p);
hipError_t launch_conv_wgrad_f32(const ConvProblem &p, const float *X, const float *dY,
                                 float *dW, float *partials, hipStream_t s);
hipError_t launch_conv_wgrad_reduce_f32(const ConvProblem &p, const float *partials, float *dW,
                                        hipStream_t s);

}  // namespace mg
