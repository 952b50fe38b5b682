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

// Division of 0 <= n < 2^31 by a fixed d >= 1 without a divide:
// n / d == (mulhi(n, mul) + n) >> shift with shift = ceil(log2 d) and
// mul = floor(2^32 (2^shift - d) / d) + 1 (the round-up method of Granlund
// and Montgomery, 1994).
struct FastDiv {
    unsigned mul, shift;
};
FastDiv make_fastdiv(unsigned d);

// Both derivatives are implicit GEMMs: the data gradient over (n, h, w) x c
// summing (r, s, k), the filter gradient over k x (r, s, c) summing
// (n, p, q).  When the output tiles alone leave the GPU mostly idle, the sum
// is split over conv_*_splits(p) workgroups per tile; they write f32
// partials [split][output elements] to `partials`, which
// launch_conv_split_reduce_f32 adds in split order into the output.
int conv_tile_n(const ConvProblem &p);   // output tile width, 64 or 128
int conv_dgrad_splits(const ConvProblem &p);
int conv_wgrad_splits(const ConvProblem &p);
hipError_t launch_conv_dgrad_f32(const ConvProblem &p, const float *dY, const float *Wt,
                                 float *dX, float *partials, hipStream_t s);
hipError_t launch_conv_wgrad_f32(const ConvProblem &p, const float *X, const float *dY,
                                 float *dW, float *partials, hipStream_t s);
hipError_t launch_conv_split_reduce_f32(const float *partials, int nsplit, int total,
                                        float *out, hipStream_t s);

// Both derivatives in one launch (the data gradient's tiles first), and both
// split reductions in one launch.
hipError_t launch_conv_bwd_f32(const ConvProblem &p, const float *X, const float *Wt,
                               const float *dY, float *dX, float *dW, float *dpart,
                               float *wpart, hipStream_t s);
hipError_t launch_conv_split_reduce2_f32(const float *part_a, int nsplit_a, int total_a,
                                         float *out_a, const float *part_b, int nsplit_b,
                                         int total_b, float *out_b, hipStream_t s);

}  // namespace mg
