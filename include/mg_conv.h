/*
 * mg_conv.h -- C ABI of the convolution-derivative kernels in libmg.so
 * (MI355X / gfx950).
 *
 * The paper's kernel archetypes include implicit-GEMM convolution kernels and
 * their derivatives (Sec. 3.3); its per-dispatch profile of ResNet-50
 * training attributes most of the step to three derivative shaders, a
 * weight gradient for small outputs, an input gradient and a weight gradient
 * (Sec. 7.3, "Where the remaining time goes").  These entry points compute
 * the two derivatives of a 2-D convolution (no dilation, one group):
 *
 *   data gradient   dX[n][h][w][c] = sum over (k, r, s) with h = p*sh - ph + r,
 *                                    w = q*sw - pw + s of dY[n][p][q][k] W[k][r][s][c]
 *   filter gradient dW[k][r][s][c] = sum over (n, p, q) of
 *                                    dY[n][p][q][k] X[n][p*sh - ph + r][q*sw - pw + s][c]
 *
 * where X is zero outside [0,H) x [0,W) (zero padding).
 *
 * Layouts (channels-last, every tensor contiguous, f32):
 *   X, dX  [N][H][W][C]      dY  [N][P][Q][K]      W, dW  [K][R][S][C]
 *   P = (H + 2*pad_h - R) / stride_h + 1,  Q = (W + 2*pad_w - S) / stride_w + 1
 *
 * Contracts: MG_CONTRACT_STRICT_F32 and MG_CONTRACT_ACCELERATED (whose
 * backward matrices stay f32, Sec. 4.2) both run f32 matrix cores with f32
 * accumulation and give identical results; MG_CONTRACT_FAST_BF16 returns
 * MG_ERR_UNSUPPORTED.  Status codes, the error detail and the per-launch
 * timing hooks are those of mg_attn.h.
 *
 * Ownership, asynchrony and errors: as for mg_attn.h.  The caller owns every
 * buffer; all work is enqueued on `stream` (0 = null stream) and the calls
 * return without waiting; arguments are validated on the host before
 * anything is enqueued (sizes, then pointers: non-null, 16-byte aligned,
 * device memory).  Results are deterministic: no atomics, a fixed order of
 * every sum.
 */
#ifndef MG_CONV_H
#define MG_CONV_H

#include <stddef.h>
#include <stdint.h>

#include "mg_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct mg_conv2d_shape {
    int N, H, W, C;           /* input  [N][H][W][C]  */
    int K, R, S;              /* filter [K][R][S][C]  */
    int stride_h, stride_w;   /* >= 1                 */
    int pad_h, pad_w;         /* >= 0, zero padding   */
} mg_conv2d_shape_t;

/*
 * Workspace.  Each derivative is one implicit GEMM; when its 64x64 output
 * tiles number fewer than 512, the sum behind each output element is split
 * over S = min(ceil(1024 / tiles), floor(ceil(terms / 16) / 16)) workgroups
 * (terms = N*P*Q for the filter gradient; for the data gradient, whose
 * pixels split into stride-parity classes that each sum only the filter taps
 * reaching them, tiles are counted over all classes and terms = the largest
 * class's taps times K), which
 * write f32 partial outputs that a second kernel adds in split order.  The
 * workspace holds those partials: S * (output elements) floats when S > 1,
 * else nothing.  The *_workspace_bytes queries return that size (0 also for
 * invalid arguments); `workspace` is caller-owned device memory of at least
 * that many bytes, may be NULL when the size is 0, and its contents on entry
 * are ignored.
 */
size_t mg_conv2d_bwd_data_workspace_bytes(const mg_conv2d_shape_t *shape,
                                          mg_contract_t contract);
size_t mg_conv2d_bwd_filter_workspace_bytes(const mg_conv2d_shape_t *shape,
                                            mg_contract_t contract);

/*
 * Data gradient dX [N][H][W][C] from dY [N][P][Q][K] and W [K][R][S][C].
 * MG_ERR_INVALID_ARGUMENT for sizes < 1, negative padding, no output
 * position (P < 1 or Q < 1), or any tensor above 2^31-1 bytes;
 * MG_ERR_WORKSPACE for a missing or short workspace.
 */
mg_status_t mg_conv2d_bwd_data(const float *dY, const float *W, float *dX,
                               const mg_conv2d_shape_t *shape, mg_contract_t contract,
                               void *workspace, size_t workspace_bytes,
                               hipStream_t stream);

/*
 * Filter gradient dW [K][R][S][C] from X [N][H][W][C] and dY [N][P][Q][K].
 * Errors as for the data gradient.
 */
mg_status_t mg_conv2d_bwd_filter(const float *X, const float *dY, float *dW,
                                 const mg_conv2d_shape_t *shape, mg_contract_t contract,
                                 void *workspace, size_t workspace_bytes,
                                 hipStream_t stream);

/*
 * Both derivatives in one call (what a training step needs for every layer
 * whose input takes a gradient): the two implicit GEMMs run as one launch,
 * so each fills the GPU the other leaves idle, and their split sums are
 * added by one more launch.  Results are bit for bit those of
 * mg_conv2d_bwd_data and mg_conv2d_bwd_filter.  The workspace holds the data
 * gradient's partials, then, from the next 256-byte boundary, the filter
 * gradient's (mg_conv2d_bwd_workspace_bytes returns the total).
 */
size_t mg_conv2d_bwd_workspace_bytes(const mg_conv2d_shape_t *shape, mg_contract_t contract);

mg_status_t mg_conv2d_bwd(const float *X, const float *W, const float *dY, float *dX,
                          float *dW, const mg_conv2d_shape_t *shape, mg_contract_t contract,
                          void *workspace, size_t workspace_bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* MG_CONV_H */
