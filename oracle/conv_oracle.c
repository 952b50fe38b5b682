/*
 * conv_oracle.c -- double-precision reference of 2-D convolution and of its
 * two derivatives.  TEST INFRASTRUCTURE ONLY: the test suite, the smoke check
 * and the benchmark's CPU-baseline leg call it; the product library never
 * does, and this file shares no code with it.
 *
 * The paper's kernel archetypes include implicit-GEMM and spatial
 * convolution kernels with their derivatives (Sec. 3.3), and its profile of
 * ResNet-50 training finds the weight-gradient and input-gradient shaders
 * to be most of the step (Sec. 7.3, "Where the remaining time goes").  The
 * paper does not write the operations out; they are the textbook ones, and
 * every function below is that definition evaluated element by element:
 *
 *   forward     Y[n][p][q][k]  = sum_{r,s,c} X[n][p*sh-ph+r][q*sw-pw+s][c] W[k][r][s][c]
 *   data grad   dX[n][h][w][c] = sum_{k,r,s} dY[n][p][q][k] W[k][r][s][c]
 *                                over the (p, q) with p*sh-ph+r = h, q*sw-pw+s = w
 *   filter grad dW[k][r][s][c] = sum_{n,p,q} dY[n][p][q][k] X[n][p*sh-ph+r][q*sw-pw+s][c]
 *
 * with X zero outside [0,H) x [0,W) (zero padding), no dilation, one group.
 * Layouts are channels-last: X, dX [N][H][W][C]; Y, dY [N][P][Q][K];
 * W, dW [K][R][S][C]; P = (H + 2ph - R)/sh + 1, Q = (W + 2pw - S)/sw + 1.
 *
 * No tiling, no reordering into matrix products: each output element is one
 * plain sum.  OpenMP splits the output elements over threads, so results do
 * not depend on the thread count.  Built with -ffp-contract=off.
 */
#include <stddef.h>
#include <stdint.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static int out_len(int in, int pad, int k, int stride) {
    const int span = in + 2 * pad - k;
    return span < 0 ? 0 : span / stride + 1;
}

static int bad_shape(int N, int H, int W, int C, int K, int R, int S, int sh, int sw,
                     int ph, int pw) {
    if (N < 1 || H < 1 || W < 1 || C < 1 || K < 1 || R < 1 || S < 1) return 1;
    if (sh < 1 || sw < 1 || ph < 0 || pw < 0) return 1;
    if (out_len(H, ph, R, sh) < 1 || out_len(W, pw, S, sw) < 1) return 1;
    return 0;
}

int oracle_conv_out_size(int H, int W, int R, int S, int sh, int sw, int ph, int pw,
                         int *P, int *Q) {
    *P = out_len(H, ph, R, sh);
    *Q = out_len(W, pw, S, sw);
    return (*P < 1 || *Q < 1) ? 1 : 0;
}

/* Forward: one sum over the filter taps and input channels per output. */
static double fwd_at(const double *X, const double *Wt, int H, int W, int C, int R, int S,
                     int sh, int sw, int ph, int pw, int n, int p, int q, int k) {
    double acc = 0.0;
    for (int r = 0; r < R; ++r) {
        const int hi = p * sh - ph + r;   /* input row and column under tap (r, s) */
        if (hi < 0 || hi >= H) continue;
        for (int s = 0; s < S; ++s) {
            const int wi = q * sw - pw + s;
            if (wi < 0 || wi >= W) continue;
            const double *x = X + (((size_t)n * H + hi) * W + wi) * C;
            const double *f = Wt + (((size_t)k * R + r) * S + s) * C;
            for (int c = 0; c < C; ++c) acc += x[c] * f[c];
        }
    }
    return acc;
}

/* Data gradient at one input element: every (k, r, s) whose output position
 * (p, q) lands on input (h, w) contributes dY[n][p][q][k] W[k][r][s][c]. */
static double bwd_data_at(const double *dY, const double *Wt, int C, int K, int R, int S,
                          int P, int Q, int sh, int sw, int ph, int pw, int n, int h, int w,
                          int c) {
    double acc = 0.0;
    for (int r = 0; r < R; ++r) {
        const int hp = h + ph - r;        /* = p * sh */
        if (hp < 0 || hp % sh != 0) continue;
        const int p = hp / sh;
        if (p >= P) continue;
        for (int s = 0; s < S; ++s) {
            const int wq = w + pw - s;    /* = q * sw */
            if (wq < 0 || wq % sw != 0) continue;
            const int q = wq / sw;
            if (q >= Q) continue;
            const double *g = dY + (((size_t)n * P + p) * Q + q) * K;
            for (int k = 0; k < K; ++k)
                acc += g[k] * Wt[(((size_t)k * R + r) * S + s) * C + c];
        }
    }
    return acc;
}

/* Filter gradient at one filter element: a sum over every batch item and
 * output position whose receptive field puts tap (r, s) inside the input. */
static double bwd_filter_at(const double *X, const double *dY, int N, int H, int W, int C,
                            int K, int P, int Q, int sh, int sw, int ph, int pw, int k, int r,
                            int s, int c) {
    double acc = 0.0;
    for (int n = 0; n < N; ++n)
        for (int p = 0; p < P; ++p) {
            const int h = p * sh - ph + r;
            if (h < 0 || h >= H) continue;
            for (int q = 0; q < Q; ++q) {
                const int w = q * sw - pw + s;
                if (w < 0 || w >= W) continue;
                acc += dY[(((size_t)n * P + p) * Q + q) * K + k] *
                       X[(((size_t)n * H + h) * W + w) * C + c];
            }
        }
    return acc;
}

int oracle_conv2d_fwd(const double *X, const double *Wt, int N, int H, int W, int C, int K,
                      int R, int S, int sh, int sw, int ph, int pw, double *Y) {
    if (bad_shape(N, H, W, C, K, R, S, sh, sw, ph, pw)) return 1;
    const int P = out_len(H, ph, R, sh), Q = out_len(W, pw, S, sw);
    const long total = (long)N * P * Q * K;
#pragma omp parallel for schedule(static)
    for (long i = 0; i < total; ++i) {
        const int k = (int)(i % K);
        const long pix = i / K;
        const int q = (int)(pix % Q);
        const int p = (int)((pix / Q) % P);
        const int n = (int)(pix / ((long)Q * P));
        Y[i] = fwd_at(X, Wt, H, W, C, R, S, sh, sw, ph, pw, n, p, q, k);
    }
    return 0;
}

int oracle_conv2d_bwd_data(const double *dY, const double *Wt, int N, int H, int W, int C,
                           int K, int R, int S, int sh, int sw, int ph, int pw, double *dX) {
    if (bad_shape(N, H, W, C, K, R, S, sh, sw, ph, pw)) return 1;
    const int P = out_len(H, ph, R, sh), Q = out_len(W, pw, S, sw);
    const long total = (long)N * H * W * C;
#pragma omp parallel for schedule(static)
    for (long i = 0; i < total; ++i) {
        const int c = (int)(i % C);
        const long pix = i / C;
        const int w = (int)(pix % W);
        const int h = (int)((pix / W) % H);
        const int n = (int)(pix / ((long)W * H));
        dX[i] = bwd_data_at(dY, Wt, C, K, R, S, P, Q, sh, sw, ph, pw, n, h, w, c);
    }
    return 0;
}

int oracle_conv2d_bwd_filter(const double *X, const double *dY, int N, int H, int W, int C,
                             int K, int R, int S, int sh, int sw, int ph, int pw, double *dW) {
    if (bad_shape(N, H, W, C, K, R, S, sh, sw, ph, pw)) return 1;
    const int P = out_len(H, ph, R, sh), Q = out_len(W, pw, S, sw);
    const long total = (long)K * R * S * C;
#pragma omp parallel for schedule(dynamic, 16)
    for (long i = 0; i < total; ++i) {
        const int c = (int)(i % C);
        const int s = (int)((i / C) % S);
        const int r = (int)((i / ((long)C * S)) % R);
        const int k = (int)(i / ((long)C * S * R));
        dW[i] = bwd_filter_at(X, dY, N, H, W, C, K, P, Q, sh, sw, ph, pw, k, r, s, c);
    }
    return 0;
}

/* The same sums at selected flat output indices only (for checks of full-size
 * problems): out[j] is element idx[j] of Y (forward), dX (data) or dW (filter). */
int oracle_conv2d_fwd_at(const double *X, const double *Wt, int N, int H, int W, int C, int K,
                         int R, int S, int sh, int sw, int ph, int pw, const int64_t *idx,
                         int nidx, double *out) {
    if (bad_shape(N, H, W, C, K, R, S, sh, sw, ph, pw)) return 1;
    const int P = out_len(H, ph, R, sh), Q = out_len(W, pw, S, sw);
    const int64_t total = (int64_t)N * P * Q * K;
    for (int j = 0; j < nidx; ++j)
        if (idx[j] < 0 || idx[j] >= total) return 2;
#pragma omp parallel for schedule(dynamic, 4)
    for (int j = 0; j < nidx; ++j) {
        const int64_t i = idx[j];
        const int k = (int)(i % K);
        const int64_t pix = i / K;
        const int q = (int)(pix % Q);
        const int p = (int)((pix / Q) % P);
        const int n = (int)(pix / ((int64_t)Q * P));
        out[j] = fwd_at(X, Wt, H, W, C, R, S, sh, sw, ph, pw, n, p, q, k);
    }
    return 0;
}

int oracle_conv2d_bwd_data_at(const double *dY, const double *Wt, int N, int H, int W, int C,
                              int K, int R, int S, int sh, int sw, int ph, int pw,
                              const int64_t *idx, int nidx, double *out) {
    if (bad_shape(N, H, W, C, K, R, S, sh, sw, ph, pw)) return 1;
    const int P = out_len(H, ph, R, sh), Q = out_len(W, pw, S, sw);
    const int64_t total = (int64_t)N * H * W * C;
    for (int j = 0; j < nidx; ++j)
        if (idx[j] < 0 || idx[j] >= total) return 2;
#pragma omp parallel for schedule(dynamic, 4)
    for (int j = 0; j < nidx; ++j) {
        const int64_t i = idx[j];
        const int c = (int)(i % C);
        const int64_t pix = i / C;
        const int w = (int)(pix % W);
        const int h = (int)((pix / W) % H);
        const int n = (int)(pix / ((int64_t)W * H));
        out[j] = bwd_data_at(dY, Wt, C, K, R, S, P, Q, sh, sw, ph, pw, n, h, w, c);
    }
    return 0;
}

int oracle_conv2d_bwd_filter_at(const double *X, const double *dY, int N, int H, int W, int C,
                                int K, int R, int S, int sh, int sw, int ph, int pw,
                                const int64_t *idx, int nidx, double *out) {
    if (bad_shape(N, H, W, C, K, R, S, sh, sw, ph, pw)) return 1;
    const int P = out_len(H, ph, R, sh), Q = out_len(W, pw, S, sw);
    const int64_t total = (int64_t)K * R * S * C;
    for (int j = 0; j < nidx; ++j)
        if (idx[j] < 0 || idx[j] >= total) return 2;
#pragma omp parallel for schedule(dynamic, 4)
    for (int j = 0; j < nidx; ++j) {
        const int64_t i = idx[j];
        const int c = (int)(i % C);
        const int s = (int)((i / C) % S);
        const int r = (int)((i / ((int64_t)C * S)) % R);
        const int k = (int)(i / ((int64_t)C * S * R));
        out[j] = bwd_filter_at(X, dY, N, H, W, C, K, P, Q, sh, sw, ph, pw, k, r, s, c);
    }
    return 0;
}
