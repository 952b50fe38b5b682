/*
 * attn_oracle.c -- CPU oracle for multi-head scaled-dot-product attention,
 * forward and backward, in IEEE double precision.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library calls, links or
 * loads this file; only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark use it.  It shares no code, header, table or helper
 * with the HIP path.
 *
 * What it computes.  The paper builds attention as one mid-level graph node
 * with its own derivative rule (Sec. 3.1) and lowers it to a tiled forward
 * kernel plus a dQ kernel and a fused dK+dV kernel (Sec. 3.3, Sec. 7.3).  The
 * paper does not write the equations out; tiling changes only the order of
 * the floating-point operations, so the oracle is the plain textbook
 * definition of exact attention, evaluated row by row without any tiling,
 * online rescaling or fusion:
 *
 *   allowed(i,j) = (!causal || j <= i + Lk - Lq) && j < key_len[b]
 *   S_ij   = scale * sum_k Q_ik K_jk             (allowed pairs only)
 *   LSE_i  = m_i + ln sum_j exp(S_ij - m_i),  m_i = max_j S_ij
 *   P_ij   = exp(S_ij - LSE_i), exactly 0 for a masked pair
 *   O_i    = sum_j P_ij V_j
 *
 *   D_i    = sum_k dO_ik O_ik
 *   dP_ij  = sum_k dO_ik V_jk
 *   dS_ij  = P_ij (dP_ij - D_i)
 *   dQ_i   = scale * sum_j dS_ij K_j
 *   dK_j   = scale * sum_i dS_ij Q_i
 *   dV_j   = sum_i P_ij dO_i
 *
 * The factor `scale` in dQ and dK comes from the chain rule through
 * S = scale * Q K^T; the finite-difference tests pin its placement.
 *
 * Conventions where the paper is silent:
 *   - a row with no allowed key (only possible with key_len[b] == 0) has
 *     O_i = 0, LSE_i = -inf and contributes nothing to any gradient;
 *   - LSE is in natural-log units;
 *   - causal masking is bottom-right aligned: query row i sees keys up to
 *     i + Lk - Lq, so the last query row sees every key (with Lq == Lk this
 *     is the usual j <= i);
 *   - with Lk < Lq the first Lq - Lk query rows therefore see no key.
 *
 * Layout: Q, O, dO, dQ are [B][H][Lq][d], K, V, dK, dV are [B][H][Lk][d],
 * contiguous with d fastest; LSE and D are [B][H][Lq].  Heads (b,h) are independent; OpenMP runs whole heads per
 * thread, so results do not depend on the thread count.  head_mask (length
 * B*H, nullable) selects the heads to compute; the outputs of unselected
 * heads are left untouched.
 *
 * Build: plain C99, -O2 -ffp-contract=off (no fused multiply-add, so the
 * arithmetic is the written one).
 */
#include <math.h>
#include <stddef.h>
#ifdef _OPENMP
#include <omp.h>
#endif
#include <stdlib.h>
#include <string.h>

static int key_limit(const int *key_len, int b, int Lk)
{
    if (key_len == NULL) return Lk;
    int n = key_len[b];
    if (n < 0) n = 0;
    if (n > Lk) n = Lk;
    return n;
}

/* `off` = Lk - Lq, the bottom-right alignment of the causal mask. */
static int allowed(int i, int j, int causal, int off, int klen)
{
    return (!causal || j <= i + off) && j < klen;
}

static double dot(const double *x, const double *y, int d)
{
    double s = 0.0;
    for (int k = 0; k < d; ++k) s += x[k] * y[k];
    return s;
}

/* Forward pass of one head.  S is scratch of length Lk. */
static void head_forward(const double *Q, const double *K, const double *V,
                         int Lq, int Lk, int d, int causal, int klen, double scale,
                         double *O, double *LSE, double *S)
{
    const int off = Lk - Lq;
    for (int i = 0; i < Lq; ++i) {
        const double *q = Q + (size_t)i * d;
        double *o = O + (size_t)i * d;
        double m = -INFINITY;
        for (int j = 0; j < Lk; ++j) {
            if (!allowed(i, j, causal, off, klen)) continue;
            S[j] = scale * dot(q, K + (size_t)j * d, d);
            if (S[j] > m) m = S[j];
        }
        for (int k = 0; k < d; ++k) o[k] = 0.0;
        if (m == -INFINITY) {           /* no allowed key in this row */
            LSE[i] = -INFINITY;
            continue;
        }
        double sum = 0.0;
        for (int j = 0; j < Lk; ++j)
            if (allowed(i, j, causal, off, klen)) sum += exp(S[j] - m);
        LSE[i] = m + log(sum);
        for (int j = 0; j < Lk; ++j) {
            if (!allowed(i, j, causal, off, klen)) continue;
            double p = exp(S[j] - LSE[i]);
            const double *v = V + (size_t)j * d;
            for (int k = 0; k < d; ++k) o[k] += p * v[k];
        }
    }
}

/* The backward equations of one head evaluated at a given O and LSE (the
 * saved forward outputs a recompute-based backward consumes): P_ij =
 * exp(S_ij - LSE_i) for allowed pairs, D_i = sum_k dO_ik O_ik, and dP, dS,
 * dQ, dK, dV as above.  A row with LSE_i = -inf contributes nothing. */
static void head_backward_from(const double *Q, const double *K, const double *V,
                               const double *O, const double *LSE, const double *dO,
                               int Lq, int Lk, int d, int causal, int klen, double scale,
                               double *dQ, double *dK, double *dV, double *Dout)
{
    const int off = Lk - Lq;
    for (size_t t = 0; t < (size_t)Lq * d; ++t) dQ[t] = 0.0;
    for (size_t t = 0; t < (size_t)Lk * d; ++t) { dK[t] = 0.0; dV[t] = 0.0; }

    for (int i = 0; i < Lq; ++i) {
        const double *q = Q + (size_t)i * d;
        const double *go = dO + (size_t)i * d;
        double *gq = dQ + (size_t)i * d;
        double Di = dot(go, O + (size_t)i * d, d);
        if (Dout) Dout[i] = Di;
        if (LSE[i] == -INFINITY) continue;          /* row has no allowed key */
        for (int j = 0; j < Lk; ++j) {
            if (!allowed(i, j, causal, off, klen)) continue;
            const double *kj = K + (size_t)j * d;
            const double *vj = V + (size_t)j * d;
            double Pij = exp(scale * dot(q, kj, d) - LSE[i]);
            double dPij = dot(go, vj, d);
            double dSij = Pij * (dPij - Di);
            double *gk = dK + (size_t)j * d;
            double *gv = dV + (size_t)j * d;
            for (int k = 0; k < d; ++k) {
                gq[k] += scale * dSij * kj[k];
                gk[k] += scale * dSij * q[k];
                gv[k] += Pij * go[k];
            }
        }
    }
}

/* Backward pass of one head from its inputs.  O and LSE are recomputed here
 * by head_forward (not taken from the caller), so the gradients depend only
 * on Q, K, V, dO.  S is scratch of length Lk, O and LSE scratch of Lq*d and
 * Lq. */
static void head_backward(const double *Q, const double *K, const double *V,
                          const double *dO, int Lq, int Lk, int d, int causal, int klen,
                          double scale, double *dQ, double *dK, double *dV,
                          double *Dout, double *S, double *O, double *LSE)
{
    head_forward(Q, K, V, Lq, Lk, d, causal, klen, scale, O, LSE, S);
    head_backward_from(Q, K, V, O, LSE, dO, Lq, Lk, d, causal, klen, scale, dQ, dK, dV, Dout);
}

static int head_selected(const unsigned char *head_mask, int bh)
{
    return head_mask == NULL || head_mask[bh] != 0;
}

/* Forward over all selected heads.  Returns 0, or -1 on a bad argument or
 * allocation failure. */
int oracle_attn_fwd(const double *Q, const double *K, const double *V,
                    const int *key_len, int B, int H, int Lq, int Lk, int d, int causal,
                    double scale, const unsigned char *head_mask,
                    double *O, double *LSE)
{
    if (B < 1 || H < 1 || Lq < 1 || Lk < 1 || d < 1) return -1;
    int nheads = B * H, failed = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(|: failed)
    for (int bh = 0; bh < nheads; ++bh) {
        if (!head_selected(head_mask, bh)) continue;
        double *S = (double *)malloc(sizeof(double) * (size_t)Lk);
        if (!S) { failed = 1; continue; }
        size_t qo = (size_t)bh * Lq * d, ko = (size_t)bh * Lk * d;
        head_forward(Q + qo, K + ko, V + ko, Lq, Lk, d, causal,
                     key_limit(key_len, bh / H, Lk), scale,
                     O + qo, LSE + (size_t)bh * Lq, S);
        free(S);
    }
    return failed ? -1 : 0;
}

/* Backward over all selected heads.  D (nullable, [B][H][L]) receives
 * D_i = sum_k dO_ik O_ik.  Returns 0, or -1 on a bad argument or allocation
 * failure. */
int oracle_attn_bwd(const double *Q, const double *K, const double *V,
                    const double *dO, const int *key_len, int B, int H, int Lq, int Lk,
                    int d, int causal, double scale,
                    const unsigned char *head_mask,
                    double *dQ, double *dK, double *dV, double *D)
{
    if (B < 1 || H < 1 || Lq < 1 || Lk < 1 || d < 1) return -1;
    int nheads = B * H, failed = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(|: failed)
    for (int bh = 0; bh < nheads; ++bh) {
        if (!head_selected(head_mask, bh)) continue;
        double *S = (double *)malloc(sizeof(double) * (size_t)Lk);
        double *O = (double *)malloc(sizeof(double) * (size_t)Lq * d);
        double *LSE = (double *)malloc(sizeof(double) * (size_t)Lq);
        if (!S || !O || !LSE) { failed = 1; free(S); free(O); free(LSE); continue; }
        size_t qo = (size_t)bh * Lq * d, ko = (size_t)bh * Lk * d;
        head_backward(Q + qo, K + ko, V + ko, dO + qo, Lq, Lk, d, causal,
                      key_limit(key_len, bh / H, Lk), scale,
                      dQ + qo, dK + ko, dV + ko,
                      D ? D + (size_t)bh * Lq : NULL, S, O, LSE);
        free(S); free(O); free(LSE);
    }
    return failed ? -1 : 0;
}

/* Backward over all selected heads at a given O ([B][H][Lq][d]) and LSE
 * ([B][H][Lq]) instead of the ones the forward equations give for Q, K, V:
 * the gradients of a backward that consumes another forward's outputs (the
 * accelerated contract's f32 backward after its rounded-input forward).
 * D as in oracle_attn_bwd.  Returns 0, or -1 on a bad argument. */
int oracle_attn_bwd_from(const double *Q, const double *K, const double *V,
                         const double *O, const double *LSE, const double *dO,
                         const int *key_len, int B, int H, int Lq, int Lk, int d, int causal,
                         double scale, const unsigned char *head_mask,
                         double *dQ, double *dK, double *dV, double *D)
{
    if (B < 1 || H < 1 || Lq < 1 || Lk < 1 || d < 1) return -1;
    int nheads = B * H;
#pragma omp parallel for schedule(dynamic, 1)
    for (int bh = 0; bh < nheads; ++bh) {
        if (!head_selected(head_mask, bh)) continue;
        size_t qo = (size_t)bh * Lq * d, ko = (size_t)bh * Lk * d;
        head_backward_from(Q + qo, K + ko, V + ko, O + qo, LSE + (size_t)bh * Lq, dO + qo,
                           Lq, Lk, d, causal, key_limit(key_len, bh / H, Lk), scale,
                           dQ + qo, dK + ko, dV + ko, D ? D + (size_t)bh * Lq : NULL);
    }
    return 0;
}

/* Full P and dS matrices of one head (b,h), [Lq][Lk] each, for the
 * invariant tests on small shapes.  Masked entries are exactly 0.  Also
 * returns Dalt_i = sum_j P_ij dP_ij, the second form of D (equal to D_i in
 * exact arithmetic because sum_j P_ij V_j = O_i).  Returns 0 or -1. */
int oracle_head_matrices(const double *Q, const double *K, const double *V,
                         const double *dO, const int *key_len, int B, int H,
                         int Lq, int Lk, int d, int causal, double scale, int b, int h,
                         double *P, double *dS, double *Dalt)
{
    if (B < 1 || H < 1 || Lq < 1 || Lk < 1 || d < 1 || b < 0 || b >= B || h < 0 || h >= H)
        return -1;
    size_t qo = ((size_t)b * H + h) * Lq * d, ko = ((size_t)b * H + h) * Lk * d;
    int klen = key_limit(key_len, b, Lk);
    const int off = Lk - Lq;
    double *S = (double *)malloc(sizeof(double) * (size_t)Lk);
    double *O = (double *)malloc(sizeof(double) * (size_t)Lq * d);
    double *LSE = (double *)malloc(sizeof(double) * (size_t)Lq);
    if (!S || !O || !LSE) { free(S); free(O); free(LSE); return -1; }
    const double *q0 = Q + qo, *k0 = K + ko, *v0 = V + ko, *g0 = dO + qo;
    head_forward(q0, k0, v0, Lq, Lk, d, causal, klen, scale, O, LSE, S);
    for (int i = 0; i < Lq; ++i) {
        double Di = dot(g0 + (size_t)i * d, O + (size_t)i * d, d);
        double acc = 0.0;
        for (int j = 0; j < Lk; ++j) {
            double p = 0.0, ds = 0.0;
            if (allowed(i, j, causal, off, klen) && LSE[i] != -INFINITY) {
                p = exp(scale * dot(q0 + (size_t)i * d, k0 + (size_t)j * d, d) - LSE[i]);
                double dp = dot(g0 + (size_t)i * d, v0 + (size_t)j * d, d);
                ds = p * (dp - Di);
                acc += p * dp;
            }
            P[(size_t)i * Lk + j] = p;
            dS[(size_t)i * Lk + j] = ds;
        }
        Dalt[i] = acc;
    }
    free(S); free(O); free(LSE);
    return 0;
}

/* Number of threads the parallel loops above use (1 without OpenMP). */
int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
