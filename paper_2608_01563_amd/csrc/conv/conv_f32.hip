// conv_f32.hip -- data and filter gradients of a 2-D convolution as
// implicit GEMMs on the f32 matrix cores (v_mfma_f32_16x16x4_f32).
//
// Neither derivative materialises an unfolded (im2col) matrix: each
// workgroup gathers the operand rows it needs straight from the
// channels-last tensors while it stages them into LDS.
//
//   filter gradient  dW[k][j]  = sum_m dY[m][k] * Xg[m][j]
//       k = output channel, j = (r, s, c) flattened (the [K][R][S][C] order of
//       dW), m = (n, p, q) flattened, Xg[m][j] = X[n][p*sh-ph+r][q*sw-pw+s][c]
//   data gradient    dX[m][c]  = sum_j dYg[m][j] * W[j][c]
//       m = (n, h, w) flattened, j = (r, s, k) flattened with k fastest,
//       W[j][c] = W[k][r][s][c], dYg[m][j] = dY[n][p][q][k] for the output
//       position (p, q) with p*sh-ph+r = h and q*sw-pw+s = w, 0 if none.
//
// Both run 64x64 output tiles on 256 threads: each of the four waves owns a
// 32x32 quarter as 2x2 blocks of 16x16 accumulators, and the reduction
// advances 16 at a time through double-buffered LDS tiles (one barrier per
// step; the global loads of step t+1 are in flight during the products of
// step t).  Operands reach LDS through raw buffer loads whose offset is
// pushed past the end of the buffer for a padded or out-of-range element,
// which reads as zero: the padding of the convolution, the tails of every
// dimension and the positions a strided data gradient skips all become
// zeros without a branch.  Every output element is one fixed-order sum
// (within a workgroup, then across splits in split order): no atomics.
#include "../device_common.h"
#include "conv_launch.h"

namespace mg {
namespace {

constexpr int BM = 64;        // output rows per workgroup
constexpr int BN = 64;        // output columns per workgroup
constexpr int BK = 16;        // reduction step
constexpr int NT = 256;       // four waves
constexpr int LDR = 64 + 16;  // reduction-major tiles: rows 80 floats (16 banks) apart
constexpr int LDM = BK + 4;   // the data gradient's pixel-major A tile: 20 floats per row
constexpr int kOOB = 0x7ffffff0;   // byte offset past every buffer: reads as zero

__device__ __forceinline__ float buffer_load_f32(__amdgpu_buffer_rsrc_t r, int byte_offset) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, byte_offset, 0, 0));
}

// VEC = 4: one 16-byte chunk per thread and step; VEC = 1: four floats,
// 16 apart (used when the contiguous dimension is not a multiple of 4).
template <int VEC>
__device__ __forceinline__ f32x4 load_vec(__amdgpu_buffer_rsrc_t r, const int (&off)[4]) {
    if (VEC == 4) return buffer_load_f32x4(r, off[0]);
    f32x4 v;
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = buffer_load_f32(r, off[e]);
    return v;
}

// 2x2 blocks of v_mfma_f32_16x16x4_f32 over one 16-deep reduction step.
// a(kk, i) and b(kk, jb) return this lane's operand: A[row 16i + l%16][red 4kk + l/16]
// and B[red 4kk + l/16][col 16jb + l%16] of the wave's 32x32 quarter.
template <typename FA, typename FB>
__device__ __forceinline__ void mma_step(f32x4 (&acc)[2][2], FA &&a, FB &&b) {
#pragma unroll
    for (int kk = 0; kk < BK / 4; ++kk) {
        const float a0 = a(kk, 0), a1 = a(kk, 1);
        const float b0 = b(kk, 0), b1 = b(kk, 1);
        acc[0][0] = mfma16x16x4(a0, b0, acc[0][0]);
        acc[0][1] = mfma16x16x4(a0, b1, acc[0][1]);
        acc[1][0] = mfma16x16x4(a1, b0, acc[1][0]);
        acc[1][1] = mfma16x16x4(a1, b1, acc[1][1]);
    }
}

// ------------------------------------------------------- filter gradient --
// Grid: (k tile, j tile, split) with the split fastest.  Split `split` of
// `nsplit` sums the reduction steps [st0, st1) of the N*P*Q positions and
// writes dW (one split) or its partial out[split][K][R*S*C].
template <int VA, int VB>
__global__ __launch_bounds__(NT) void conv_wgrad_f32(const float *__restrict__ X,
                                                     const float *__restrict__ dY,
                                                     float *__restrict__ out, ConvProblem p,
                                                     int tiles_j, int nsplit, int nsteps) {
    __shared__ __attribute__((aligned(16))) float As[2][BK][LDR];   // dY tile, [m][k]
    __shared__ __attribute__((aligned(16))) float Bs[2][BK][LDR];   // X gather, [m][j]

    const int RSC = p.R * p.S * p.C;
    const int PQ = p.P * p.Q;
    const int M = p.N * PQ;
    int bid = blockIdx.x;
    const int split = bid % nsplit;
    bid /= nsplit;
    const int k0 = (bid / tiles_j) * BM;
    const int j0 = (bid % tiles_j) * BN;
    const int st0 = (int)((long)nsteps * split / nsplit);
    const int st1 = (int)((long)nsteps * (split + 1) / nsplit);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int il = lane & 15, g = lane >> 4;
    const int wm = w & 1, wn = w >> 1;
    const int lrow = tid >> 4;   // reduction row this thread stages
    const int lcol = tid & 15;

    const auto rdy = buffer_rsrc(dY, M * p.K * 4);
    const auto rx = buffer_rsrc(X, p.N * p.H * p.W * p.C * 4);

    // Columns this thread stages: k for A, j = (r, s, c) for B (fixed for
    // the whole reduction).
    int ka[4], br[4], bsx[4], boff[4];
    bool bok[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        ka[e] = (VA == 4) ? k0 + 4 * lcol + e : k0 + lcol + 16 * e;
        const int j = (VB == 4) ? j0 + 4 * lcol : j0 + lcol + 16 * e;
        const int c = j % p.C, rs = j / p.C;
        br[e] = rs / p.S;
        bsx[e] = rs - br[e] * p.S;
        boff[e] = (br[e] * p.W + bsx[e]) * p.C + c;
        bok[e] = j < RSC;
    }

    auto load = [&](int st, f32x4 &ra, f32x4 &rb) {
        const int m = st * BK + lrow;
        const bool mok = m < M;
        const int n = m / PQ, pq = m - n * PQ;
        const int pp = pq / p.Q, qq = pq - pp * p.Q;
        const int hb = pp * p.sh - p.ph, wb = qq * p.sw - p.pw;
        const int xbase = ((n * p.H + hb) * p.W + wb) * p.C;
        int oa[4], ob[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            oa[e] = (mok && ka[e] < p.K) ? (m * p.K + ka[e]) * 4 : kOOB;
            const int h = hb + br[e], wi = wb + bsx[e];
            const bool ok = mok && bok[e] && h >= 0 && h < p.H && wi >= 0 && wi < p.W;
            ob[e] = ok ? (xbase + boff[e]) * 4 : kOOB;
        }
        ra = load_vec<VA>(rdy, oa);
        rb = load_vec<VB>(rx, ob);
    };
    auto store = [&](int buf, const f32x4 &ra, const f32x4 &rb) {
        if (VA == 4) {
            *reinterpret_cast<f32x4 *>(&As[buf][lrow][4 * lcol]) = ra;
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) As[buf][lrow][lcol + 16 * e] = ra[e];
        }
        if (VB == 4) {
            *reinterpret_cast<f32x4 *>(&Bs[buf][lrow][4 * lcol]) = rb;
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) Bs[buf][lrow][lcol + 16 * e] = rb[e];
        }
    };

    f32x4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int jb = 0; jb < 2; ++jb) acc[i][jb] = zero4();

    f32x4 ra, rb;
    if (st0 < st1) {
        load(st0, ra, rb);
        store(0, ra, rb);
    }
    __syncthreads();
    for (int st = st0; st < st1; ++st) {
        const int cur = (st - st0) & 1;
        const bool more = st + 1 < st1;
        if (more) load(st + 1, ra, rb);
        mma_step(acc,
                 [&](int kk, int i) { return As[cur][4 * kk + g][32 * wm + 16 * i + il]; },
                 [&](int kk, int jb) { return Bs[cur][4 * kk + g][32 * wn + 16 * jb + il]; });
        if (more) store(cur ^ 1, ra, rb);
        __syncthreads();
    }

    float *dst = out + (size_t)split * p.K * RSC;   // split 0 of 1 is dW itself
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int jb = 0; jb < 2; ++jb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int k = k0 + 32 * wm + 16 * i + 4 * g + r;
                const int j = j0 + 32 * wn + 16 * jb + il;
                if (k < p.K && j < RSC) dst[(size_t)k * RSC + j] = acc[i][jb][r];
            }
}

// dW[i] = sum over splits of partial[split][i], in split order.
__global__ __launch_bounds__(256) void conv_wgrad_reduce_f32(const float *__restrict__ part,
                                                             float *__restrict__ dW,
                                                             int nsplit, int total) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= total) return;
    float s = 0.f;
    for (int k = 0; k < nsplit; ++k) s += part[(size_t)k * total + i];
    dW[i] = s;
}

// --------------------------------------------------------- data gradient --
// Grid: (m tile, c tile) with the c tile fastest.  The whole reduction
// (r, s, k) runs in one workgroup.
template <int VA, int VB>
__global__ __launch_bounds__(NT) void conv_dgrad_f32(const float *__restrict__ dY,
                                                     const float *__restrict__ Wt,
                                                     float *__restrict__ dX, ConvProblem p,
                                                     int tiles_c) {
    __shared__ __attribute__((aligned(16))) float As[2][BM][LDM];   // dY gather, [m][j]
    __shared__ __attribute__((aligned(16))) float Bs[2][BK][LDR];   // W rows, [j][c]

    const int M = p.N * p.H * p.W;
    const int RSK = p.R * p.S * p.K;
    const int nsteps = (RSK + BK - 1) / BK;
    const int m0 = (blockIdx.x / tiles_c) * BM;
    const int c0 = (blockIdx.x % tiles_c) * BN;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int il = lane & 15, g = lane >> 4;
    const int wm = w & 1, wn = w >> 1;

    const auto rdy = buffer_rsrc(dY, p.N * p.P * p.Q * p.K * 4);
    const auto rw = buffer_rsrc(Wt, p.K * p.R * p.S * p.C * 4);

    // A staging: pixel row ar (fixed), reduction columns 4*jq .. 4*jq+3 of a step.
    const int ar = tid >> 2, jq = tid & 3;
    const int m = m0 + ar;
    const bool mok = m < M;
    const int n = m / (p.H * p.W), hw = m - n * (p.H * p.W);
    const int h = hw / p.W, wpix = hw - h * p.W;
    // B staging: reduction row jr of a step, channel columns.
    const int jr = tid >> 4, cc = tid & 15;
    int cb[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) cb[e] = (VB == 4) ? c0 + 4 * cc + e : c0 + cc + 16 * e;

    auto load = [&](int st, f32x4 &ra, f32x4 &rb) {
        int oa[4], ob[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            // dY[n][p][q][k] for reduction index j = (r, s, k), k fastest; a
            // 16-byte chunk (VA == 4, K % 4 == 0) never straddles two taps
            const int j = st * BK + 4 * jq + e;
            const int k = j % p.K, rs = j / p.K;
            const int r = rs / p.S, s = rs - r * p.S;
            const int hp = h + p.ph - r, wq = wpix + p.pw - s;
            const int pp = hp / p.sh, qq = wq / p.sw;
            const bool ok = mok && j < RSK && hp >= 0 && wq >= 0 && pp * p.sh == hp &&
                            qq * p.sw == wq && pp < p.P && qq < p.Q;
            oa[e] = ok ? (((n * p.P + pp) * p.Q + qq) * p.K + k) * 4 : kOOB;
            if (VA == 4) break;
        }
        {
            // W[k][r][s][c] for reduction row j = (r, s, k)
            const int j = st * BK + jr;
            const int k = j % p.K, rs = j / p.K;
            const int row = (k * p.R * p.S + rs) * p.C;   // (k*R + r)*S + s = k*R*S + rs
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                ob[e] = (j < RSK && cb[e] < p.C) ? (row + cb[e]) * 4 : kOOB;
                if (VB == 4) break;
            }
        }
        ra = load_vec<VA>(rdy, oa);
        rb = load_vec<VB>(rw, ob);
    };
    auto store = [&](int buf, const f32x4 &ra, const f32x4 &rb) {
        *reinterpret_cast<f32x4 *>(&As[buf][ar][4 * jq]) = ra;
        if (VB == 4) {
            *reinterpret_cast<f32x4 *>(&Bs[buf][jr][4 * cc]) = rb;
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) Bs[buf][jr][cc + 16 * e] = rb[e];
        }
    };

    f32x4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int jb = 0; jb < 2; ++jb) acc[i][jb] = zero4();

    f32x4 ra, rb;
    load(0, ra, rb);
    store(0, ra, rb);
    __syncthreads();
    for (int st = 0; st < nsteps; ++st) {
        const int cur = st & 1;
        const bool more = st + 1 < nsteps;
        if (more) load(st + 1, ra, rb);
        mma_step(acc,
                 [&](int kk, int i) { return As[cur][32 * wm + 16 * i + il][4 * kk + g]; },
                 [&](int kk, int jb) { return Bs[cur][4 * kk + g][32 * wn + 16 * jb + il]; });
        if (more) store(cur ^ 1, ra, rb);
        __syncthreads();
    }

#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int jb = 0; jb < 2; ++jb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int mo = m0 + 32 * wm + 16 * i + 4 * g + r;
                const int c = c0 + 32 * wn + 16 * jb + il;
                if (mo < M && c < p.C) dX[(size_t)mo * p.C + c] = acc[i][jb][r];
            }
}

int cdiv(int a, int b) { return (a + b - 1) / b; }

}  // namespace

// Split the filter gradient's reduction when its output tiles fill fewer
// than 512 workgroups (two per CU): aim at about 1024 workgroups, with at
// least 16 reduction steps (256 output positions) per split.
int conv_wgrad_splits(const ConvProblem &p) {
    const long tiles = (long)cdiv(p.K, BM) * cdiv(p.R * p.S * p.C, BN);
    if (tiles >= 512) return 1;
    const long steps = cdiv(p.N * p.P * p.Q, BK);
    const long by_grid = (1024 + tiles - 1) / tiles;
    const long by_steps = steps / 16;
    long s = by_grid < by_steps ? by_grid : by_steps;
    return s < 1 ? 1 : (int)s;
}

hipError_t launch_conv_wgrad_f32(const ConvProblem &p, const float *X, const float *dY,
                                 float *dW, float *partials, hipStream_t s) {
    const int ns = conv_wgrad_splits(p);
    if (ns > 1 && partials == nullptr) return hipErrorInvalidValue;
    const int tiles_j = cdiv(p.R * p.S * p.C, BN);
    const int nsteps = cdiv(p.N * p.P * p.Q, BK);
    const dim3 grid(cdiv(p.K, BM) * tiles_j * ns), block(NT);
    float *out = ns > 1 ? partials : dW;
    const bool va = p.K % 4 == 0, vb = p.C % 4 == 0;
    if (va && vb)
        conv_wgrad_f32<4, 4><<<grid, block, 0, s>>>(X, dY, out, p, tiles_j, ns, nsteps);
    else if (va)
        conv_wgrad_f32<4, 1><<<grid, block, 0, s>>>(X, dY, out, p, tiles_j, ns, nsteps);
    else if (vb)
        conv_wgrad_f32<1, 4><<<grid, block, 0, s>>>(X, dY, out, p, tiles_j, ns, nsteps);
    else
        conv_wgrad_f32<1, 1><<<grid, block, 0, s>>>(X, dY, out, p, tiles_j, ns, nsteps);
    return hipGetLastError();
}

hipError_t launch_conv_wgrad_reduce_f32(const ConvProblem &p, const float *partials, float *dW,
                                        hipStream_t s) {
    const int total = p.K * p.R * p.S * p.C;
    conv_wgrad_reduce_f32<<<dim3(cdiv(total, 256)), dim3(256), 0, s>>>(
        partials, dW, conv_wgrad_splits(p), total);
    return hipGetLastError();
}

hipError_t launch_conv_dgrad_f32(const ConvProblem &p, const float *dY, const float *Wt,
                                 float *dX, hipStream_t s) {
    const int tiles_c = cdiv(p.C, BN);
    const dim3 grid(cdiv(p.N * p.H * p.W, BM) * tiles_c), block(NT);
    const bool va = p.K % 4 == 0, vb = p.C % 4 == 0;
    if (va && vb)
        conv_dgrad_f32<4, 4><<<grid, block, 0, s>>>(dY, Wt, dX, p, tiles_c);
    else if (va)
        conv_dgrad_f32<4, 1><<<grid, block, 0, s>>>(dY, Wt, dX, p, tiles_c);
    else if (vb)
        conv_dgrad_f32<1, 4><<<grid, block, 0, s>>>(dY, Wt, dX, p, tiles_c);
    else
        conv_dgrad_f32<1, 1><<<grid, block, 0, s>>>(dY, Wt, dX, p, tiles_c);
    return hipGetLastError();
}

}  // namespace mg
