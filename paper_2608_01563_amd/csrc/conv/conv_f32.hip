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
// advances BK (32) at a time through double-buffered LDS tiles (one barrier
// per step; the global loads of steps t+1 and t+2 are in flight, in two
// register sets, during the products of step t).  Operands reach LDS through raw buffer loads whose offset is
// pushed past the end of the buffer for a padded or out-of-range element,
// which reads as zero: the padding of the convolution, the tails of every
// dimension and the positions a strided data gradient skips all become
// zeros without a branch.  Every output element is one fixed-order sum
// (within a workgroup, then across splits in split order): no atomics.
#include "../device_common.h"
#include "conv_launch.h"

namespace mg {
namespace {

#ifndef MG_CONV_BK
#define MG_CONV_BK 32
#endif
constexpr int BM = 64;          // output rows per workgroup
constexpr int BN = 64;          // output columns per workgroup
constexpr int BK = MG_CONV_BK;  // reduction step (16 or 32)
constexpr int NSUB = BK / 16;   // staged rows per thread and operand in one step
constexpr int NT = 256;         // four waves
constexpr int LDR = 64 + 16;    // reduction-major tiles: rows 80 floats (16 banks) apart
constexpr int LDM = BK + 4;     // the data gradient's pixel-major A tile: 20 or 36 floats
                                // per row, both conflict-free for the operand reads
static_assert(BK == 16 || BK == 32, "reduction step");
constexpr int kOOB = 0x7ffffff0;   // byte offset past every buffer: reads as zero

__device__ __forceinline__ int fdiv(int n, FastDiv f) {
    return (int)((__umulhi((unsigned)n, f.mul) + (unsigned)n) >> f.shift);
}

// Divisors the kernels use in their per-step index arithmetic.
struct ConvDivs {
    FastDiv PQ, Q, K, S, sh, sw, C, HW, W;
};

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

// 2x2 blocks of v_mfma_f32_16x16x4_f32 over one reduction step.
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

// LDS of one workgroup: the two derivatives' double-buffered tiles share it.
struct WgradLds {
    float As[2][BK][LDR];   // dY tile, [m][k]
    float Bs[2][BK][LDR];   // X gather, [m][j]
};
struct DgradLds {
    float As[2][BM][LDM];   // dY gather, [m][j]
    float Bs[2][BK][LDR];   // W rows, [j][c]
};
union __attribute__((aligned(16))) ConvLds {
    WgradLds w;
    DgradLds d;
};

// Work of one filter-gradient launch: grid (k tile, j tile, split), split fastest.
struct WgradJob {
    const float *X, *dY;
    float *out;        // dW (one split) or the partials [split][K][R*S*C]
    int tiles_j, nsplit, nsteps, blocks;
};
// Work of one data-gradient launch: grid (m tile, c tile, split), split fastest.
struct DgradJob {
    const float *dY, *Wt;
    float *out;        // dX (one split) or the partials [split][N*H*W][C]
    int tiles_c, nsplit, blocks;
};

// ------------------------------------------------------- filter gradient --
// Block `bid` of the job: split `split` of `nsplit` sums the reduction steps
// [st0, st1) of the N*P*Q positions for one 64x64 tile of dW.
template <int VA, int VB>
__device__ __forceinline__ void wgrad_tile(int bid, WgradLds &L, const WgradJob &job,
                                           const ConvProblem &p, const ConvDivs &dv) {
    auto &As = L.As;
    auto &Bs = L.Bs;
    const float *__restrict__ X = job.X;
    const float *__restrict__ dY = job.dY;
    float *__restrict__ out = job.out;
    const int tiles_j = job.tiles_j, nsplit = job.nsplit, nsteps = job.nsteps;

    const int RSC = p.R * p.S * p.C;
    const int PQ = p.P * p.Q;
    const int M = p.N * PQ;
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
    int ka4[4], br[4], bsx[4], boff[4];   // byte offsets (ka4, boff) and taps
    bool kok[4], bok[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int ka = (VA == 4) ? k0 + 4 * lcol : k0 + lcol + 16 * e;
        ka4[e] = 4 * ka;
        kok[e] = ka < p.K;
        const int j = (VB == 4) ? j0 + 4 * lcol : j0 + lcol + 16 * e;
        const int rs = fdiv(j, dv.C), c = j - rs * p.C;
        br[e] = fdiv(rs, dv.S);
        bsx[e] = rs - br[e] * p.S;
        boff[e] = 4 * ((br[e] * p.W + bsx[e]) * p.C + c);
        bok[e] = j < RSC;
    }

    // Step st stages reduction rows st*BK + lrow + 16u, u < NSUB.
    auto load = [&](int st, f32x4 (&ra)[NSUB], f32x4 (&rb)[NSUB]) {
#pragma unroll
        for (int u = 0; u < NSUB; ++u) {
            const int m = st * BK + lrow + 16 * u;
            const bool mok = m < M;
            const int n = fdiv(m, dv.PQ), pq = m - n * PQ;
            const int pp = fdiv(pq, dv.Q), qq = pq - pp * p.Q;
            const int hb = pp * p.sh - p.ph, wb = qq * p.sw - p.pw;
            const int xbase = ((n * p.H + hb) * p.W + wb) * p.C;
            int oa[4], ob[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                oa[e] = (mok && kok[e]) ? m * (4 * p.K) + ka4[e] : kOOB;
                const int h = hb + br[e], wi = wb + bsx[e];
                const bool ok = mok && bok[e] && (unsigned)h < (unsigned)p.H &&
                                (unsigned)wi < (unsigned)p.W;
                ob[e] = ok ? xbase * 4 + boff[e] : kOOB;
                if (VA == 4 && VB == 4) break;
            }
            ra[u] = load_vec<VA>(rdy, oa);
            rb[u] = load_vec<VB>(rx, ob);
        }
    };
    auto store = [&](int buf, const f32x4 (&ra)[NSUB], const f32x4 (&rb)[NSUB]) {
#pragma unroll
        for (int u = 0; u < NSUB; ++u) {
            const int row = lrow + 16 * u;
            if (VA == 4) {
                *reinterpret_cast<f32x4 *>(&As[buf][row][4 * lcol]) = ra[u];
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) As[buf][row][lcol + 16 * e] = ra[u][e];
            }
            if (VB == 4) {
                *reinterpret_cast<f32x4 *>(&Bs[buf][row][4 * lcol]) = rb[u];
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) Bs[buf][row][lcol + 16 * e] = rb[u][e];
            }
        }
    };

    f32x4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int jb = 0; jb < 2; ++jb) acc[i][jb] = zero4();

    // Two register sets keep the loads of the next two steps in flight while
    // the current step, already in LDS, is multiplied.
    f32x4 ra0[NSUB], rb0[NSUB], ra1[NSUB], rb1[NSUB];
    if (st0 < st1) load(st0, ra0, rb0);
    if (st0 + 1 < st1) load(st0 + 1, ra1, rb1);
    if (st0 < st1) store(0, ra0, rb0);
    __syncthreads();
    // step st: `na`/`nb` hold step st+1 (in flight), `fa`/`fb` are free
    auto body = [&](int st, f32x4 (&na)[NSUB], f32x4 (&nb)[NSUB], f32x4 (&fa)[NSUB],
                    f32x4 (&fb)[NSUB]) {
        const int cur = (st - st0) & 1;
        if (st + 2 < st1) load(st + 2, fa, fb);
        mma_step(acc,
                 [&](int kk, int i) { return As[cur][4 * kk + g][32 * wm + 16 * i + il]; },
                 [&](int kk, int jb) { return Bs[cur][4 * kk + g][32 * wn + 16 * jb + il]; });
        if (st + 1 < st1) store(cur ^ 1, na, nb);
        __syncthreads();
    };
    for (int st = st0; st < st1; st += 2) {
        body(st, ra1, rb1, ra0, rb0);
        if (st + 1 < st1) body(st + 1, ra0, rb0, ra1, rb1);
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

template <int VA, int VB>
__global__ __launch_bounds__(NT) void conv_wgrad_f32(WgradJob job, ConvProblem p, ConvDivs dv) {
    __shared__ ConvLds lds;
    wgrad_tile<VA, VB>(blockIdx.x, lds.w, job, p, dv);
}

// out[i] = sum over splits of part[split][i].  A group of G consecutive lanes
// (G a power of two, up to 64) owns four consecutive elements (one when
// total % 4 != 0): lane t of the group adds splits t, t + G, t + 2G, ... in
// increasing order, then the group combines its G sums by a butterfly over
// lane distances G/2, ..., 1.  The order of every addition is fixed by
// (nsplit, G), so results repeat bit for bit.
struct ReduceJob {
    const float *part;
    float *out;
    int nsplit, total, G, vec, blocks;
};

__device__ __forceinline__ void split_reduce(int block, const ReduceJob &job) {
    const int G = job.G;
    const int gid = (block * 256 + (int)threadIdx.x) / G;   // element group
    const int t = threadIdx.x & (G - 1);
    const int E = job.vec ? 4 : 1;
    const int i = E * gid;
    const bool live = i < job.total;
    f32x4 sum = zero4();
    if (live) {
        for (int k = t; k < job.nsplit; k += G) {
            const float *src = job.part + (size_t)k * job.total + i;
            if (job.vec)
                sum += *reinterpret_cast<const f32x4 *>(src);
            else
                sum[0] += *src;
        }
    }
    for (int d = G >> 1; d > 0; d >>= 1)
#pragma unroll
        for (int e = 0; e < 4; ++e) sum[e] += __shfl_xor(sum[e], d, 64);
    if (live && t == 0) {
        if (job.vec)
            *reinterpret_cast<f32x4 *>(job.out + i) = sum;
        else
            job.out[i] = sum[0];
    }
}

// One or two reductions in one launch (b.blocks == 0 for one).
__global__ __launch_bounds__(256) void conv_split_reduce_f32(ReduceJob a, ReduceJob b) {
    if ((int)blockIdx.x < a.blocks)
        split_reduce(blockIdx.x, a);
    else
        split_reduce(blockIdx.x - a.blocks, b);
}

// --------------------------------------------------------- data gradient --
// Block `bid` of the job: split `split` of `nsplit` sums the reduction steps
// [st0, st1) of (r, s, k) for one 64x64 tile of dX.
template <int VA, int VB>
__device__ __forceinline__ void dgrad_tile(int bid, DgradLds &L, const DgradJob &job,
                                           const ConvProblem &p, const ConvDivs &dv) {
    auto &As = L.As;
    auto &Bs = L.Bs;
    const float *__restrict__ dY = job.dY;
    const float *__restrict__ Wt = job.Wt;
    float *__restrict__ out = job.out;
    const int tiles_c = job.tiles_c, nsplit = job.nsplit;

    const int M = p.N * p.H * p.W;
    const int RSK = p.R * p.S * p.K;
    const int nsteps = (RSK + BK - 1) / BK;
    const int split = bid % nsplit;
    bid /= nsplit;
    const int m0 = (bid / tiles_c) * BM;
    const int c0 = (bid % tiles_c) * BN;
    const int st0 = (int)((long)nsteps * split / nsplit);
    const int st1 = (int)((long)nsteps * (split + 1) / nsplit);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int il = lane & 15, g = lane >> 4;
    const int wm = w & 1, wn = w >> 1;

    const auto rdy = buffer_rsrc(dY, p.N * p.P * p.Q * p.K * 4);
    const auto rw = buffer_rsrc(Wt, p.K * p.R * p.S * p.C * 4);

    // A staging: pixel row ar (fixed), reduction columns 4*jq + 16u .. +3 of
    // a step; B staging: reduction rows jr + 16u of a step, channel columns.
    const int ar = tid >> 2, jq = tid & 3;
    const int m = m0 + ar;
    const bool mok = m < M;
    const int n = fdiv(m, dv.HW), hw = m - n * (p.H * p.W);
    const int h = fdiv(hw, dv.W), wpix = hw - h * p.W;
    const int jr = tid >> 4, cc = tid & 15;
    int cb[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) cb[e] = (VB == 4) ? c0 + 4 * cc + e : c0 + cc + 16 * e;

    const int nP = n * p.P, hph = h + p.ph, wpw = wpix + p.pw;
    const int RS = p.R * p.S;
    // K % BK == 0: every step lies within one tap (r, s), known to the whole
    // workgroup; otherwise each staged element finds its own tap.
    const bool tap_uniform = p.K % BK == 0;

    // dY offset of reduction index (tap t = r*S + s, channel k) for this
    // thread's pixel, or kOOB when no output position (p, q) reads it.
    auto dy_offset = [&](int r, int s, int k) {
        const int hp = hph - r, wq = wpw - s;   // = p*sh, q*sw
        const int pp = fdiv(hp < 0 ? 0 : hp, dv.sh), qq = fdiv(wq < 0 ? 0 : wq, dv.sw);
        const bool ok = mok && hp >= 0 && wq >= 0 && pp * p.sh == hp && qq * p.sw == wq &&
                        pp < p.P && qq < p.Q;
        return ok ? (((nP + pp) * p.Q + qq) * p.K + k) * 4 : kOOB;
    };

    auto load = [&](int st, f32x4 (&ra)[NSUB], f32x4 (&rb)[NSUB]) {
        const int j0 = st * BK;
        int t0 = 0, kb = 0, r0 = 0, s0 = 0;
        if (tap_uniform) {
            t0 = fdiv(j0, dv.K);
            kb = j0 - t0 * p.K;
            r0 = fdiv(t0, dv.S);
            s0 = t0 - r0 * p.S;
        }
#pragma unroll
        for (int u = 0; u < NSUB; ++u) {
            int oa[4], ob[4];
            if (tap_uniform) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int dk = 16 * u + 4 * jq + e;
                    oa[e] = j0 + dk < RSK ? dy_offset(r0, s0, kb + dk) : kOOB;
                    if (VA == 4) break;
                }
                // W[k][r][s][c] for reduction row k = kb + 16u + jr of tap t0
                const int row = ((kb + 16 * u + jr) * RS + t0) * p.C;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    ob[e] = (j0 + 16 * u + jr < RSK && cb[e] < p.C) ? (row + cb[e]) * 4 : kOOB;
                    if (VB == 4) break;
                }
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    // a 16-byte chunk (VA == 4, K % 4 == 0) never straddles two taps
                    const int j = j0 + 16 * u + 4 * jq + e;
                    const int t = fdiv(j, dv.K), k = j - t * p.K;
                    const int r = fdiv(t, dv.S), s = t - r * p.S;
                    oa[e] = j < RSK ? dy_offset(r, s, k) : kOOB;
                    if (VA == 4) break;
                }
                const int j = j0 + 16 * u + jr;
                const int t = fdiv(j, dv.K), k = j - t * p.K;
                const int row = (k * RS + t) * p.C;   // ((k*R + r)*S + s) * C
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    ob[e] = (j < RSK && cb[e] < p.C) ? (row + cb[e]) * 4 : kOOB;
                    if (VB == 4) break;
                }
            }
            ra[u] = load_vec<VA>(rdy, oa);
            rb[u] = load_vec<VB>(rw, ob);
        }
    };
    auto store = [&](int buf, const f32x4 (&ra)[NSUB], const f32x4 (&rb)[NSUB]) {
#pragma unroll
        for (int u = 0; u < NSUB; ++u) {
            *reinterpret_cast<f32x4 *>(&As[buf][ar][16 * u + 4 * jq]) = ra[u];
            if (VB == 4) {
                *reinterpret_cast<f32x4 *>(&Bs[buf][jr + 16 * u][4 * cc]) = rb[u];
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) Bs[buf][jr + 16 * u][cc + 16 * e] = rb[u][e];
            }
        }
    };

    f32x4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int jb = 0; jb < 2; ++jb) acc[i][jb] = zero4();

    // Two register sets keep the loads of the next two steps in flight while
    // the current step, already in LDS, is multiplied.
    f32x4 ra0[NSUB], rb0[NSUB], ra1[NSUB], rb1[NSUB];
    if (st0 < st1) load(st0, ra0, rb0);
    if (st0 + 1 < st1) load(st0 + 1, ra1, rb1);
    if (st0 < st1) store(0, ra0, rb0);
    __syncthreads();
    // step st: `na`/`nb` hold step st+1 (in flight), `fa`/`fb` are free
    auto body = [&](int st, f32x4 (&na)[NSUB], f32x4 (&nb)[NSUB], f32x4 (&fa)[NSUB],
                    f32x4 (&fb)[NSUB]) {
        const int cur = (st - st0) & 1;
        if (st + 2 < st1) load(st + 2, fa, fb);
        mma_step(acc,
                 [&](int kk, int i) { return As[cur][32 * wm + 16 * i + il][4 * kk + g]; },
                 [&](int kk, int jb) { return Bs[cur][4 * kk + g][32 * wn + 16 * jb + il]; });
        if (st + 1 < st1) store(cur ^ 1, na, nb);
        __syncthreads();
    };
    for (int st = st0; st < st1; st += 2) {
        body(st, ra1, rb1, ra0, rb0);
        if (st + 1 < st1) body(st + 1, ra0, rb0, ra1, rb1);
    }

    float *dst = out + (size_t)split * M * p.C;   // split 0 of 1 is dX itself
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int jb = 0; jb < 2; ++jb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int mo = m0 + 32 * wm + 16 * i + 4 * g + r;
                const int c = c0 + 32 * wn + 16 * jb + il;
                if (mo < M && c < p.C) dst[(size_t)mo * p.C + c] = acc[i][jb][r];
            }
}

template <int VA, int VB>
__global__ __launch_bounds__(NT) void conv_dgrad_f32(DgradJob job, ConvProblem p, ConvDivs dv) {
    __shared__ ConvLds lds;
    dgrad_tile<VA, VB>(blockIdx.x, lds.d, job, p, dv);
}

// Both derivatives of one convolution in one launch: the first d.blocks
// workgroups run the data gradient, the rest the filter gradient.
template <int VA, int VB>
__global__ __launch_bounds__(NT) void conv_bwd_f32(DgradJob d, WgradJob w, ConvProblem p,
                                                   ConvDivs dv) {
    __shared__ ConvLds lds;
    if ((int)blockIdx.x < d.blocks)
        dgrad_tile<VA, VB>(blockIdx.x, lds.d, d, p, dv);
    else
        wgrad_tile<VA, VB>(blockIdx.x - d.blocks, lds.w, w, p, dv);
}

int cdiv(int a, int b) { return (a + b - 1) / b; }

ConvDivs make_divs(const ConvProblem &p) {
    return ConvDivs{make_fastdiv(p.P * p.Q), make_fastdiv(p.Q), make_fastdiv(p.K),
                    make_fastdiv(p.S), make_fastdiv(p.sh), make_fastdiv(p.sw),
                    make_fastdiv(p.C), make_fastdiv(p.H * p.W), make_fastdiv(p.W)};
}

}  // namespace

FastDiv make_fastdiv(unsigned d) {
    unsigned l = 0;
    while ((1ull << l) < d) ++l;
    const unsigned long long m = ((1ull << 32) * ((1ull << l) - d)) / d + 1;
    return FastDiv{(unsigned)m, l};
}

// Split a reduction when the output tiles alone fill fewer than
// MG_CONV_SPLIT_BELOW workgroups: aim at about MG_CONV_SPLIT_TARGET
// workgroups, with at least MG_CONV_SPLIT_TERMS summed terms per split.
#ifndef MG_CONV_SPLIT_BELOW
#define MG_CONV_SPLIT_BELOW 512
#endif
#ifndef MG_CONV_SPLIT_TARGET
#define MG_CONV_SPLIT_TARGET 1024
#endif
#ifndef MG_CONV_SPLIT_TERMS
#define MG_CONV_SPLIT_TERMS 128
#endif
static int splits_for(long tiles, long steps) {
    if (tiles >= MG_CONV_SPLIT_BELOW) return 1;
    const long by_grid = (MG_CONV_SPLIT_TARGET + tiles - 1) / tiles;
    const long by_steps = steps / (MG_CONV_SPLIT_TERMS / BK);
    const long s = by_grid < by_steps ? by_grid : by_steps;
    return s < 1 ? 1 : (int)s;
}

int conv_wgrad_splits(const ConvProblem &p) {
    return splits_for((long)cdiv(p.K, BM) * cdiv(p.R * p.S * p.C, BN),
                      cdiv(p.N * p.P * p.Q, BK));
}

int conv_dgrad_splits(const ConvProblem &p) {
    return splits_for((long)cdiv(p.N * p.H * p.W, BM) * cdiv(p.C, BN),
                      cdiv(p.R * p.S * p.K, BK));
}

namespace {

WgradJob wgrad_job(const ConvProblem &p, const float *X, const float *dY, float *dW,
                   float *partials) {
    const int ns = conv_wgrad_splits(p);
    const int tiles_j = cdiv(p.R * p.S * p.C, BN);
    return WgradJob{X, dY, ns > 1 ? partials : dW, tiles_j, ns, cdiv(p.N * p.P * p.Q, BK),
                    cdiv(p.K, BM) * tiles_j * ns};
}

DgradJob dgrad_job(const ConvProblem &p, const float *dY, const float *Wt, float *dX,
                   float *partials) {
    const int ns = conv_dgrad_splits(p);
    const int tiles_c = cdiv(p.C, BN);
    return DgradJob{dY, Wt, ns > 1 ? partials : dX, tiles_c, ns,
                    cdiv(p.N * p.H * p.W, BM) * tiles_c * ns};
}

ReduceJob reduce_job(const float *partials, int nsplit, int total, float *out) {
    // lanes per element group: about nsplit / 4 splits each, at most 64
    int G = 1;
    while (G < 64 && 4 * G < nsplit) G *= 2;
    const int vec = total % 4 == 0;
    const long groups = vec ? total / 4 : total;
    return ReduceJob{partials, out, nsplit, total, G, vec, (int)((groups * G + 255) / 256)};
}

// The kernel instance for the operands' vector widths: 16-byte loads along
// k (K % 4 == 0) and along c (C % 4 == 0), else 4-byte loads.
template <template <int, int> class Launch, typename... Args>
hipError_t by_widths(const ConvProblem &p, Args &&...args) {
    const bool va = p.K % 4 == 0, vb = p.C % 4 == 0;
    if (va && vb) return Launch<4, 4>::run(args...);
    if (va) return Launch<4, 1>::run(args...);
    if (vb) return Launch<1, 4>::run(args...);
    return Launch<1, 1>::run(args...);
}

template <int VA, int VB>
struct LaunchW {
    static hipError_t run(const WgradJob &j, const ConvProblem &p, const ConvDivs &dv,
                          hipStream_t s) {
        conv_wgrad_f32<VA, VB><<<dim3(j.blocks), dim3(NT), 0, s>>>(j, p, dv);
        return hipGetLastError();
    }
};
template <int VA, int VB>
struct LaunchD {
    static hipError_t run(const DgradJob &j, const ConvProblem &p, const ConvDivs &dv,
                          hipStream_t s) {
        conv_dgrad_f32<VA, VB><<<dim3(j.blocks), dim3(NT), 0, s>>>(j, p, dv);
        return hipGetLastError();
    }
};
template <int VA, int VB>
struct LaunchDW {
    static hipError_t run(const DgradJob &d, const WgradJob &w, const ConvProblem &p,
                          const ConvDivs &dv, hipStream_t s) {
        conv_bwd_f32<VA, VB><<<dim3(d.blocks + w.blocks), dim3(NT), 0, s>>>(d, w, p, dv);
        return hipGetLastError();
    }
};

hipError_t launch_reduce(const ReduceJob &a, const ReduceJob &b, hipStream_t s) {
    conv_split_reduce_f32<<<dim3(a.blocks + b.blocks), dim3(256), 0, s>>>(a, b);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_conv_wgrad_f32(const ConvProblem &p, const float *X, const float *dY,
                                 float *dW, float *partials, hipStream_t s) {
    const WgradJob j = wgrad_job(p, X, dY, dW, partials);
    if (j.nsplit > 1 && partials == nullptr) return hipErrorInvalidValue;
    return by_widths<LaunchW>(p, j, p, make_divs(p), s);
}

hipError_t launch_conv_dgrad_f32(const ConvProblem &p, const float *dY, const float *Wt,
                                 float *dX, float *partials, hipStream_t s) {
    const DgradJob j = dgrad_job(p, dY, Wt, dX, partials);
    if (j.nsplit > 1 && partials == nullptr) return hipErrorInvalidValue;
    return by_widths<LaunchD>(p, j, p, make_divs(p), s);
}

hipError_t launch_conv_bwd_f32(const ConvProblem &p, const float *X, const float *Wt,
                               const float *dY, float *dX, float *dW, float *dpart,
                               float *wpart, hipStream_t s) {
    const DgradJob d = dgrad_job(p, dY, Wt, dX, dpart);
    const WgradJob w = wgrad_job(p, X, dY, dW, wpart);
    if ((d.nsplit > 1 && dpart == nullptr) || (w.nsplit > 1 && wpart == nullptr))
        return hipErrorInvalidValue;
    return by_widths<LaunchDW>(p, d, w, p, make_divs(p), s);
}

hipError_t launch_conv_split_reduce_f32(const float *partials, int nsplit, int total,
                                        float *out, hipStream_t s) {
    return launch_reduce(reduce_job(partials, nsplit, total, out),
                         ReduceJob{nullptr, nullptr, 0, 0, 1, 0, 0}, s);
}

hipError_t launch_conv_split_reduce2_f32(const float *part_a, int nsplit_a, int total_a,
                                         float *out_a, const float *part_b, int nsplit_b,
                                         int total_b, float *out_b, hipStream_t s) {
    return launch_reduce(reduce_job(part_a, nsplit_a, total_a, out_a),
                         reduce_job(part_b, nsplit_b, total_b, out_b), s);
}

}  // namespace mg
