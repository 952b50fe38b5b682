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
//       per stride-parity class of pixels (see DgradJob): m = (n, i, j) of
//       the class, j = (tr, ts, k) over the class's filter taps with k
//       fastest, W[j][c] = W[k][r][s][c], dYg[m][j] = dY at the output
//       position the tap reads, 0 outside dY.
//
// Both run 64x64 output tiles on 256 threads: each of the four waves owns a
// 32x32 quarter as 2x2 blocks of 16x16 accumulators, and the reduction
// advances BK (16) at a time through double-buffered LDS tiles (one barrier
// per step; the global loads of steps t+1 and t+2 are in flight, in two
// register sets, during the products of step t).  Operands reach LDS
// through raw buffer loads whose offset is pushed past the end of the buffer
// for a padded or out-of-range element, which reads as zero: the padding of
// the convolution and the tails of every dimension become zeros without a
// branch.  Every output element is one fixed-order sum (within a workgroup,
// then across splits in a fixed order): no atomics.
#include <algorithm>
#include <vector>

#include "../device_common.h"
#include "conv_launch.h"

namespace mg {
namespace {

#ifndef MG_CONV_BK
#define MG_CONV_BK 16
#endif
constexpr int BM = 64;          // output rows per workgroup (columns: 64 or 128, TN)
constexpr int BK = MG_CONV_BK;  // reduction step (16 or 32)
constexpr int NSUB = BK / 16;   // staged rows per thread and operand in one step
constexpr int NT = 256;         // four waves
constexpr int LDR = 64 + 16;    // reduction-major 64-wide tiles: rows 80 floats (16 banks)
                                // apart; 128-wide ones use 144 (also 16 banks)
constexpr int LDM = BK + 4;     // the data gradient's pixel-major A tile: 20 (or 36)
                                // floats per row, conflict-free for the operand reads
static_assert(BK == 16 || BK == 32, "reduction step");
// Waves per SIMD the register allocator must allow (measured best of 4, 6
// and 8 at a 16-deep step; 4 also fits 40 KB workgroups at a 32-deep one).
#ifndef MG_CONV_OCC
#define MG_CONV_OCC 4
#endif
constexpr int kOOB = 0x7ffffff0;   // byte offset past every buffer: reads as zero

__device__ __forceinline__ int fdiv(int n, FastDiv f) {
    return (int)((__umulhi((unsigned)n, f.mul) + (unsigned)n) >> f.shift);
}

// Divisors the kernels use in their per-step index arithmetic.
struct ConvDivs {
    FastDiv PQ, Q, K, S, C;
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

// 2 x NJ blocks of v_mfma_f32_16x16x4_f32 over one reduction step.
// a(kk, i) and b(kk, jb) return this lane's operand: A[row 16i + l%16][red 4kk + l/16]
// and B[red 4kk + l/16][col 16jb + l%16] of the wave's 32 x 16NJ part of the tile.
template <int NJ, typename FA, typename FB>
__device__ __forceinline__ void mma_step(f32x4 (&acc)[2][NJ], FA &&a, FB &&b) {
#pragma unroll
    for (int kk = 0; kk < BK / 4; ++kk) {
        const float a0 = a(kk, 0), a1 = a(kk, 1);
        float bj[NJ];
#pragma unroll
        for (int jb = 0; jb < NJ; ++jb) bj[jb] = b(kk, jb);
#pragma unroll
        for (int jb = 0; jb < NJ; ++jb) {
            acc[0][jb] = mfma16x16x4(a0, bj[jb], acc[0][jb]);
            acc[1][jb] = mfma16x16x4(a1, bj[jb], acc[1][jb]);
        }
    }
}

// Staged B columns of one thread: with 16-byte chunks (VB == 4), TN/64
// chunks at columns 4*col + 64v; with 4-byte loads (VB == 1, TN == 64), four
// floats at columns col + 16e.
template <int VB, int TN>
struct BCols {
    static_assert(TN == 64 || (TN == 128 && VB == 4), "tile width");
    static constexpr int NV = VB == 4 ? TN / 64 : 1;   // f32x4 registers per row
    static constexpr int NE = VB == 4 ? TN / 64 : 4;   // separately addressed elements
    __device__ static int col(int c, int e) { return VB == 4 ? 4 * c + 64 * e : c + 16 * e; }
};

// LDS of one workgroup: the two derivatives' double-buffered tiles share it.
template <int TN>
struct WgradLds {
    float As[2][BK][LDR];      // dY tile, [m][k]
    float Bs[2][BK][TN + 16];  // X gather, [m][j]
};
template <int TN>
struct DgradLds {
    float As[2][BM][LDM];      // dY gather, [m][j]
    float Bs[2][BK][TN + 16];  // W rows, [j][c]
};
template <int TN>
union __attribute__((aligned(16))) ConvLds {
    WgradLds<TN> w;
    DgradLds<TN> d;
};

// Work of one filter-gradient launch: grid (k tile, j tile, split), split fastest.
struct WgradJob {
    const float *X, *dY;
    float *out;        // dW (one split) or the partials [split][K][R*S*C]
    int tiles_j, nsplit, nsteps, blocks;
};
// Data-gradient work of one stride-parity class.  With strides (sh, sw) the
// input pixels split into sh*sw classes h = a + sh*i, w = b + sw*j, and the
// only filter taps that reach a pixel of class (a, b) are r = r0 + sh*tr,
// s = s0 + sw*ts with r0 = (a + ph) mod sh, s0 = (b + pw) mod sw; such a tap
// reads output position p = i + da - tr, q = j + db - ts.  Each class is a
// dense GEMM over (n, i, j) x c summing only its (tr, ts, k): no tap that
// skips the pixel is ever multiplied (stride 1 is one class with every tap).
// Grid of a class: (m tile, c tile, split), split fastest.
struct DgradJob {
    const float *dY, *Wt;
    float *out;        // dX (one split) or the partials [split][N*H*W][C], dX layout
    int tiles_c, nsplit, blocks;
    int a, b, Hc, Wc, r0, s0, Rc, Sc, da, db;
    FastDiv HWc, Wc_, Sc_;
};
constexpr int kMaxClasses = 16;   // strides up to 4 x 4 in one launch
struct DgradJobs {
    DgradJob c[kMaxClasses];
    int n;
};

// ------------------------------------------------------- filter gradient --
// Block `bid` of the job: split `split` of `nsplit` sums the reduction steps
// [st0, st1) of the N*P*Q positions for one 64x64 tile of dW.
template <int VA, int VB, int TN>
__device__ __forceinline__ void wgrad_tile(int bid, WgradLds<TN> &L, const WgradJob &job,
                                           const ConvProblem &p, const ConvDivs &dv) {
    using BC = BCols<VB, TN>;
    constexpr int NJ = TN / 32;   // 16-column blocks per wave
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
    const int j0 = (bid % tiles_j) * TN;
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
    int ka4[4], br[BC::NE], bsx[BC::NE], boff[BC::NE];   // byte offsets (ka4, boff), taps
    bool kok[4], bok[BC::NE];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int ka = (VA == 4) ? k0 + 4 * lcol : k0 + lcol + 16 * e;
        ka4[e] = 4 * ka;
        kok[e] = ka < p.K;
    }
#pragma unroll
    for (int e = 0; e < BC::NE; ++e) {
        const int j = j0 + BC::col(lcol, e);
        const int rs = fdiv(j, dv.C), c = j - rs * p.C;
        br[e] = fdiv(rs, dv.S);
        bsx[e] = rs - br[e] * p.S;
        boff[e] = 4 * ((br[e] * p.W + bsx[e]) * p.C + c);
        bok[e] = j < RSC;
    }

    // Step st stages reduction rows st*BK + lrow + 16u, u < NSUB.
    using Regs = f32x4[NSUB][1 + BC::NV];   // [u][0]: A (dY), [u][1 + v]: B (X)
    auto load = [&](int st, Regs &rg) {
#pragma unroll
        for (int u = 0; u < NSUB; ++u) {
            const int m = st * BK + lrow + 16 * u;
            const bool mok = m < M;
            const int n = fdiv(m, dv.PQ), pq = m - n * PQ;
            const int pp = fdiv(pq, dv.Q), qq = pq - pp * p.Q;
            const int hb = pp * p.sh - p.ph, wb = qq * p.sw - p.pw;
            const int xbase = ((n * p.H + hb) * p.W + wb) * p.C;
            int oa[4], ob[BC::NE];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                oa[e] = (mok && kok[e]) ? m * (4 * p.K) + ka4[e] : kOOB;
                if (VA == 4) break;
            }
#pragma unroll
            for (int e = 0; e < BC::NE; ++e) {
                const int h = hb + br[e], wi = wb + bsx[e];
                const bool ok = mok && bok[e] && (unsigned)h < (unsigned)p.H &&
                                (unsigned)wi < (unsigned)p.W;
                ob[e] = ok ? xbase * 4 + boff[e] : kOOB;
            }
            rg[u][0] = load_vec<VA>(rdy, oa);
            if (VB == 4) {
#pragma unroll
                for (int v = 0; v < BC::NV; ++v) rg[u][1 + v] = buffer_load_f32x4(rx, ob[v]);
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) rg[u][1][e] = buffer_load_f32(rx, ob[e]);
            }
        }
    };
    auto store = [&](int buf, const Regs &rg) {
#pragma unroll
        for (int u = 0; u < NSUB; ++u) {
            const int row = lrow + 16 * u;
            if (VA == 4) {
                *reinterpret_cast<f32x4 *>(&As[buf][row][4 * lcol]) = rg[u][0];
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) As[buf][row][lcol + 16 * e] = rg[u][0][e];
            }
            if (VB == 4) {
#pragma unroll
                for (int v = 0; v < BC::NV; ++v)
                    *reinterpret_cast<f32x4 *>(&Bs[buf][row][BC::col(lcol, v)]) = rg[u][1 + v];
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) Bs[buf][row][BC::col(lcol, e)] = rg[u][1][e];
            }
        }
    };

    f32x4 acc[2][NJ];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int jb = 0; jb < NJ; ++jb) acc[i][jb] = zero4();

    // Two register sets keep the loads of the next two steps in flight while
    // the current step, already in LDS, is multiplied.
    Regs r0, r1;
    if (st0 < st1) load(st0, r0);
    if (st0 + 1 < st1) load(st0 + 1, r1);
    if (st0 < st1) store(0, r0);
    __syncthreads();
    // step st: `nx` holds step st+1 (in flight), `fr` is free
    auto body = [&](int st, Regs &nx, Regs &fr) {
        const int cur = (st - st0) & 1;
        if (st + 2 < st1) load(st + 2, fr);
        mma_step<NJ>(acc,
                     [&](int kk, int i) { return As[cur][4 * kk + g][32 * wm + 16 * i + il]; },
                     [&](int kk, int jb) { return Bs[cur][4 * kk + g][(TN / 2) * wn + 16 * jb + il]; });
        if (st + 1 < st1) store(cur ^ 1, nx);
        __syncthreads();
    };
    for (int st = st0; st < st1; st += 2) {
        body(st, r1, r0);
        if (st + 1 < st1) body(st + 1, r0, r1);
    }

    float *dst = out + (size_t)split * p.K * RSC;   // split 0 of 1 is dW itself
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int jb = 0; jb < NJ; ++jb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int k = k0 + 32 * wm + 16 * i + 4 * g + r;
                const int j = j0 + (TN / 2) * wn + 16 * jb + il;
                if (k < p.K && j < RSC) dst[(size_t)k * RSC + j] = acc[i][jb][r];
            }
}

template <int VA, int VB, int TN>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(MG_CONV_OCC, 8)))
void conv_wgrad_f32(WgradJob job, ConvProblem p, ConvDivs dv) {
    __shared__ ConvLds<TN> lds;
    wgrad_tile<VA, VB, TN>(blockIdx.x, lds.w, job, p, dv);
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
// Block `bid` of a class job: split `split` of `nsplit` sums the reduction
// steps [st0, st1) of the class's (tr, ts, k) for one 64x64 tile of its
// pixels x channels.
template <int VA, int VB, int TN>
__device__ __forceinline__ void dgrad_tile(int bid, DgradLds<TN> &L, const DgradJob &job,
                                           const ConvProblem &p, const ConvDivs &dv) {
    using BC = BCols<VB, TN>;
    constexpr int NJ = TN / 32;   // 16-column blocks per wave
    auto &As = L.As;
    auto &Bs = L.Bs;
    const float *__restrict__ dY = job.dY;
    const float *__restrict__ Wt = job.Wt;
    float *__restrict__ out = job.out;
    const int tiles_c = job.tiles_c, nsplit = job.nsplit;

    const int HWc = job.Hc * job.Wc;
    const int Mc = p.N * HWc;
    const int RSKc = job.Rc * job.Sc * p.K;
    const int nsteps = (RSKc + BK - 1) / BK;
    const int split = bid % nsplit;
    bid /= nsplit;
    const int m0 = (bid / tiles_c) * BM;
    const int c0 = (bid % tiles_c) * TN;
    const int st0 = (int)((long)nsteps * split / nsplit);
    const int st1 = (int)((long)nsteps * (split + 1) / nsplit);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int il = lane & 15, g = lane >> 4;
    const int wm = w & 1, wn = w >> 1;

    const auto rdy = buffer_rsrc(dY, p.N * p.P * p.Q * p.K * 4);
    const auto rw = buffer_rsrc(Wt, p.K * p.R * p.S * p.C * 4);

    // A staging: class pixel row ar (fixed), reduction columns 4*jq + 16u ..
    // +3 of a step; B staging: reduction rows jr + 16u of a step, channel columns.
    const int ar = tid >> 2, jq = tid & 3;
    const int m = m0 + ar;
    const bool mok = m < Mc;
    const int n = fdiv(m, job.HWc), ij = m - n * HWc;
    const int i = fdiv(ij, job.Wc_), jw = ij - i * job.Wc;
    const int jr = tid >> 4, cc = tid & 15;
    int cb[BC::NE];   // channel columns this thread stages
#pragma unroll
    for (int e = 0; e < BC::NE; ++e) cb[e] = c0 + BC::col(cc, e);

    const int nP = n * p.P, pi = i + job.da, qj = jw + job.db;   // p = pi - tr, q = qj - ts
    // K % BK == 0: every step lies within one tap (tr, ts), known to the
    // whole workgroup; otherwise each staged element finds its own tap.
    const bool tap_uniform = p.K % BK == 0;

    // dY offset of (tap (tr, ts), channel k) for this thread's pixel, or kOOB
    // when the tap's output position lies outside dY.
    auto dy_offset = [&](int tr, int ts, int k) {
        const int pp = pi - tr, qq = qj - ts;
        const bool ok = mok && (unsigned)pp < (unsigned)p.P && (unsigned)qq < (unsigned)p.Q;
        return ok ? (((nP + pp) * p.Q + qq) * p.K + k) * 4 : kOOB;
    };
    // first float of W[k][r][s][:] for tap (tr, ts)
    auto w_row = [&](int k, int tr, int ts) {
        return ((k * p.R + job.r0 + p.sh * tr) * p.S + job.s0 + p.sw * ts) * p.C;
    };

    using Regs = f32x4[NSUB][1 + BC::NV];   // [u][0]: A (dY), [u][1 + v]: B (W)
    auto load = [&](int st, Regs &rg) {
        const int j0 = st * BK;
        int kb = 0, tr0 = 0, ts0 = 0;
        if (tap_uniform) {
            const int t0 = fdiv(j0, dv.K);
            kb = j0 - t0 * p.K;
            tr0 = fdiv(t0, job.Sc_);
            ts0 = t0 - tr0 * job.Sc;
        }
#pragma unroll
        for (int u = 0; u < NSUB; ++u) {
            int oa[4], ob[BC::NE];
            if (tap_uniform) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int dk = 16 * u + 4 * jq + e;
                    oa[e] = j0 + dk < RSKc ? dy_offset(tr0, ts0, kb + dk) : kOOB;
                    if (VA == 4) break;
                }
                // W[k][r][s][c] for reduction row k = kb + 16u + jr of the tap
                const int row = w_row(kb + 16 * u + jr, tr0, ts0);
#pragma unroll
                for (int e = 0; e < BC::NE; ++e)
                    ob[e] = (j0 + 16 * u + jr < RSKc && cb[e] < p.C) ? (row + cb[e]) * 4 : kOOB;
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    // a 16-byte chunk (VA == 4, K % 4 == 0) never straddles two taps
                    const int j = j0 + 16 * u + 4 * jq + e;
                    const int t = fdiv(j, dv.K), k = j - t * p.K;
                    const int tr = fdiv(t, job.Sc_), ts = t - tr * job.Sc;
                    oa[e] = j < RSKc ? dy_offset(tr, ts, k) : kOOB;
                    if (VA == 4) break;
                }
                const int j = j0 + 16 * u + jr;
                const int t = fdiv(j, dv.K), k = j - t * p.K;
                const int tr = fdiv(t, job.Sc_), ts = t - tr * job.Sc;
                const int row = w_row(k, tr, ts);
#pragma unroll
                for (int e = 0; e < BC::NE; ++e)
                    ob[e] = (j < RSKc && cb[e] < p.C) ? (row + cb[e]) * 4 : kOOB;
            }
            rg[u][0] = load_vec<VA>(rdy, oa);
            if (VB == 4) {
#pragma unroll
                for (int v = 0; v < BC::NV; ++v) rg[u][1 + v] = buffer_load_f32x4(rw, ob[v]);
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) rg[u][1][e] = buffer_load_f32(rw, ob[e]);
            }
        }
    };
    auto store = [&](int buf, const Regs &rg) {
#pragma unroll
        for (int u = 0; u < NSUB; ++u) {
            *reinterpret_cast<f32x4 *>(&As[buf][ar][16 * u + 4 * jq]) = rg[u][0];
            if (VB == 4) {
#pragma unroll
                for (int v = 0; v < BC::NV; ++v)
                    *reinterpret_cast<f32x4 *>(&Bs[buf][jr + 16 * u][BC::col(cc, v)]) = rg[u][1 + v];
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) Bs[buf][jr + 16 * u][BC::col(cc, e)] = rg[u][1][e];
            }
        }
    };

    f32x4 acc[2][NJ];
#pragma unroll
    for (int ii = 0; ii < 2; ++ii)
#pragma unroll
        for (int jb = 0; jb < NJ; ++jb) acc[ii][jb] = zero4();

    // Two register sets keep the loads of the next two steps in flight while
    // the current step, already in LDS, is multiplied.
    Regs r0, r1;
    if (st0 < st1) load(st0, r0);
    if (st0 + 1 < st1) load(st0 + 1, r1);
    if (st0 < st1) store(0, r0);
    __syncthreads();
    // step st: `nx` holds step st+1 (in flight), `fr` is free
    auto body = [&](int st, Regs &nx, Regs &fr) {
        const int cur = (st - st0) & 1;
        if (st + 2 < st1) load(st + 2, fr);
        mma_step<NJ>(acc,
                     [&](int kk, int ii) { return As[cur][32 * wm + 16 * ii + il][4 * kk + g]; },
                     [&](int kk, int jb) { return Bs[cur][4 * kk + g][(TN / 2) * wn + 16 * jb + il]; });
        if (st + 1 < st1) store(cur ^ 1, nx);
        __syncthreads();
    };
    for (int st = st0; st < st1; st += 2) {
        body(st, r1, r0);
        if (st + 1 < st1) body(st + 1, r0, r1);
    }

    // rows of this lane's accumulators back to dX pixels (n, a + sh*i, b + sw*j)
    float *dst = out + (size_t)split * p.N * p.H * p.W * p.C;   // split 0 of 1 is dX
#pragma unroll
    for (int ii = 0; ii < 2; ++ii)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int mo = m0 + 32 * wm + 16 * ii + 4 * g + r;
            if (mo >= Mc) continue;
            const int on = fdiv(mo, job.HWc), oij = mo - on * HWc;
            const int oi = fdiv(oij, job.Wc_), oj = oij - oi * job.Wc;
            const size_t pix = ((size_t)on * p.H + job.a + p.sh * oi) * p.W + job.b + p.sw * oj;
#pragma unroll
            for (int jb = 0; jb < NJ; ++jb) {
                const int c = c0 + (TN / 2) * wn + 16 * jb + il;
                if (c < p.C) dst[pix * p.C + c] = acc[ii][jb][r];
            }
        }
}

// Which class job a block belongs to (job counts and sizes are uniform).
__device__ __forceinline__ int find_class(const DgradJobs &jobs, int &bid) {
    int c = 0;
    while (c + 1 < jobs.n && bid >= jobs.c[c].blocks) {
        bid -= jobs.c[c].blocks;
        ++c;
    }
    return c;
}

template <int VA, int VB, int TN>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(MG_CONV_OCC, 8)))
void conv_dgrad_f32(DgradJobs jobs, ConvProblem p, ConvDivs dv) {
    __shared__ ConvLds<TN> lds;
    int bid = blockIdx.x;
    const int c = find_class(jobs, bid);
    dgrad_tile<VA, VB, TN>(bid, lds.d, jobs.c[c], p, dv);
}

// Both derivatives of one convolution in one launch: the first `dblocks`
// workgroups run the data gradient's class jobs, the rest the filter gradient.
template <int VA, int VB, int TN>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(MG_CONV_OCC, 8)))
void conv_bwd_f32(DgradJobs d, int dblocks, WgradJob w, ConvProblem p, ConvDivs dv) {
    __shared__ ConvLds<TN> lds;
    int bid = blockIdx.x;
    if (bid < dblocks) {
        const int c = find_class(d, bid);
        dgrad_tile<VA, VB, TN>(bid, lds.d, d.c[c], p, dv);
    } else {
        wgrad_tile<VA, VB, TN>(bid - dblocks, lds.w, w, p, dv);
    }
}

int cdiv(int a, int b) { return (a + b - 1) / b; }

ConvDivs make_divs(const ConvProblem &p) {
    return ConvDivs{make_fastdiv(p.P * p.Q), make_fastdiv(p.Q), make_fastdiv(p.K),
                    make_fastdiv(p.S), make_fastdiv(p.C)};
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
#define MG_CONV_SPLIT_TERMS 256
#endif
static int splits_for(long tiles, long steps) {
    if (tiles >= MG_CONV_SPLIT_BELOW) return 1;
    const long by_grid = (MG_CONV_SPLIT_TARGET + tiles - 1) / tiles;
    const long by_steps = steps / (MG_CONV_SPLIT_TERMS / BK);
    const long s = by_grid < by_steps ? by_grid : by_steps;
    return s < 1 ? 1 : (int)s;
}

// Output tile width: 64 columns.  A build option (MG_CONV_WIDE=1) selects
// 128 columns, with half the operand loads per product, when the channel
// vectors allow 16-byte loads and there are that many channels; on the
// ResNet-50 step it measured 6 % slower (fewer tiles, more splits, five
// waves per SIMD instead of seven).
#ifndef MG_CONV_WIDE
#define MG_CONV_WIDE 0
#endif
int conv_tile_n(const ConvProblem &p) {
    return (MG_CONV_WIDE && p.C % 4 == 0 && p.C >= 128) ? 128 : 64;
}

int conv_wgrad_splits(const ConvProblem &p) {
    return splits_for((long)cdiv(p.K, BM) * cdiv(p.R * p.S * p.C, conv_tile_n(p)),
                      cdiv(p.N * p.P * p.Q, BK));
}

namespace {

// The stride-parity classes of the data gradient (see DgradJob), without
// the pointers and split; classes without pixels are left out.
std::vector<DgradJob> dgrad_classes(const ConvProblem &p) {
    std::vector<DgradJob> cls;
    for (int a = 0; a < p.sh; ++a)
        for (int b = 0; b < p.sw; ++b) {
            DgradJob j{};
            j.a = a;
            j.b = b;
            j.Hc = a < p.H ? cdiv(p.H - a, p.sh) : 0;
            j.Wc = b < p.W ? cdiv(p.W - b, p.sw) : 0;
            if (j.Hc == 0 || j.Wc == 0) continue;
            j.r0 = (a + p.ph) % p.sh;
            j.s0 = (b + p.pw) % p.sw;
            j.Rc = j.r0 < p.R ? cdiv(p.R - j.r0, p.sh) : 0;
            j.Sc = j.s0 < p.S ? cdiv(p.S - j.s0, p.sw) : 0;
            j.da = (a + p.ph - j.r0) / p.sh;
            j.db = (b + p.pw - j.s0) / p.sw;
            j.HWc = make_fastdiv(j.Hc * j.Wc);
            j.Wc_ = make_fastdiv(j.Wc);
            j.Sc_ = make_fastdiv(j.Sc > 0 ? j.Sc : 1);
            j.tiles_c = cdiv(p.C, conv_tile_n(p));
            cls.push_back(j);
        }
    return cls;
}

}  // namespace

// One split count for every class: from the classes' total tiles and the
// longest class reduction.
int conv_dgrad_splits(const ConvProblem &p) {
    long tiles = 0, steps = 0;
    for (const DgradJob &j : dgrad_classes(p)) {
        tiles += (long)cdiv(p.N * j.Hc * j.Wc, BM) * j.tiles_c;
        steps = std::max<long>(steps, cdiv(j.Rc * j.Sc * p.K, BK));
    }
    return splits_for(tiles, steps);
}

namespace {

WgradJob wgrad_job(const ConvProblem &p, const float *X, const float *dY, float *dW,
                   float *partials) {
    const int ns = conv_wgrad_splits(p);
    const int tiles_j = cdiv(p.R * p.S * p.C, conv_tile_n(p));
    return WgradJob{X, dY, ns > 1 ? partials : dW, tiles_j, ns, cdiv(p.N * p.P * p.Q, BK),
                    cdiv(p.K, BM) * tiles_j * ns};
}

// The data gradient's class jobs, in launches of at most kMaxClasses.
std::vector<DgradJobs> dgrad_jobs(const ConvProblem &p, const float *dY, const float *Wt,
                                  float *dX, float *partials) {
    const int ns = conv_dgrad_splits(p);
    std::vector<DgradJobs> launches;
    for (DgradJob j : dgrad_classes(p)) {
        j.dY = dY;
        j.Wt = Wt;
        j.out = ns > 1 ? partials : dX;
        j.nsplit = ns;
        j.blocks = cdiv(p.N * j.Hc * j.Wc, BM) * j.tiles_c * ns;
        if (launches.empty() || launches.back().n == kMaxClasses) launches.push_back(DgradJobs{});
        DgradJobs &l = launches.back();
        l.c[l.n++] = j;
    }
    return launches;
}

int total_blocks(const DgradJobs &d) {
    int b = 0;
    for (int i = 0; i < d.n; ++i) b += d.c[i].blocks;
    return b;
}

ReduceJob reduce_job(const float *partials, int nsplit, int total, float *out) {
    // lanes per element group: about nsplit / 4 splits each, at most 64
    int G = 1;
    while (G < 64 && 4 * G < nsplit) G *= 2;
    const int vec = total % 4 == 0;
    const long groups = vec ? total / 4 : total;
    return ReduceJob{partials, out, nsplit, total, G, vec, (int)((groups * G + 255) / 256)};
}

// The kernel instance for the operands' vector widths (16-byte loads along
// k when K % 4 == 0 and along c when C % 4 == 0, else 4-byte loads) and the
// output tile width.
template <template <int, int, int> class Launch, typename... Args>
hipError_t by_widths(const ConvProblem &p, Args &&...args) {
    const bool va = p.K % 4 == 0, vb = p.C % 4 == 0;
#if MG_CONV_WIDE
    if (conv_tile_n(p) == 128) {
        if (va) return Launch<4, 4, 128>::run(args...);
        return Launch<1, 4, 128>::run(args...);
    }
#endif
    if (va && vb) return Launch<4, 4, 64>::run(args...);
    if (va) return Launch<4, 1, 64>::run(args...);
    if (vb) return Launch<1, 4, 64>::run(args...);
    return Launch<1, 1, 64>::run(args...);
}

template <int VA, int VB, int TN>
struct LaunchW {
    static hipError_t run(const WgradJob &j, const ConvProblem &p, const ConvDivs &dv,
                          hipStream_t s) {
        conv_wgrad_f32<VA, VB, TN><<<dim3(j.blocks), dim3(NT), 0, s>>>(j, p, dv);
        return hipGetLastError();
    }
};
template <int VA, int VB, int TN>
struct LaunchD {
    static hipError_t run(const DgradJobs &j, const ConvProblem &p, const ConvDivs &dv,
                          hipStream_t s) {
        conv_dgrad_f32<VA, VB, TN><<<dim3(total_blocks(j)), dim3(NT), 0, s>>>(j, p, dv);
        return hipGetLastError();
    }
};
template <int VA, int VB, int TN>
struct LaunchDW {
    static hipError_t run(const DgradJobs &d, const WgradJob &w, const ConvProblem &p,
                          const ConvDivs &dv, hipStream_t s) {
        const int db = total_blocks(d);
        conv_bwd_f32<VA, VB, TN><<<dim3(db + w.blocks), dim3(NT), 0, s>>>(d, db, w, p, dv);
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
    if (conv_dgrad_splits(p) > 1 && partials == nullptr) return hipErrorInvalidValue;
    const ConvDivs dv = make_divs(p);
    for (const DgradJobs &j : dgrad_jobs(p, dY, Wt, dX, partials)) {
        const hipError_t e = by_widths<LaunchD>(p, j, p, dv, s);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_conv_bwd_f32(const ConvProblem &p, const float *X, const float *Wt,
                               const float *dY, float *dX, float *dW, float *dpart,
                               float *wpart, hipStream_t s) {
    const WgradJob w = wgrad_job(p, X, dY, dW, wpart);
    if ((conv_dgrad_splits(p) > 1 && dpart == nullptr) || (w.nsplit > 1 && wpart == nullptr))
        return hipErrorInvalidValue;
    const ConvDivs dv = make_divs(p);
    const std::vector<DgradJobs> d = dgrad_jobs(p, dY, Wt, dX, dpart);
    // the filter gradient shares the first launch; strides beyond 4 x 4 add
    // data-gradient-only launches for the remaining classes
    hipError_t e = by_widths<LaunchDW>(p, d[0], w, p, dv, s);
    for (size_t i = 1; i < d.size() && e == hipSuccess; ++i) e = by_widths<LaunchD>(p, d[i], p, dv, s);
    return e;
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
