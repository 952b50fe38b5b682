// attn_bf16.hip -- fast_bf16 attention kernels for gfx950 (bf16 MFMA, f32
// accumulation).
//
// Same three-kernel structure as the strict-f32 path (tiled forward, fused
// dK+dV with the key tile stationary, separate dQ; the paper's attention
// archetype, Sec. 3.3 and Sec. 8), on v_mfma_f32_16x16x32_bf16.  The
// reduced-input contract of Sec. 4.2 rounds matrix inputs locally and
// accumulates in f32; here Q, K, V, O, dO and the gradients are stored bf16,
// and the softmax probabilities P and dS are rounded to bf16 (nearest even)
// only as inputs of the second product of each pass.  Softmax statistics,
// LSE and D stay f32.
//
// Contraction order inside one 16x16x32 product: for products over the head
// dimension a lane holds d = 32s + 8g + e (e = 0..7, g = lane/16), one
// 16-byte load; for products over streamed rows it holds row
// 32t + 16*(e/4) + 4g + e%4, which is exactly the pair of 16x16 accumulator
// blocks (2t, 2t+1) a lane already owns, so P and dS become the B operand
// without leaving registers, and the LDS operand is read transposed.
#include "device_common.h"
#include "launch.h"
#include "tiles_bf16.h"

namespace mg {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kStatRows = 16 * kWaves;   // stationary rows per workgroup
constexpr int kStream = 64;              // streamed rows per step
constexpr int kBlk = kStream / 16;       // 16-row blocks per streamed tile

// Stationary operand of a wave: row `row` of X, d = 32s + 8g + e.
template <int D>
__device__ __forceinline__ void load_stationary(bf16x8 (&reg)[D / 32], const uint16_t *X,
                                                int row, int L, int g) {
#pragma unroll
    for (int s = 0; s < D / 32; ++s) {
        if (row < L) {
            reg[s] = load_bf16x8(X + (size_t)row * D + 32 * s + 8 * g);
        } else {
            reg[s] = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
        }
    }
}

// ---------------------------------------------------------------- forward --
template <int D>
__global__ __launch_bounds__(kThreads) void attn_fwd_bf16(
    const uint16_t *__restrict__ Q, const uint16_t *__restrict__ K,
    const uint16_t *__restrict__ V, uint16_t *__restrict__ O, float *__restrict__ LSE,
    const int32_t *__restrict__ key_len, int H, int L, int causal, float scale_log2,
    int n_qtiles, int BH) {
    constexpr int NS = D / 32;
    constexpr int NC = D / 16;
    using KSt = Bf16TileStager<kStream, D, kThreads, true, false>;
    using VSt = Bf16TileStager<kStream, D, kThreads, false, true>;
    __shared__ __attribute__((aligned(16))) uint16_t Kr[kStream][KSt::kLdR];
    __shared__ __attribute__((aligned(16))) uint16_t Vt[D][VSt::kLdT];

    const int rank = blockIdx.x / BH;
    const int head = blockIdx.x - rank * BH;
    const int qt = causal ? (n_qtiles - 1 - rank) : rank;
    const int b = head / H;
    const size_t hoff = (size_t)head * L * D;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int il = lane & 15;
    const int g = lane >> 4;
    const int q0 = qt * kStatRows;
    const int qi = q0 + 16 * (tid >> 6) + il;

    const int klen = key_limit(key_len, b, L);
    const int kend = causal ? min(klen, q0 + kStatRows) : klen;
    const int ntiles = (kend + kStream - 1) / kStream;

    bf16x8 qreg[NS];
    load_stationary<D>(qreg, Q + hoff, qi, L, g);

    float m_run = -INFINITY, l_run = 0.f;
    f32x4 oacc[NC];   // O^T[16c + 4g + r][qi]
#pragma unroll
    for (int c = 0; c < NC; ++c) oacc[c] = zero4();

    KSt kst;
    VSt vst;
    if (ntiles > 0) {
        kst.load(K + hoff, 0, L, tid);
        vst.load(V + hoff, 0, L, tid);
    }
    for (int kt = 0; kt < ntiles; ++kt) {
        __syncthreads();
        kst.store(Kr, nullptr, tid);
        vst.store(nullptr, Vt, tid);
        __syncthreads();
        if (kt + 1 < ntiles) {
            kst.load(K + hoff, (kt + 1) * kStream, L, tid);
            vst.load(V + hoff, (kt + 1) * kStream, L, tid);
        }

        f32x4 sacc[kBlk];
#pragma unroll
        for (int jb = 0; jb < kBlk; ++jb) sacc[jb] = zero4();
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
            for (int jb = 0; jb < kBlk; ++jb)
                sacc[jb] = mfma16x16x32bf16(load_bf16x8(&Kr[16 * jb + il][32 * s + 8 * g]),
                                            qreg[s], sacc[jb]);

        const int j0 = kt * kStream + 4 * g;
        float mx = -INFINITY;
#pragma unroll
        for (int jb = 0; jb < kBlk; ++jb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int j = j0 + 16 * jb + r;
                const bool ok = (j < klen) && (!causal || j <= qi);
                const float t = ok ? sacc[jb][r] * scale_log2 : -INFINITY;
                sacc[jb][r] = t;
                mx = fmaxf(mx, t);
            }
        mx = max_over_groups(mx);
        const float m_new = fmaxf(m_run, mx);
        const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
        const float alpha = exp2_fast(m_run - m_use);
        float psum = 0.f;
#pragma unroll
        for (int jb = 0; jb < kBlk; ++jb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float p = exp2_fast(sacc[jb][r] - m_use);
                sacc[jb][r] = p;
                psum += p;
            }
        l_run = l_run * alpha + psum;
        m_run = m_new;
#pragma unroll
        for (int c = 0; c < NC; ++c) oacc[c] *= alpha;

        // O^T[16c + 4g + r][qi] += sum_j V^T[16c + il'][j] P^T[j][qi]
#pragma unroll
        for (int t = 0; t < kBlk / 2; ++t) {
            const bf16x8 pb = pack_bf16(sacc[2 * t], sacc[2 * t + 1]);
#pragma unroll
            for (int c = 0; c < NC; ++c)
                oacc[c] = mfma16x16x32bf16(
                    load_bf16x4x2(&Vt[16 * c + il][32 * t + 4 * g],
                                  &Vt[16 * c + il][32 * t + 16 + 4 * g]),
                    pb, oacc[c]);
        }
    }

    const float l = sum_over_groups(l_run);
    if (qi < L) {
        const float inv = (l > 0.f) ? 1.f / l : 0.f;
        uint16_t *orow = O + hoff + (size_t)qi * D;
#pragma unroll
        for (int c = 0; c < NC; ++c) store_bf16x4(orow + 16 * c + 4 * g, oacc[c] * inv);
        if (g == 0)
            LSE[(size_t)head * L + qi] = (l > 0.f) ? (m_run + log2f(l)) * kLn2 : -INFINITY;
    }
}

// ------------------------------------------------- backward: D = rowsum(dO o O)
template <int D>
__global__ __launch_bounds__(256) void attn_rowdot_bf16(const uint16_t *__restrict__ O,
                                                        const uint16_t *__restrict__ dO,
                                                        float *__restrict__ Dws, int rows) {
    constexpr int TPR = D / 8;   // threads per row, 8 bf16 each
    const int row = blockIdx.x * (256 / TPR) + threadIdx.x / TPR;
    const int c8 = threadIdx.x % TPR;
    float v = 0.f;
    if (row < rows) {
        const u32x4 o = *reinterpret_cast<const u32x4 *>(O + (size_t)row * D + 8 * c8);
        const u32x4 go = *reinterpret_cast<const u32x4 *>(dO + (size_t)row * D + 8 * c8);
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            v += __uint_as_float(o[m] << 16) * __uint_as_float(go[m] << 16);
            v += __uint_as_float(o[m] & 0xffff0000u) * __uint_as_float(go[m] & 0xffff0000u);
        }
    }
#pragma unroll
    for (int m = TPR / 2; m >= 1; m >>= 1) v += xor_lanes(v, m);
    if (row < rows && c8 == 0) Dws[row] = v;
}

// ------------------------------------------------------- backward: dK, dV
template <int D>
__global__ __launch_bounds__(kThreads) void attn_dkdv_bf16(
    const uint16_t *__restrict__ Q, const uint16_t *__restrict__ K,
    const uint16_t *__restrict__ V, const uint16_t *__restrict__ dO,
    const float *__restrict__ LSE, const float *__restrict__ Dws, uint16_t *__restrict__ dK,
    uint16_t *__restrict__ dV, const int32_t *__restrict__ key_len, int H, int L, int causal,
    float scale, float scale_log2, int BH) {
    constexpr int NS = D / 32;
    constexpr int NC = D / 16;
    using St = Bf16TileStager<kStream, D, kThreads, true, true>;
    __shared__ __attribute__((aligned(16))) uint16_t Qr[kStream][St::kLdR];
    __shared__ __attribute__((aligned(16))) uint16_t Qt[D][St::kLdT];
    __shared__ __attribute__((aligned(16))) uint16_t Or[kStream][St::kLdR];
    __shared__ __attribute__((aligned(16))) uint16_t Ot[D][St::kLdT];
    __shared__ __attribute__((aligned(16))) float lse2s[kStream];
    __shared__ __attribute__((aligned(16))) float Ds[kStream];

    const int rank = blockIdx.x / BH;
    const int head = blockIdx.x - rank * BH;
    const int kt = rank;
    const int b = head / H;
    const size_t hoff = (size_t)head * L * D;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int il = lane & 15;
    const int g = lane >> 4;
    const int k0 = kt * kStatRows;
    const int kj = k0 + 16 * (tid >> 6) + il;

    const int klen = key_limit(key_len, b, L);
    const int nq = (L + kStream - 1) / kStream;
    const int qstart = causal ? (k0 / kStream) : 0;
    const int qstop = (k0 < klen) ? nq : qstart;

    bf16x8 kreg[NS], vreg[NS];
    load_stationary<D>(kreg, K + hoff, kj, L, g);
    load_stationary<D>(vreg, V + hoff, kj, L, g);

    f32x4 dkacc[NC], dvacc[NC];   // dK^T[16c + 4g + r][kj], dV^T likewise
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        dkacc[c] = zero4();
        dvacc[c] = zero4();
    }

    St qst, ost;
    float lse_pre = 0.f, d_pre = 0.f;
    auto load_rows = [&](int qt) {
        qst.load(Q + hoff, qt * kStream, L, tid);
        ost.load(dO + hoff, qt * kStream, L, tid);
        if (tid < kStream) {
            const int row = qt * kStream + tid;
            lse_pre = (row < L) ? LSE[(size_t)head * L + row] * kLog2e : 0.f;
            d_pre = (row < L) ? Dws[(size_t)head * L + row] : 0.f;
        }
    };
    if (qstart < qstop) load_rows(qstart);

    for (int qt = qstart; qt < qstop; ++qt) {
        __syncthreads();
        qst.store(Qr, Qt, tid);
        ost.store(Or, Ot, tid);
        if (tid < kStream) {
            lse2s[tid] = lse_pre;
            Ds[tid] = d_pre;
        }
        __syncthreads();
        if (qt + 1 < qstop) load_rows(qt + 1);

        f32x4 sacc[kBlk], pacc[kBlk];
#pragma unroll
        for (int ib = 0; ib < kBlk; ++ib) {
            sacc[ib] = zero4();
            pacc[ib] = zero4();
        }
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
            for (int ib = 0; ib < kBlk; ++ib) {
                sacc[ib] = mfma16x16x32bf16(load_bf16x8(&Qr[16 * ib + il][32 * s + 8 * g]),
                                            kreg[s], sacc[ib]);
                pacc[ib] = mfma16x16x32bf16(load_bf16x8(&Or[16 * ib + il][32 * s + 8 * g]),
                                            vreg[s], pacc[ib]);
            }

        const int ibase = qt * kStream + 4 * g;
#pragma unroll
        for (int ib = 0; ib < kBlk; ++ib) {
            const f32x4 l2 = *reinterpret_cast<const f32x4 *>(&lse2s[16 * ib + 4 * g]);
            const f32x4 dd = *reinterpret_cast<const f32x4 *>(&Ds[16 * ib + 4 * g]);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int i = ibase + 16 * ib + r;
                const bool ok = (i < L) && (kj < klen) && (!causal || kj <= i);
                const float p = ok ? exp2_fast(sacc[ib][r] * scale_log2 - l2[r]) : 0.f;
                sacc[ib][r] = p;
                pacc[ib][r] = p * (pacc[ib][r] - dd[r]);
            }
        }

#pragma unroll
        for (int t = 0; t < kBlk / 2; ++t) {
            const bf16x8 pb = pack_bf16(sacc[2 * t], sacc[2 * t + 1]);
            const bf16x8 sb = pack_bf16(pacc[2 * t], pacc[2 * t + 1]);
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                dvacc[c] = mfma16x16x32bf16(
                    load_bf16x4x2(&Ot[16 * c + il][32 * t + 4 * g],
                                  &Ot[16 * c + il][32 * t + 16 + 4 * g]),
                    pb, dvacc[c]);
                dkacc[c] = mfma16x16x32bf16(
                    load_bf16x4x2(&Qt[16 * c + il][32 * t + 4 * g],
                                  &Qt[16 * c + il][32 * t + 16 + 4 * g]),
                    sb, dkacc[c]);
            }
        }
    }

    if (kj < L) {
        uint16_t *dkrow = dK + hoff + (size_t)kj * D;
        uint16_t *dvrow = dV + hoff + (size_t)kj * D;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            store_bf16x4(dkrow + 16 * c + 4 * g, dkacc[c] * scale);
            store_bf16x4(dvrow + 16 * c + 4 * g, dvacc[c]);
        }
    }
}

// ------------------------------------------------------------ backward: dQ
template <int D>
__global__ __launch_bounds__(kThreads) void attn_dq_bf16(
    const uint16_t *__restrict__ Q, const uint16_t *__restrict__ K,
    const uint16_t *__restrict__ V, const uint16_t *__restrict__ dO,
    const float *__restrict__ LSE, const float *__restrict__ Dws, uint16_t *__restrict__ dQ,
    const int32_t *__restrict__ key_len, int H, int L, int causal, float scale,
    float scale_log2, int n_qtiles, int BH) {
    constexpr int NS = D / 32;
    constexpr int NC = D / 16;
    using KSt = Bf16TileStager<kStream, D, kThreads, true, true>;
    using VSt = Bf16TileStager<kStream, D, kThreads, true, false>;
    __shared__ __attribute__((aligned(16))) uint16_t Kr[kStream][KSt::kLdR];
    __shared__ __attribute__((aligned(16))) uint16_t Kt[D][KSt::kLdT];
    __shared__ __attribute__((aligned(16))) uint16_t Vr[kStream][VSt::kLdR];

    const int rank = blockIdx.x / BH;
    const int head = blockIdx.x - rank * BH;
    const int qt = causal ? (n_qtiles - 1 - rank) : rank;
    const int b = head / H;
    const size_t hoff = (size_t)head * L * D;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int il = lane & 15;
    const int g = lane >> 4;
    const int q0 = qt * kStatRows;
    const int qi = q0 + 16 * (tid >> 6) + il;

    const int klen = key_limit(key_len, b, L);
    const int kend = causal ? min(klen, q0 + kStatRows) : klen;
    const int ntiles = (kend + kStream - 1) / kStream;

    bf16x8 qreg[NS], oreg[NS];
    load_stationary<D>(qreg, Q + hoff, qi, L, g);
    load_stationary<D>(oreg, dO + hoff, qi, L, g);
    const float lse2 = (qi < L) ? LSE[(size_t)head * L + qi] * kLog2e : 0.f;
    const float Di = (qi < L) ? Dws[(size_t)head * L + qi] : 0.f;

    f32x4 dqacc[NC];   // dQ^T[16c + 4g + r][qi]
#pragma unroll
    for (int c = 0; c < NC; ++c) dqacc[c] = zero4();

    KSt kst;
    VSt vst;
    if (ntiles > 0) {
        kst.load(K + hoff, 0, L, tid);
        vst.load(V + hoff, 0, L, tid);
    }
    for (int kt = 0; kt < ntiles; ++kt) {
        __syncthreads();
        kst.store(Kr, Kt, tid);
        vst.store(Vr, nullptr, tid);
        __syncthreads();
        if (kt + 1 < ntiles) {
            kst.load(K + hoff, (kt + 1) * kStream, L, tid);
            vst.load(V + hoff, (kt + 1) * kStream, L, tid);
        }

        f32x4 sacc[kBlk], pacc[kBlk];
#pragma unroll
        for (int jb = 0; jb < kBlk; ++jb) {
            sacc[jb] = zero4();
            pacc[jb] = zero4();
        }
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
            for (int jb = 0; jb < kBlk; ++jb) {
                sacc[jb] = mfma16x16x32bf16(load_bf16x8(&Kr[16 * jb + il][32 * s + 8 * g]),
                                            qreg[s], sacc[jb]);
                pacc[jb] = mfma16x16x32bf16(load_bf16x8(&Vr[16 * jb + il][32 * s + 8 * g]),
                                            oreg[s], pacc[jb]);
            }

        const int j0 = kt * kStream + 4 * g;
#pragma unroll
        for (int jb = 0; jb < kBlk; ++jb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int j = j0 + 16 * jb + r;
                const bool ok = (qi < L) && (j < klen) && (!causal || j <= qi);
                const float p = ok ? exp2_fast(sacc[jb][r] * scale_log2 - lse2) : 0.f;
                pacc[jb][r] = p * (pacc[jb][r] - Di);
            }

#pragma unroll
        for (int t = 0; t < kBlk / 2; ++t) {
            const bf16x8 sb = pack_bf16(pacc[2 * t], pacc[2 * t + 1]);
#pragma unroll
            for (int c = 0; c < NC; ++c)
                dqacc[c] = mfma16x16x32bf16(
                    load_bf16x4x2(&Kt[16 * c + il][32 * t + 4 * g],
                                  &Kt[16 * c + il][32 * t + 16 + 4 * g]),
                    sb, dqacc[c]);
        }
    }

    if (qi < L) {
        uint16_t *dqrow = dQ + hoff + (size_t)qi * D;
#pragma unroll
        for (int c = 0; c < NC; ++c) store_bf16x4(dqrow + 16 * c + 4 * g, dqacc[c] * scale);
    }
}

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

}  // namespace

// ---------------------------------------------------------------- launchers
hipError_t launch_fwd_bf16(const AttnProblem &p, const uint16_t *Q, const uint16_t *K,
                           const uint16_t *V, uint16_t *O, float *LSE, hipStream_t s) {
    const int BH = p.B * p.H;
    const int nqt = cdiv(p.L, kStatRows);
    const dim3 grid(nqt * BH), block(kThreads);
    const float sl2 = p.scale * kLog2e;
    switch (p.d) {
    case 32: attn_fwd_bf16<32><<<grid, block, 0, s>>>(Q, K, V, O, LSE, p.key_len, p.H, p.L, p.causal, sl2, nqt, BH); break;
    case 64: attn_fwd_bf16<64><<<grid, block, 0, s>>>(Q, K, V, O, LSE, p.key_len, p.H, p.L, p.causal, sl2, nqt, BH); break;
    case 128: attn_fwd_bf16<128><<<grid, block, 0, s>>>(Q, K, V, O, LSE, p.key_len, p.H, p.L, p.causal, sl2, nqt, BH); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_bwd_rowdot_bf16(const AttnProblem &p, const uint16_t *O, const uint16_t *dO,
                                  float *Dws, hipStream_t s) {
    const int rows = p.B * p.H * p.L;
    const dim3 block(256);
    switch (p.d) {
    case 32: attn_rowdot_bf16<32><<<dim3(cdiv(rows, 256 / 4)), block, 0, s>>>(O, dO, Dws, rows); break;
    case 64: attn_rowdot_bf16<64><<<dim3(cdiv(rows, 256 / 8)), block, 0, s>>>(O, dO, Dws, rows); break;
    case 128: attn_rowdot_bf16<128><<<dim3(cdiv(rows, 256 / 16)), block, 0, s>>>(O, dO, Dws, rows); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_bwd_dkdv_bf16(const AttnProblem &p, const uint16_t *Q, const uint16_t *K,
                                const uint16_t *V, const uint16_t *dO, const float *LSE,
                                const float *Dws, uint16_t *dK, uint16_t *dV, hipStream_t s) {
    const int BH = p.B * p.H;
    const dim3 grid(cdiv(p.L, kStatRows) * BH), block(kThreads);
    const float sl2 = p.scale * kLog2e;
    switch (p.d) {
    case 32: attn_dkdv_bf16<32><<<grid, block, 0, s>>>(Q, K, V, dO, LSE, Dws, dK, dV, p.key_len, p.H, p.L, p.causal, p.scale, sl2, BH); break;
    case 64: attn_dkdv_bf16<64><<<grid, block, 0, s>>>(Q, K, V, dO, LSE, Dws, dK, dV, p.key_len, p.H, p.L, p.causal, p.scale, sl2, BH); break;
    case 128: attn_dkdv_bf16<128><<<grid, block, 0, s>>>(Q, K, V, dO, LSE, Dws, dK, dV, p.key_len, p.H, p.L, p.causal, p.scale, sl2, BH); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_bwd_dq_bf16(const AttnProblem &p, const uint16_t *Q, const uint16_t *K,
                              const uint16_t *V, const uint16_t *dO, const float *LSE,
                              const float *Dws, uint16_t *dQ, hipStream_t s) {
    const int BH = p.B * p.H;
    const int nqt = cdiv(p.L, kStatRows);
    const dim3 grid(nqt * BH), block(kThreads);
    const float sl2 = p.scale * kLog2e;
    switch (p.d) {
    case 32: attn_dq_bf16<32><<<grid, block, 0, s>>>(Q, K, V, dO, LSE, Dws, dQ, p.key_len, p.H, p.L, p.causal, p.scale, sl2, nqt, BH); break;
    case 64: attn_dq_bf16<64><<<grid, block, 0, s>>>(Q, K, V, dO, LSE, Dws, dQ, p.key_len, p.H, p.L, p.causal, p.scale, sl2, nqt, BH); break;
    case 128: attn_dq_bf16<128><<<grid, block, 0, s>>>(Q, K, V, dO, LSE, Dws, dQ, p.key_len, p.H, p.L, p.causal, p.scale, sl2, nqt, BH); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace mg
