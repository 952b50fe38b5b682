// attn_accel.hip -- forward attention under the paper's practical default
// (accelerated) arithmetic contract, for gfx950.
//
// The paper's arithmetic permissions (Sec. 4.2, table of arithmetic
// permissions): persistent tensors and outputs are f32; eligible forward
// matrix and attention inputs may be rounded locally to f16 and multiplied
// with f32 accumulation; backward matrices stay f32.  Here Q, K, V are f32 in
// HBM, rounded to f16 (nearest even) as they enter the matrix cores, the
// probabilities P are rounded to f16 as the operand of P V, and O and LSE are
// written in f32.  The backward under this contract is the strict-f32 one.
//
// Structure as the bf16 forward (32 queries per wave on
// v_mfma_f32_32x32x16_f16, K and V streamed 64 keys at a time through padded
// row-major LDS tiles, V^T operands by 16-bit transpose reads), except that
// the f32 tiles pass through registers to be rounded.  For d = 128 the plain
// form: the next K tile is loaded while S of the current tile runs and
// written to LDS (as f16) after the barrier that frees it, the next V tile
// likewise during P V, and since the two never overlap in time one set of
// staging registers serves both.  For d <= 64 the software-pipelined form
// below (double-buffered K and V, one barrier per tile).
#include "device_common.h"
#include "launch.h"
#include "tiles_bf16.h"

namespace mg {
namespace {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kRows = 32 * kWaves;   // queries per workgroup
constexpr int kKeys = 64;            // keys per streamed tile

__device__ __forceinline__ f32x16 mfma32x32x16f16(f16x8 a, f16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

// Eight f32 -> eight f16 (nearest even).
__device__ __forceinline__ f16x8 to_f16x8(f32x4 lo, f32x4 hi) {
    f16x8 v;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        v[e] = (_Float16)lo[e];
        v[4 + e] = (_Float16)hi[e];
    }
    return v;
}

// Accumulator registers [8t, 8t+8) of a 32x32 block rounded to f16, as the B
// operand of a 32x32x16 product contracting over its rows.
__device__ __forceinline__ f16x8 pack_f16_half(const f32x16 &a, int t) {
    f16x8 v;
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = (_Float16)a[8 * t + e];
    return v;
}

// An f32 [ROWS][D] tile staged through registers and written to LDS as f16
// (row stride LDD in 16-bit units, a parameter of the store).  Chunk f (4 floats) of the tile is row
// f / (D/4), columns 4*(f % (D/4)); consecutive threads take consecutive
// chunks, so global reads are coalesced and LDS writes contiguous per row.
// Rows at or beyond L read as zeros (buffer descriptor over rows below L).
template <int ROWS, int D, int NT>
struct F16ConvStager {
    static constexpr int kCpr = D / 4;
    static constexpr int kPer = ROWS * kCpr / NT;
    static_assert(ROWS * kCpr % NT == 0, "tile must split evenly over the threads");
    f32x4 buf[kPer];

    __device__ __forceinline__ void load(const float *__restrict__ src, int row0, int L,
                                         int tid) {
        const int rows = min(max(L - row0, 0), ROWS);
        const auto rsrc = buffer_rsrc(src + (size_t)row0 * D, rows * D * 4);
#pragma unroll
        for (int u = 0; u < kPer; ++u) buf[u] = buffer_load_f32x4(rsrc, 16 * (tid + u * NT));
    }
    template <int LDD>
    __device__ __forceinline__ void store(uint16_t (*dst)[LDD], int tid) const {
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
            const int f = tid + u * NT;
            const int r = f / kCpr;
            const int c4 = f - r * kCpr;
            f16x4 h;
#pragma unroll
            for (int e = 0; e < 4; ++e) h[e] = (_Float16)buf[u][e];
            *reinterpret_cast<uint64_t *>(&dst[r][4 * c4]) = __builtin_bit_cast(uint64_t, h);
        }
    }
};

template <int D, bool POS_SCALE>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 8)))
void attn_fwd_accel(const float *__restrict__ Q, const float *__restrict__ K,
                    const float *__restrict__ V, float *__restrict__ O, float *__restrict__ LSE,
                    const int32_t *__restrict__ key_len, int H, int Lq, int Lk, int causal,
                    float scale_log2, int n_qtiles, int BH, int layer) {
    constexpr int NS = D / 16;    // 16-deep contraction steps over d
    constexpr int NCB = D / 32;   // 32-column blocks of d
    constexpr int NKB = kKeys / 32;
    constexpr int LD = Bf16Ld<D>::value;     // K rows: 16-byte reads of 32 rows
    constexpr int LDV = Bf16LdTr<D>::value;  // V rows: transpose reads only
    using St = F16ConvStager<kKeys, D, kThreads>;
    __shared__ __attribute__((aligned(16))) uint16_t Kr[kKeys][LD];
    __shared__ __attribute__((aligned(16))) uint16_t Vr[kKeys][LDV];

    const int slot = blockIdx.x / BH;
    const int head = blockIdx.x - slot * BH;
    const int rank = serpentine_rank(slot, n_qtiles, layer);
    const int qt = causal ? (n_qtiles - 1 - rank) : rank;
    const int b = head / H;
    const size_t qoff = (size_t)head * Lq * D, hoff = (size_t)head * Lk * D;
    const float *Kh = K + hoff;
    const float *Vh = V + hoff;
    const int diag = Lk - Lq;   // causal: row i sees keys j <= i + diag

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c = lane & 31;
    const int h = lane >> 5;
    const int jr = (lane & 15) >> 2, jc = 4 * (lane & 3);   // transpose-read block offsets
    const int q0 = qt * kRows;
    const int qi = q0 + 32 * w + c;

    const int klen = key_limit(key_len, b, Lk);
    const int kend = causal ? min(klen, q0 + kRows + diag) : klen;
    const int ntiles = (kend + kKeys - 1) / kKeys;

    // B operand of S^T = K Q^T: lane holds f16(Q[qi][16s + 8h + e]).
    f16x8 qreg[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        const float *qp = Q + qoff + (size_t)qi * D + 16 * s + 8 * h;
        qreg[s] = (qi < Lq) ? to_f16x8(*reinterpret_cast<const f32x4 *>(qp),
                                      *reinterpret_cast<const f32x4 *>(qp + 4))
                           : f16x8{};
    }

    St st;
    if (ntiles > 0) {
        st.load(Kh, 0, Lk, tid);
        st.store(Kr, tid);
        st.load(Vh, 0, Lk, tid);
        st.store(Vr, tid);
        if (ntiles > 1) st.load(Kh, kKeys, Lk, tid);
    }
    __syncthreads();

    // Running max in raw-score units when POS_SCALE, else in base-2 units.
    float m_run = -INFINITY, l_run = 0.f;
    f32x16 oacc[NCB];   // O^T[32cb + 8a + 4h + r][qi] in register 4a + r
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) oacc[cb] = zero16();

    for (int kt = 0; kt < ntiles; ++kt) {
        // S^T[32kb + 8a + 4h + r][qi] in sacc[kb] register 4a + r
        f32x16 sacc[NKB];
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
            sacc[kb] = zero16();
#pragma unroll
            for (int s = 0; s < NS; ++s)
                sacc[kb] = mfma32x32x16f16(
                    __builtin_bit_cast(f16x8, *reinterpret_cast<const u32x4 *>(
                                                  &Kr[32 * kb + c][16 * s + 8 * h])),
                    qreg[s], sacc[kb]);
        }
        __syncthreads();   // every wave is done with K(kt)
        if (kt + 1 < ntiles) {
            st.store(Kr, tid);                      // K(kt+1), loaded during S(kt)
            st.load(Vh, (kt + 1) * kKeys, Lk, tid);  // V(kt+1), lands during P V(kt)
        }
        if (!POS_SCALE) {
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) sacc[kb] *= scale_log2;
        }

        // Masking only where the tile crosses the diagonal or the key length.
        const bool full = (kt + 1) * kKeys <= klen && (!causal || (kt + 1) * kKeys - 1 <= q0 + diag);
        if (!full) {
            const int j0 = kt * kKeys + 4 * h;
            const int thr = causal ? min(klen - j0, qi + diag - j0 + 1) : klen - j0;
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    if (32 * kb + 8 * (v >> 2) + (v & 3) >= thr) sacc[kb][v] = -INFINITY;
        }
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
            for (int v = 0; v < 16; v += 2) mx = max3_f32(mx, sacc[kb][v], sacc[kb][v + 1]);
        mx = max_xor32(mx);
        // The running maximum is only an offset: the probabilities are
        // exp2(s - m) for any m at or below the true row maximum, so O and l
        // are rescaled only when some row's maximum grew by more than kSlack
        // (base 2); otherwise the stale m stays and this tile's probabilities
        // are at most 2^kSlack (no overflow, the same relative rounding).
        const float grow2 = POS_SCALE ? (mx - m_run) * scale_log2 : mx - m_run;
        if (__any(grow2 > kSlack)) {
            const float m_new = fmaxf(m_run, mx);
            const float m2_old = POS_SCALE ? m_run * scale_log2 : m_run;
            const float m2_new =
                (m_new == -INFINITY) ? 0.f : (POS_SCALE ? m_new * scale_log2 : m_new);
            const float alpha = exp2_fast(m2_old - m2_new);
            l_run *= alpha;
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) oacc[cb] *= alpha;
            m_run = m_new;
        }
        // exponent offset in base-2 units; a row with nothing allowed yet
        // keeps all-zero probabilities
        const float m2 = (m_run == -INFINITY) ? 0.f : (POS_SCALE ? m_run * scale_log2 : m_run);
        float psum = 0.f;
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const float p = POS_SCALE ? exp2_fast(fmaf(sacc[kb][v], scale_log2, -m2))
                                          : exp2_fast(sacc[kb][v] - m2);
                sacc[kb][v] = p;
                psum += p;
            }
        l_run += psum;

        // O^T[32cb + .][qi] += sum_j V^T[32cb + c'][j] P^T[j][qi], 16 keys per step
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                const f16x8 pb = pack_f16_half(sacc[kb], t);
                const int r0 = 32 * kb + 16 * t + 4 * h;
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb)
                    oacc[cb] = mfma32x32x16f16(
                        __builtin_bit_cast(f16x8, load_tr_pair<LDV>(Vr, r0, r0 + 8,
                                                                   32 * cb + 16 * (c >> 4), jr, jc)),
                        pb, oacc[cb]);
            }

        __syncthreads();   // every wave is done with V(kt); K(kt+1) is visible
        if (kt + 1 < ntiles) {
            st.store(Vr, tid);                                       // V(kt+1)
            if (kt + 2 < ntiles) st.load(Kh, (kt + 2) * kKeys, Lk, tid);   // K(kt+2)
        }
        // V(kt+1) becomes visible at the first barrier of the next iteration,
        // before P V reads it
    }

    const float l = sum_xor32(l_run);
    if (qi < Lq) {
        const float inv = (l > 0.f) ? 1.f / l : 0.f;
        float *orow = O + qoff + (size_t)qi * D;
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
            for (int a = 0; a < 4; ++a)
                *reinterpret_cast<f32x4 *>(orow + 32 * cb + 8 * a + 4 * h) =
                    f32x4{oacc[cb][4 * a], oacc[cb][4 * a + 1], oacc[cb][4 * a + 2],
                          oacc[cb][4 * a + 3]} * inv;
        if (h == 0) {
            const float m2 = POS_SCALE ? m_run * scale_log2 : m_run;
            LSE[(size_t)head * Lq + qi] = (l > 0.f) ? (m2 + log2f(l)) * kLn2 : -INFINITY;
        }
    }
}

// The forward with its key tiles software-pipelined, for d <= 64 (as the bf16
// forward of the same sizes): iteration kt issues the register loads of K(kt+2)
// and V(kt+1), then the score product of tile kt+1, then the softmax and P V of
// tile kt, and only then rounds the staged tiles to f16 and writes them into
// the buffers that the iteration's barrier freed.  Every load has a whole
// iteration to land, and one barrier per tile suffices.  K and V are
// double-buffered.  At d = 128 the second score block and the second staging
// set do not fit two waves per SIMD, and the plain form above is used.
//
// KS = 2 is the key-split form for causal grids that the chip holds in one or
// two rounds: the longest query tile's chain of key tiles, not the total
// work, sets the kernel's time there.  A workgroup of eight waves holds two
// key groups of four; both take the same 128 queries, group 0 the first
// ceil(n/2) of the tile's n key tiles and group 1 the rest, each through its
// own double-buffered K and V.  The groups run the same number of
// iterations (group 1 idles through the last one when n is odd), so the
// workgroup's barriers stay matched.  At the end group 1 leaves its (offset,
// sum, O) state in LDS and group 0 merges it: with offsets m_a, m_b (base 2)
// and m = max(m_a, m_b), l = l_a 2^(m_a - m) + l_b 2^(m_b - m), likewise O.
template <int D, bool POS_SCALE, int KS>
__global__ __launch_bounds__(kThreads * KS) __attribute__((amdgpu_waves_per_eu(2, 8)))
void attn_fwd_accel_pipe(const float *__restrict__ Q, const float *__restrict__ K,
                         const float *__restrict__ V, float *__restrict__ O,
                         float *__restrict__ LSE, const int32_t *__restrict__ key_len, int H,
                         int Lq, int Lk, int causal, float scale_log2, int n_qtiles, int BH,
                         int layer) {
    static_assert(KS == 1 || KS == 2, "one or two key groups");
    constexpr int NS = D / 16;
    constexpr int NCB = D / 32;
    constexpr int NKB = kKeys / 32;
    constexpr int LD = Bf16Ld<D>::value;     // K rows: 16-byte reads of 32 rows
    constexpr int LDV = Bf16LdTr<D>::value;  // V rows: transpose reads only
    using St = F16ConvStager<kKeys, D, kThreads>;
    using KBuf = uint16_t[kKeys][LD];
    using VBuf = uint16_t[kKeys][LDV];
    struct Bufs {
        KBuf K0, K1;
        VBuf V0, V1;
    };
    // Group 1's state for the merge: per query wave and lane, the offset, the
    // sum and the 16 * NCB registers of O^T, slot-major (lane-contiguous).
    constexpr int NX = 2 + 16 * NCB;
    static_assert(KS == 1 || (size_t)kWaves * NX * 64 * sizeof(float) <= KS * sizeof(Bufs),
                  "merge state fits in the tile buffers");
    __shared__ __attribute__((aligned(16))) unsigned char smem[KS * sizeof(Bufs)];

    const int slot = blockIdx.x / BH;
    const int head = blockIdx.x - slot * BH;
    const int rank = serpentine_rank(slot, n_qtiles, layer);
    const int qt = causal ? (n_qtiles - 1 - rank) : rank;
    const int b = head / H;
    const size_t qoff = (size_t)head * Lq * D, hoff = (size_t)head * Lk * D;
    const float *Kh = K + hoff;
    const float *Vh = V + hoff;
    const int diag = Lk - Lq;   // causal: row i sees keys j <= i + diag

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = (KS == 1) ? 0 : w / kWaves;   // key group
    const int wq = w - g * kWaves;              // query wave within the group
    const int tg = tid - g * kThreads;          // thread index within the group
    const int c = lane & 31;
    const int h = lane >> 5;
    const int jr = (lane & 15) >> 2, jc = 4 * (lane & 3);   // transpose-read block offsets
    const int q0 = qt * kRows;
    const int qi = q0 + 32 * wq + c;
    Bufs &bf = *reinterpret_cast<Bufs *>(smem + g * sizeof(Bufs));

    const int klen = key_limit(key_len, b, Lk);
    const int kend = causal ? min(klen, q0 + kRows + diag) : klen;
    const int ntiles = max((kend + kKeys - 1) / kKeys, 0);
    // This group's key tiles [kbeg, kbeg + kcnt); both groups iterate nloop times.
    const int nloop = (KS == 1) ? ntiles : (ntiles + 1) / 2;
    const int kbeg = (KS == 1) ? 0 : g * nloop;
    const int kcnt = (KS == 1) ? ntiles : min(nloop, ntiles - kbeg);

    // B operand of S^T = K Q^T: lane holds f16(Q[qi][16s + 8h + e]).
    f16x8 qreg[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        const float *qp = Q + qoff + (size_t)qi * D + 16 * s + 8 * h;
        qreg[s] = (qi < Lq) ? to_f16x8(*reinterpret_cast<const f32x4 *>(qp),
                                      *reinterpret_cast<const f32x4 *>(qp + 4))
                           : f16x8{};
    }

    float m_run = -INFINITY, l_run = 0.f;
    f32x16 oacc[NCB];   // O^T[32cb + 8a + 4h + r][qi] in register 4a + r
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) oacc[cb] = zero16();

    // S^T[32kb + 8a + 4h + r][qi] in sacc[kb] register 4a + r
    auto scores = [&](const KBuf &Kb, f32x16 (&sacc)[NKB]) {
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
            sacc[kb] = zero16();
#pragma unroll
            for (int s = 0; s < NS; ++s)
                sacc[kb] = mfma32x32x16f16(
                    __builtin_bit_cast(f16x8, *reinterpret_cast<const u32x4 *>(
                                                  &Kb[32 * kb + c][16 * s + 8 * h])),
                    qreg[s], sacc[kb]);
        }
    };
    auto softmax_pv = [&](int kt, f32x16 (&sacc)[NKB], const VBuf &Vb) {
        if (!POS_SCALE) {
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) sacc[kb] *= scale_log2;
        }
        // Masking only where the tile crosses the diagonal or the key length.
        const bool full =
            (kt + 1) * kKeys <= klen && (!causal || (kt + 1) * kKeys - 1 <= q0 + diag);
        if (!full) {
            const int j0 = kt * kKeys + 4 * h;
            const int thr = causal ? min(klen - j0, qi + diag - j0 + 1) : klen - j0;
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    if (32 * kb + 8 * (v >> 2) + (v & 3) >= thr) sacc[kb][v] = -INFINITY;
        }
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
            for (int v = 0; v < 16; v += 2) mx = max3_f32(mx, sacc[kb][v], sacc[kb][v + 1]);
        mx = max_xor32(mx);
        // Rescale O and l only when some row's maximum grew by more than
        // kSlack (base 2), as in the plain form.
        const float grow2 = POS_SCALE ? (mx - m_run) * scale_log2 : mx - m_run;
        if (__any(grow2 > kSlack)) {
            const float m_new = fmaxf(m_run, mx);
            const float m2_old = POS_SCALE ? m_run * scale_log2 : m_run;
            const float m2_new =
                (m_new == -INFINITY) ? 0.f : (POS_SCALE ? m_new * scale_log2 : m_new);
            const float alpha = exp2_fast(m2_old - m2_new);
            l_run *= alpha;
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) oacc[cb] *= alpha;
            m_run = m_new;
        }
        const float m2 = (m_run == -INFINITY) ? 0.f : (POS_SCALE ? m_run * scale_log2 : m_run);
        float psum = 0.f;
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const float p = POS_SCALE ? exp2_fast(fmaf(sacc[kb][v], scale_log2, -m2))
                                          : exp2_fast(sacc[kb][v] - m2);
                sacc[kb][v] = p;
                psum += p;
            }
        l_run += psum;
        // O^T[32cb + .][qi] += sum_j V^T[32cb + c'][j] P^T[j][qi], 16 keys per step
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                const f16x8 pb = pack_f16_half(sacc[kb], t);
                const int r0 = 32 * kb + 16 * t + 4 * h;
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb)
                    oacc[cb] = mfma32x32x16f16(
                        __builtin_bit_cast(f16x8, load_tr_pair<LDV>(Vb, r0, r0 + 8,
                                                                   32 * cb + 16 * (c >> 4), jr, jc)),
                        pb, oacc[cb]);
            }
    };

    // Prologue: K(0) into K0, V(0) into V0, K(1) into K1; S(0).  The
    // group's j-th tile lives in buffer j % 2.
    St sk, sv;
    f32x16 sa[NKB], sb[NKB];
    if (kcnt > 0) {
        sk.load(Kh, kbeg * kKeys, Lk, tg);
        sv.load(Vh, kbeg * kKeys, Lk, tg);
        sk.store(bf.K0, tg);
        sv.store(bf.V0, tg);
        if (kcnt > 1) {
            sk.load(Kh, (kbeg + 1) * kKeys, Lk, tg);
            sk.store(bf.K1, tg);
        }
    }
    __syncthreads();
    if (kcnt > 0) scores(bf.K0, sa);
    // Iteration j: S(j) is in `cur`; K(j+1) is in Kn and V(j) in Vc, written
    // an iteration earlier; K(j+2) goes to Kc, whose K(j) the last iteration
    // consumed, and V(j+1) to Vn, whose V(j-1) likewise.
    auto iter = [&](int j, f32x16 (&cur)[NKB], f32x16 (&nxt)[NKB], KBuf &Kc, const KBuf &Kn,
                    const VBuf &Vc, VBuf &Vn) {
        __syncthreads();   // K(j+1), V(j) visible; K(j) and V(j-1) buffers free
        if (j + 2 < kcnt) sk.load(Kh, (kbeg + j + 2) * kKeys, Lk, tg);
        if (j + 1 < kcnt) sv.load(Vh, (kbeg + j + 1) * kKeys, Lk, tg);
        if (j + 1 < kcnt) scores(Kn, nxt);
        if (KS == 1 || j < kcnt) softmax_pv(kbeg + j, cur, Vc);
        if (j + 2 < kcnt) sk.store(Kc, tg);
        if (j + 1 < kcnt) sv.store(Vn, tg);
    };
    for (int j = 0; j < nloop; j += 2) {
        iter(j, sa, sb, bf.K0, bf.K1, bf.V0, bf.V1);
        if (j + 1 < nloop) iter(j + 1, sb, sa, bf.K1, bf.K0, bf.V1, bf.V0);
    }

    // Offset of the probabilities in base-2 units; -inf for a row that saw
    // no allowed key (its sum and O are zero).
    float m2f = (m_run == -INFINITY) ? -INFINITY : (POS_SCALE ? m_run * scale_log2 : m_run);
    if constexpr (KS == 2) {
        float *xs = reinterpret_cast<float *>(smem) + wq * NX * 64 + lane;
        __syncthreads();   // every wave is done with its tiles; smem is free
        if (g == 1) {
            xs[0] = m2f;
            xs[64] = l_run;
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
                for (int v = 0; v < 16; ++v) xs[(2 + 16 * cb + v) * 64] = oacc[cb][v];
        }
        __syncthreads();
        if (g == 1) return;   // no barrier follows
        const float mb = xs[0];
        const float mm = fmaxf(m2f, mb);
        const float fa = (mm == -INFINITY) ? 0.f : exp2_fast(m2f - mm);
        const float fb = (mm == -INFINITY) ? 0.f : exp2_fast(mb - mm);
        l_run = l_run * fa + xs[64] * fb;
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
            for (int v = 0; v < 16; ++v)
                oacc[cb][v] = oacc[cb][v] * fa + xs[(2 + 16 * cb + v) * 64] * fb;
        m2f = mm;
    }

    const float l = sum_xor32(l_run);
    if (qi < Lq) {
        const float inv = (l > 0.f) ? 1.f / l : 0.f;
        float *orow = O + qoff + (size_t)qi * D;
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
            for (int a = 0; a < 4; ++a)
                *reinterpret_cast<f32x4 *>(orow + 32 * cb + 8 * a + 4 * h) =
                    f32x4{oacc[cb][4 * a], oacc[cb][4 * a + 1], oacc[cb][4 * a + 2],
                          oacc[cb][4 * a + 3]} * inv;
        if (h == 0) LSE[(size_t)head * Lq + qi] = (l > 0.f) ? (m2f + log2f(l)) * kLn2 : -INFINITY;
    }
}

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

}  // namespace

// Causal grids of at most this many query-tile workgroups take the key-split
// form (d <= 64).  The key-split kernel holds one workgroup per CU (eight
// waves, 86 KB of LDS at d = 64), so up to the CU count of MI355X it runs in
// one round, and there the longest query tile's chain of key tiles sets the
// forward's time: B2 H8 L1024 d64 took 20.9 instead of 27.2 us, B4 H8 L1024
// 22.5 instead of 27.9.  Grids that need a second round gained nothing or
// lost (B8 H8 L1024: 31.0 against 30.4 us; B32 H8 L256: 24.2 against 16.7).
#ifndef MG_ACCEL_SPLIT_UPTO
#define MG_ACCEL_SPLIT_UPTO 256
#endif

hipError_t launch_fwd_accel(const AttnProblem &p, const float *Q, const float *K,
                            const float *V, float *O, float *LSE, hipStream_t s) {
    const int BH = p.B * p.H;
    const int nqt = cdiv(p.Lq, kRows);
    const dim3 grid(nqt * BH);
    const float sl2 = p.scale * kLog2e;
    auto go = [&](auto kern, int ks) {
        const int nt = kThreads * ks;
        const int ly = causal_rank_layer((const void *)kern, nt, grid.x, BH, p.causal);
        kern<<<grid, dim3(nt), 0, s>>>(Q, K, V, O, LSE, p.key_len, p.H, p.Lq, p.Lk, p.causal,
                                       sl2, nqt, BH, ly);
    };
    const bool split = p.causal && (long)grid.x <= MG_ACCEL_SPLIT_UPTO;
#define MG_FWD_ACCEL_PIPE(DD)                                                         \
    (split ? (p.scale > 0.f ? go(attn_fwd_accel_pipe<DD, true, 2>, 2)                 \
                            : go(attn_fwd_accel_pipe<DD, false, 2>, 2))               \
           : (p.scale > 0.f ? go(attn_fwd_accel_pipe<DD, true, 1>, 1)                 \
                            : go(attn_fwd_accel_pipe<DD, false, 1>, 1)))
    switch (p.d) {
    case 32: MG_FWD_ACCEL_PIPE(32); break;
    case 64: MG_FWD_ACCEL_PIPE(64); break;
    case 128:
        p.scale > 0.f ? go(attn_fwd_accel<128, true>, 1) : go(attn_fwd_accel<128, false>, 1);
        break;
    default: return hipErrorInvalidValue;
    }
#undef MG_FWD_ACCEL_PIPE
    return hipGetLastError();
}

}  // namespace mg
