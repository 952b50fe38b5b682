// attn_bf16.hip -- fast_bf16 attention kernels for gfx950 (bf16 MFMA, f32
// accumulation).
//
// Same three-kernel structure as the strict-f32 path (tiled forward, fused
// dK+dV with the key tile stationary, separate dQ; the paper's attention
// archetype, Sec. 3.3 and Sec. 8).  The reduced-input contract of Sec. 4.2
// rounds matrix inputs locally and accumulates in f32; here Q, K, V, O, dO
// and the gradients are stored bf16, and the softmax probabilities P and dS
// are rounded to bf16 (nearest even) only as inputs of the second product of
// each pass.  Softmax statistics, LSE and D stay f32.  D_i = rowsum(dO o O)
// needs no launch of its own: the dQ kernel, which holds each row's dO in
// registers, computes it on the way, writes it to the workspace, and runs
// before the dK/dV kernel that reads it.
//
// Contraction order: for products over the head dimension a lane holds 8
// consecutive d values (one 16-byte LDS read); for products over streamed
// rows it holds the rows of the accumulator registers it already owns, so
// P and dS become the B operand without leaving registers, and the LDS
// operand (a column of the row-major tile) comes from transpose reads.
//   16x16x32 (dK/dV): rows 32t + 16*(e/4) + 4g + e%4, g = lane/16
//   32x32x16 (forward, dQ): rows 16t + 8*(e/4) + 4h + e%4, h = lane/32
#include <type_traits>

#include "device_common.h"
#include "launch.h"
#include "tiles_bf16.h"
#include "tiles_direct.h"

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
// 32x32x16 products: each wave owns 32 queries (lane column l%32), so every
// 16-byte K fragment and 2x8-byte V^T fragment read from LDS feeds a
// 32-query product (half the LDS bytes per flop of 16-query waves).  The
// softmax keeps the VALU work per score low, because at bf16 matrix rates
// the vector unit, not the matrix core, is the tighter resource:
//   - the row max is taken on raw scores (POS_SCALE: scale > 0 keeps the
//     order) and each probability is one fma + one exp2;
//   - only tiles that straddle the causal diagonal or the key length are
//     masked (a workgroup-uniform branch);
//   - the output is rescaled only when some row's max moved.
constexpr int kFwdRows = 128;   // queries per workgroup (4 waves x 32)

template <int D, bool POS_SCALE>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 8)))
void attn_fwd_bf16(const uint16_t *__restrict__ Q, const uint16_t *__restrict__ K,
                   const uint16_t *__restrict__ V, uint16_t *__restrict__ O,
                   float *__restrict__ LSE, const int32_t *__restrict__ key_len, int H, int Lq, int Lk,
                   int causal, float scale_log2, int n_qtiles, int BH, int layer) {
    constexpr int NS = D / 16;    // 16-deep contraction steps over d
    constexpr int NCB = D / 32;   // 32-column blocks of d
    constexpr int NKB = kStream / 32;
    // K: 16-byte reads of 32 rows x 2 chunks (32-column blocks, swizzle
    // (r/4) % 4); V: transpose reads only, which 64-column blocks (swizzle
    // 4((r/2) % 2)) serve as well, loaded in 128-byte pieces.
    using Tile = Bf16Tile<kStream, D, kWaves, 32, 2, 3, 1>;
    constexpr int VW = (D >= 64) ? 64 : 32;
    using TileV = std::conditional_t<VW == 64, Bf16Tile<kStream, D, kWaves, 64, 1, 1, 4>, Tile>;
    constexpr int NL = Tile::kPerWave;   // loads per wave per tile (the vmcnt waits below)
    static_assert(TileV::kPerWave == NL, "K and V loads per wave");
    constexpr int BLK = Tile::kBlock, BLKV = TileV::kBlock;
    __shared__ __attribute__((aligned(16))) uint16_t Kr[Tile::kSize];
    __shared__ __attribute__((aligned(16))) uint16_t Vr[TileV::kSize];

    const int slot = blockIdx.x / BH;
    const int head = blockIdx.x - slot * BH;
    const int rank = serpentine_rank(slot, n_qtiles, layer);
    const int qt = causal ? (n_qtiles - 1 - rank) : rank;
    const int b = head / H;
    const size_t qoff = (size_t)head * Lq * D, hoff = (size_t)head * Lk * D;
    const int diag = Lk - Lq;   // causal: row i sees keys j <= i + diag

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c = lane & 31;
    const int h = lane >> 5;
    const int jr = (lane & 15) >> 2, jc = 4 * (lane & 3);   // transpose-read block offsets
    const int q0 = qt * kFwdRows;
    const int qi = q0 + 32 * w + c;

    const int klen = key_limit(key_len, b, Lk);
    const int kend = causal ? min(klen, q0 + kFwdRows + diag) : klen;
    const int ntiles = (kend + kStream - 1) / kStream;

    // K and V tiles: 16-byte direct-to-LDS loads; the next K tile is fetched
    // during P V, the next V tile during the next S = K Q^T.
    Tile tile;
    tile.init(lane);
    TileV tilev;
    tilev.init(lane);
    if (ntiles > 0) {
        tile.issue(Kr, K + hoff, 0, Lk, w);
        tilev.issue(Vr, V + hoff, 0, Lk, w);
    }
    // Lane bases of the tile reads.  K: row 32kb + c, chunk 2(s%2) + h of
    // block s/2 (kc[s%2]); V^T: rows 32kb + 16t + 4h + jr (+8) of column
    // 32cb + 16(c/16) + jc (vlo, vhi; one pair per 32 columns of a block).
    const int kc[2] = {Tile::at(c, 8 * h), Tile::at(c, 16 + 8 * h)};
    constexpr int NV = VW / 32;
    int vlo[NV], vhi[NV];
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        vlo[i] = TileV::at(4 * h + jr, 32 * i + 16 * (c >> 4) + jc);
        vhi[i] = TileV::at(4 * h + jr + 8, 32 * i + 16 * (c >> 4) + jc);
    }

    // B operand of S^T = K Q^T: lane holds Q[qi][16s + 8h + e].
    bf16x8 qreg[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s)
        qreg[s] = (qi < Lq) ? load_bf16x8(Q + qoff + (size_t)qi * D + 16 * s + 8 * h)
                           : __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});

    // Running max in raw-score units when POS_SCALE, else in base-2 units.
    float m_run = -INFINITY, l_run = 0.f;
    f32x16 oacc[NCB];   // O^T[32cb + 8a + 4h + r][qi] in register 4a + r
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) oacc[cb] = zero16();

    wait_vmcnt<NL>();   // K(0) landed (V(0) may still be in flight)
    __syncthreads();
    for (int kt = 0; kt < ntiles; ++kt) {

        // S^T[32kb + 8a + 4h + r][qi] in sacc[kb] register 4a + r
        f32x16 sacc[NKB];
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
            sacc[kb] = zero16();
#pragma unroll
            for (int s = 0; s < NS; ++s)
                sacc[kb] = mfma32x32x16bf16(
                    load_bf16x8(Kr + kc[s & 1] + (s >> 1) * BLK + 32 * 32 * kb), qreg[s],
                    sacc[kb]);
        }
        wait_vmcnt<0>();   // V(kt) landed
        __syncthreads();   // every wave is done with K(kt) and sees V(kt)
        if (kt + 1 < ntiles) tile.issue(Kr, K + hoff, (kt + 1) * kStream, Lk, w);
        if (!POS_SCALE) {
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) sacc[kb] *= scale_log2;
        }

        // Masking only where the tile crosses the diagonal or the key length.
        const bool full = (kt + 1) * kStream <= klen &&
                          (!causal || (kt + 1) * kStream - 1 <= q0 + diag);
        if (!full) {
            const int j0 = kt * kStream + 4 * h;
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
                const bf16x8 pb = pack_bf16_half(sacc[kb], t);
                const int r0 = VW * (32 * kb + 16 * t);
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb) {
                    const int o = (cb / NV) * BLKV + r0;
                    oacc[cb] = mfma32x32x16bf16(
                        load_tr_pair_at(Vr + vlo[cb % NV] + o, Vr + vhi[cb % NV] + o), pb,
                        oacc[cb]);
                }
            }

        wait_vmcnt<0>();   // K(kt+1) landed
        __syncthreads();   // every wave is done with V(kt) and sees K(kt+1)
        if (kt + 1 < ntiles) tilev.issue(Vr, V + hoff, (kt + 1) * kStream, Lk, w);
    }

    const float l = sum_xor32(l_run);
    if (qi < Lq) {
        const float inv = (l > 0.f) ? 1.f / l : 0.f;
        uint16_t *orow = O + qoff + (size_t)qi * D;
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
            for (int a = 0; a < 4; ++a)
                store_bf16x4(orow + 32 * cb + 8 * a + 4 * h,
                             f32x4{oacc[cb][4 * a], oacc[cb][4 * a + 1], oacc[cb][4 * a + 2],
                                   oacc[cb][4 * a + 3]} * inv);
        if (h == 0) {
            const float m2 = POS_SCALE ? m_run * scale_log2 : m_run;
            LSE[(size_t)head * Lq + qi] = (l > 0.f) ? (m2 + log2f(l)) * kLn2 : -INFINITY;
        }
    }
}

// The forward with its key tiles software-pipelined, for d <= 64: the score
// product of key tile kt+1 is issued in the same iteration as the softmax
// and P V of tile kt, so the matrix core has independent work while a wave
// runs its softmax; K and V are both double-buffered (separate named arrays,
// as in the backward kernels) and every load has a whole iteration to land.
// At d = 128 the second score block pushes the kernel to two waves per SIMD
// instead of three, and the plain form above is faster.
template <int D, bool POS_SCALE>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 8)))
void attn_fwd_bf16_pipe(const uint16_t *__restrict__ Q, const uint16_t *__restrict__ K,
                        const uint16_t *__restrict__ V, uint16_t *__restrict__ O,
                        float *__restrict__ LSE, const int32_t *__restrict__ key_len, int H, int Lq,
                        int Lk, int causal, float scale_log2, int n_qtiles, int BH, int layer) {
    constexpr int NS = D / 16;
    constexpr int NCB = D / 32;
    constexpr int NKB = kStream / 32;
    using Tile = Bf16Tile<kStream, D, kWaves, 32, 2, 3, 1>;
    constexpr int VW = (D >= 64) ? 64 : 32;
    using TileV = std::conditional_t<VW == 64, Bf16Tile<kStream, D, kWaves, 64, 1, 1, 4>, Tile>;
    constexpr int BLK = Tile::kBlock, BLKV = TileV::kBlock;
    __shared__ __attribute__((aligned(16))) uint16_t K0[Tile::kSize], K1[Tile::kSize];
    __shared__ __attribute__((aligned(16))) uint16_t V0[TileV::kSize], V1[TileV::kSize];

    const int slot = blockIdx.x / BH;
    const int head = blockIdx.x - slot * BH;
    const int rank = serpentine_rank(slot, n_qtiles, layer);
    const int qt = causal ? (n_qtiles - 1 - rank) : rank;
    const int b = head / H;
    const size_t qoff = (size_t)head * Lq * D, hoff = (size_t)head * Lk * D;
    const int diag = Lk - Lq;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c = lane & 31;
    const int h = lane >> 5;
    const int jr = (lane & 15) >> 2, jc = 4 * (lane & 3);
    const int q0 = qt * kFwdRows;
    const int qi = q0 + 32 * w + c;
    const int klen = key_limit(key_len, b, Lk);
    const int kend = causal ? min(klen, q0 + kFwdRows + diag) : klen;
    const int ntiles = (kend + kStream - 1) / kStream;

    Tile tile;
    tile.init(lane);
    TileV tilev;
    tilev.init(lane);
    const int kc[2] = {Tile::at(c, 8 * h), Tile::at(c, 16 + 8 * h)};
    constexpr int NV = VW / 32;
    int vlo[NV], vhi[NV];
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        vlo[i] = TileV::at(4 * h + jr, 32 * i + 16 * (c >> 4) + jc);
        vhi[i] = TileV::at(4 * h + jr + 8, 32 * i + 16 * (c >> 4) + jc);
    }
    bf16x8 qreg[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s)
        qreg[s] = (qi < Lq) ? load_bf16x8(Q + qoff + (size_t)qi * D + 16 * s + 8 * h)
                           : __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
    float m_run = -INFINITY, l_run = 0.f;
    f32x16 oacc[NCB];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) oacc[cb] = zero16();

    auto scores = [&](const uint16_t *Kb, f32x16 (&sacc)[NKB]) {
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
            sacc[kb] = zero16();
#pragma unroll
            for (int s = 0; s < NS; ++s)
                sacc[kb] = mfma32x32x16bf16(
                    load_bf16x8(Kb + kc[s & 1] + (s >> 1) * BLK + 32 * 32 * kb), qreg[s], sacc[kb]);
        }
    };
    auto softmax_pv = [&](int kt, f32x16 (&sacc)[NKB], const uint16_t *Vb) {
        if (!POS_SCALE) {
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) sacc[kb] *= scale_log2;
        }
        const bool full = (kt + 1) * kStream <= klen &&
                          (!causal || (kt + 1) * kStream - 1 <= q0 + diag);
        if (!full) {
            const int j0 = kt * kStream + 4 * h;
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
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                const bf16x8 pb = pack_bf16_half(sacc[kb], t);
                const int r0 = VW * (32 * kb + 16 * t);
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb) {
                    const int o = (cb / NV) * BLKV + r0;
                    oacc[cb] = mfma32x32x16bf16(
                        load_tr_pair_at(Vb + vlo[cb % NV] + o, Vb + vhi[cb % NV] + o), pb,
                        oacc[cb]);
                }
            }
    };

    // Prologue: K(0), V(0), K(1) in flight together; S(0).  Tile j lives in
    // buffer j % 2 (K0/K1, V0/V1).
    f32x16 sa[NKB], sb[NKB];
    if (ntiles > 0) {
        tile.issue(K0, K + hoff, 0, Lk, w);
        tilev.issue(V0, V + hoff, 0, Lk, w);
        if (ntiles > 1) tile.issue(K1, K + hoff, kStream, Lk, w);
        wait_vmcnt<0>();
        __syncthreads();
        scores(K0, sa);
    }
    // Iteration kt: S(kt) is in `cur`; K(kt+1) arrives in Kn and V(kt) in Vc
    // (both issued an iteration earlier); K(kt+2) goes to Kc, whose K(kt) the
    // last iteration consumed, and V(kt+1) to Vn, whose V(kt-1) likewise.
    auto iter = [&](int kt, f32x16 (&cur)[NKB], f32x16 (&nxt)[NKB], uint16_t *Kc, uint16_t *Kn,
                    uint16_t *Vc, uint16_t *Vn) {
        wait_vmcnt<0>();
        __syncthreads();   // K(kt+1), V(kt) visible; K(kt) and V(kt-1) buffers free
        if (kt + 2 < ntiles) tile.issue(Kc, K + hoff, (kt + 2) * kStream, Lk, w);
        if (kt + 1 < ntiles) tilev.issue(Vn, V + hoff, (kt + 1) * kStream, Lk, w);
        if (kt + 1 < ntiles) scores(Kn, nxt);
        softmax_pv(kt, cur, Vc);
    };
    for (int kt = 0; kt < ntiles; kt += 2) {
        iter(kt, sa, sb, K0, K1, V0, V1);
        if (kt + 1 < ntiles) iter(kt + 1, sb, sa, K1, K0, V1, V0);
    }

    const float l = sum_xor32(l_run);
    if (qi < Lq) {
        const float inv = (l > 0.f) ? 1.f / l : 0.f;
        uint16_t *orow = O + qoff + (size_t)qi * D;
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
            for (int a = 0; a < 4; ++a)
                store_bf16x4(orow + 32 * cb + 8 * a + 4 * h,
                             f32x4{oacc[cb][4 * a], oacc[cb][4 * a + 1], oacc[cb][4 * a + 2],
                                   oacc[cb][4 * a + 3]} * inv);
        if (h == 0) {
            const float m2 = POS_SCALE ? m_run * scale_log2 : m_run;
            LSE[(size_t)head * Lq + qi] = (l > 0.f) ? (m2 + log2f(l)) * kLn2 : -INFINITY;
        }
    }
}

// ------------------------------------------------------- backward: dK, dV
// Key tile of 64 keys stationary (16 per wave, one per lane column) on
// 16x16x32 products; query tiles of 64 rows stream through LDS row-major.
// Masks as in the strict-f32 kernel: a causal threshold per lane, padded
// keys overwritten with zeros at the end, rows past Lq inert.
//
// The two tile buffers are separate LDS arrays and the tile loop is unrolled
// by two, so that every read names the buffer it reads at compile time: the
// compiler can then tell the next tile's direct-to-LDS loads apart from the
// current tile's operand reads and does not wait for the loads before the
// reads (with one array indexed by a run-time buffer number it must assume
// they may overlap, and the prefetch would stall every iteration).
template <int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 8)))
void attn_dkdv_bf16(const uint16_t *__restrict__ Q, const uint16_t *__restrict__ K,
                    const uint16_t *__restrict__ V, const uint16_t *__restrict__ dO,
                    const float *__restrict__ LSE, const float *__restrict__ Dws,
                    uint16_t *__restrict__ dK, uint16_t *__restrict__ dV,
                    const int32_t *__restrict__ key_len, int H, int Lq, int Lk, int causal, float scale,
                    float scale_log2, int BH, int layer) {
    constexpr int NS = D / 32;
    constexpr int NC = D / 16;
    constexpr int QR = kStream;      // query rows per streamed tile
    constexpr int QB = QR / 16;      // 16-row blocks per tile
    // Q and dO tiles are double-buffered and arrive by 16-byte direct-to-LDS
    // loads: the next tile is fetched during the whole current iteration,
    // and one barrier per iteration suffices.
    constexpr int TW = 32;   // column block width of the tiles
    using Tile = Bf16Tile<QR, D, kWaves, TW, 1, 3, 1>;
    constexpr int BLK = Tile::kBlock;
    __shared__ __attribute__((aligned(16))) uint16_t Qr0[Tile::kSize], Qr1[Tile::kSize];
    __shared__ __attribute__((aligned(16))) uint16_t Or0[Tile::kSize], Or1[Tile::kSize];
    __shared__ __attribute__((aligned(16))) float lse0[QR], lse1[QR];   // LSE * log2e
    __shared__ __attribute__((aligned(16))) float Ds0[QR], Ds1[QR];     // -D

    const int slot = blockIdx.x / BH;
    const int head = blockIdx.x - slot * BH;
    const int kt = serpentine_rank(slot, (Lk + kStatRows - 1) / kStatRows, layer);
    const int b = head / H;
    const size_t qoff = (size_t)head * Lq * D, hoff = (size_t)head * Lk * D;
    const int diag = Lk - Lq;   // causal: row i sees keys j <= i + diag

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int il = lane & 15;
    const int g = lane >> 4;
    const int jr = il >> 2, jc = 4 * (il & 3);   // transpose-read block offsets
    const int k0 = kt * kStatRows;
    const int kj = k0 + 16 * w + il;

    const int klen = key_limit(key_len, b, Lk);
    const int nq = (Lq + QR - 1) / QR;
    // first query tile holding a row that sees key k0
    const int qstart = causal ? min(nq, max(0, k0 - diag) / QR) : 0;
    const int qstop = (k0 < klen) ? nq : qstart;

    bf16x8 kreg[NS], vreg[NS];
    load_stationary<D>(kreg, K + hoff, kj, Lk, g);
    load_stationary<D>(vreg, V + hoff, kj, Lk, g);

    f32x4 dkacc[NC], dvacc[NC];   // dK^T[16c + 4g + r][kj], dV^T likewise
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        dkacc[c] = zero4();
        dvacc[c] = zero4();
    }

    Tile tile;
    tile.init(lane);
    // Lane bases of the tile reads (TW-column blocks).  Q, dO rows: row
    // 16ib + il, columns 32s + 8g (qa[s % (TW/32)], block 32s/TW); Q^T, dO^T:
    // rows 32t + 4g + jr (+16) of columns 16c + jc (qb[c % (TW/16)], block
    // 16c/TW).
    constexpr int NA = TW / 32, NB = TW / 16;
    int qa[NA], qb[NB];
#pragma unroll
    for (int i = 0; i < NA; ++i) qa[i] = Tile::at(il, 32 * i + 8 * g);
#pragma unroll
    for (int i = 0; i < NB; ++i) qb[i] = Tile::at(4 * g + jr, 16 * i + jc);
    // Direct-to-LDS loads of the Q and dO rows of tile qt and of their LSE
    // (natural log; wave 0) and D (the last wave) into staging rows; rows
    // past Lq arrive as zeros.  Once the loads have landed, `publish` (the
    // same lanes) stores LSE * log2e and -D for the tile, so that each score
    // needs one fma before its exp2 and dP accumulates straight onto -D.
    using Buf = uint16_t[Tile::kSize];
    static_assert(QR == 64, "one statistic per lane");
    __shared__ __attribute__((aligned(16))) float raw[2][QR];   // LSE, D in flight
    auto fetch = [&](int qt, Buf &Qn, Buf &On) {
        tile.issue(Qn, Q + qoff, qt * QR, Lq, w);
        tile.issue(On, dO + qoff, qt * QR, Lq, w);
        if (w == 0 || w == kWaves - 1) {
            const int row0 = qt * QR;
            const int rows = min(max(Lq - row0, 0), QR);
            const float *src = (w == 0 ? LSE : Dws) + (size_t)head * Lq + row0;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                buffer_rsrc(src, rows * 4),
                (__attribute__((address_space(3))) void *)&raw[w == 0 ? 0 : 1][0], 4, lane * 4, 0,
                0, 0);
        }
    };
    auto publish = [&](float (&ln)[QR], float (&dn)[QR]) {
        if (w == 0) ln[lane] = raw[0][lane] * kLog2e;
        if (w == kWaves - 1) dn[lane] = -raw[1][lane];
    };

    // One query tile from buffers (Qc, Oc, lc, dc) while tile qt + 1 loads
    // into (Qn, On, ln, dn).
    auto step = [&](int qt, Buf &Qc, Buf &Oc, float (&lc)[QR], float (&dc)[QR], Buf &Qn,
                    Buf &On, float (&ln)[QR], float (&dn)[QR]) {
        if (qt + 1 < qstop) fetch(qt + 1, Qn, On);   // freed by the last barrier

        // S = Q K^T; dP - D = dO V^T accumulated onto -D (rows 16ib + 4g + r)
        f32x4 sacc[QB], pacc[QB];
#pragma unroll
        for (int ib = 0; ib < QB; ++ib) {
            sacc[ib] = zero4();
            pacc[ib] = *reinterpret_cast<const f32x4 *>(&dc[16 * ib + 4 * g]);
        }
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
            for (int ib = 0; ib < QB; ++ib) {
                const int o = qa[s % NA] + (s / NA) * BLK + 16 * TW * ib;
                sacc[ib] = mfma16x16x32bf16(load_bf16x8(Qc + o), kreg[s], sacc[ib]);
                pacc[ib] = mfma16x16x32bf16(load_bf16x8(Oc + o), vreg[s], pacc[ib]);
            }

        // 2*NS*QB operand reads and as many products: eight reads ahead
        // (d = 128: 279-282 -> 268-273 us at B2 H16 L4096; at d = 64 and 32,
        // where a wave has half or a quarter of the reads, 1-3 % slower)
        if constexpr (D == 128) sched_reads_ahead<2 * NS * QB, 2 * NS * QB, 8, 2, 2, 0>();

        // P = exp2(S * scale*log2e - LSE*log2e), dS = P (dP - D); the mask (row
        // qt*QR + 16ib + 4g + r sees key kj iff 16ib + r >= thr) only in tiles
        // that cross the wave's causal boundary.
        auto softmax = [&](auto masked) {
            const int thr = kj - diag - (qt * QR + 4 * g);
#pragma unroll
            for (int ib = 0; ib < QB; ++ib) {
                const f32x4 l2 = *reinterpret_cast<const f32x4 *>(&lc[16 * ib + 4 * g]);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    float p = exp2_fast(fmaf(sacc[ib][r], scale_log2, -l2[r]));
                    if (masked && 16 * ib + r < thr) p = 0.f;
                    sacc[ib][r] = p;
                    pacc[ib][r] *= p;
                }
            }
        };
        if (!causal || qt * QR + diag >= k0 + 16 * w + 15)
            softmax(std::false_type{});
        else
            softmax(std::true_type{});

        // dV^T[16c + .][kj] += dO^T[16c + il'][i] P[i][kj]; dK^T likewise with Q, dS
#pragma unroll
        for (int t = 0; t < QB / 2; ++t) {
            const bf16x8 pb = pack_bf16(sacc[2 * t], sacc[2 * t + 1]);
            const bf16x8 sb = pack_bf16(pacc[2 * t], pacc[2 * t + 1]);
            const int r0 = 32 * TW * t;
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                const int o = qb[c % NB] + (c / NB) * BLK + r0;
                dvacc[c] = mfma16x16x32bf16(load_tr_pair_at(Oc + o, Oc + o + 16 * TW), pb,
                                            dvacc[c]);
                dkacc[c] = mfma16x16x32bf16(load_tr_pair_at(Qc + o, Qc + o + 16 * TW), sb,
                                            dkacc[c]);
            }
        }

        // 2*QB*NC transpose reads for QB*NC products, eight ahead (d = 128)
        if constexpr (D == 128) sched_reads_ahead<2 * QB * NC, QB * NC, 8, 2, 1, 1>();

        if (qt + 1 < qstop) {
            wait_vmcnt<0>();   // next tile and its LSE, D landed
            publish(ln, dn);
        }
        __syncthreads();   // next tile visible; buffers (Qc, Oc) free
    };

    if (qstart < qstop) {
        fetch(qstart, Qr0, Or0);
        wait_vmcnt<0>();
        publish(lse0, Ds0);
    }
    __syncthreads();
    for (int qt = qstart; qt < qstop; qt += 2) {
        step(qt, Qr0, Or0, lse0, Ds0, Qr1, Or1, lse1, Ds1);
        if (qt + 1 < qstop) step(qt + 1, Qr1, Or1, lse1, Ds1, Qr0, Or0, lse0, Ds0);
    }

    if (kj < Lk) {
        const bool keep = kj < klen;   // padded keys get exact zeros
        uint16_t *dkrow = dK + hoff + (size_t)kj * D;
        uint16_t *dvrow = dV + hoff + (size_t)kj * D;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            store_bf16x4(dkrow + 16 * c + 4 * g, keep ? dkacc[c] * scale : zero4());
            store_bf16x4(dvrow + 16 * c + 4 * g, keep ? dvacc[c] : zero4());
        }
    }
}

// ------------------------------------------------------------ backward: dQ
// Query-stationary, 32 queries per wave on 32x32x16 products (as the forward):
// S^T = K Q^T and dP^T = V dO^T from row-major K and V tiles, then
// dQ^T += K^T dS^T with dS^T straight from registers and K^T from transpose
// reads of the row-major K tile.  KS keys per streamed tile; K and V tiles
// are double-buffered in LDS and arrive by direct-to-LDS row loads, so the
// next tile is fetched during the whole current iteration.  As in the dK/dV
// kernel, the two buffers are separate arrays and the tile loop is unrolled
// by two, so that the current tile's reads need not wait for the next
// tile's loads.
template <int D, int KS>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 8)))
void attn_dq_bf16(const uint16_t *__restrict__ Q, const uint16_t *__restrict__ K,
                  const uint16_t *__restrict__ V, const uint16_t *__restrict__ O,
                  const uint16_t *__restrict__ dO, const float *__restrict__ LSE,
                  float *__restrict__ Dws, uint16_t *__restrict__ dQ,
                  const int32_t *__restrict__ key_len, int H, int Lq, int Lk,
                  int causal, float scale, float scale_log2, int n_qtiles, int BH, int layer) {
    constexpr int NS = D / 16;
    constexpr int NCB = D / 32;
    constexpr int NKB = KS / 32;
    // K and V tiles are double-buffered and arrive by 16-byte direct-to-LDS
    // loads: the next tile is fetched during the whole current iteration.
    using Tile = Bf16Tile<KS, D, kWaves, 32, 2, 3, 1>;
    constexpr int BLK = Tile::kBlock;
    __shared__ __attribute__((aligned(16))) uint16_t Kr0[Tile::kSize], Kr1[Tile::kSize];
    __shared__ __attribute__((aligned(16))) uint16_t Vr0[Tile::kSize], Vr1[Tile::kSize];

    const int slot = blockIdx.x / BH;
    const int head = blockIdx.x - slot * BH;
    const int rank = serpentine_rank(slot, n_qtiles, layer);
    const int qt = causal ? (n_qtiles - 1 - rank) : rank;
    const int b = head / H;
    const size_t qoff = (size_t)head * Lq * D, hoff = (size_t)head * Lk * D;
    const int diag = Lk - Lq;   // causal: row i sees keys j <= i + diag

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c = lane & 31;
    const int h = lane >> 5;
    const int jr = (lane & 15) >> 2, jc = 4 * (lane & 3);
    const int q0 = qt * kFwdRows;
    const int qi = q0 + 32 * w + c;

    const int klen = key_limit(key_len, b, Lk);
    const int kend = causal ? min(klen, q0 + kFwdRows + diag) : klen;
    const int ntiles = (kend + KS - 1) / KS;

    bf16x8 qreg[NS], oreg[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        const size_t off = qoff + (size_t)qi * D + 16 * s + 8 * h;
        qreg[s] = (qi < Lq) ? load_bf16x8(Q + off) : __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
        oreg[s] = (qi < Lq) ? load_bf16x8(dO + off) : __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
    }
    // Rows past Lq: Q = dO = 0 and LSE = D = 0, so their dS is exactly 0.
    const float lse2 = (qi < Lq) ? LSE[(size_t)head * Lq + qi] * kLog2e : 0.f;
    // D_i = sum_d dO[i][d] O[i][d], in f32 from the bf16 values: this lane
    // holds the d values of oreg, its partner (lane ^ 32) the other half of
    // the row.  The row's D goes to the workspace for the dK/dV kernel,
    // which runs after this one.
    float Di = 0.f;
    if (qi < Lq) {
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            const bf16x8 o8 = load_bf16x8(O + qoff + (size_t)qi * D + 16 * s + 8 * h);
#pragma unroll
            for (int e = 0; e < 8; ++e) Di = fmaf((float)o8[e], (float)oreg[s][e], Di);
        }
    }
    Di += xor_lanes(Di, 32);
    if (qi < Lq && h == 0) Dws[(size_t)head * Lq + qi] = Di;

    f32x16 dqacc[NCB];   // dQ^T[32cb + 8a + 4h + r][qi]
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) dqacc[cb] = zero16();

    Tile tile;
    tile.init(lane);
    // Lane bases of the tile reads.  K, V rows: row 32kb + c, chunk
    // 2(s%2) + h of block s/2 (kc[s%2]); K^T: rows 32kb + 16t + 4h + jr (+8)
    // of column 32cb + 16(c/16) + jc (klo, khi).
    const int kc[2] = {Tile::at(c, 8 * h), Tile::at(c, 16 + 8 * h)};
    const int klo = Tile::at(4 * h + jr, 16 * (c >> 4) + jc);
    const int khi = Tile::at(4 * h + jr + 8, 16 * (c >> 4) + jc);
    using Buf = uint16_t[Tile::kSize];
    auto fetch = [&](int t, Buf &Kn, Buf &Vn) {
        tile.issue(Kn, K + hoff, t * KS, Lk, w);
        tile.issue(Vn, V + hoff, t * KS, Lk, w);
    };
    // key tile kt from (Kc, Vc) while tile kt + 1 loads into (Kn, Vn)
    auto step = [&](int kt, Buf &Kc, Buf &Vc, Buf &Kn, Buf &Vn) {
        if (kt + 1 < ntiles) fetch(kt + 1, Kn, Vn);   // freed by the last barrier
        const bool full = (kt + 1) * KS <= klen &&
                          (!causal || (kt + 1) * KS - 1 <= q0 + diag);
        const int j0 = kt * KS + 4 * h;
        const int thr = causal ? min(klen - j0, qi + diag - j0 + 1) : klen - j0;

#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
            // S^T = K Q^T; dP^T - D = V dO^T accumulated onto -D
            f32x16 sacc = zero16(), pacc;
#pragma unroll
            for (int v = 0; v < 16; ++v) pacc[v] = -Di;
#pragma unroll
            for (int s = 0; s < NS; ++s) {
                const int o = kc[s & 1] + (s >> 1) * BLK + 32 * 32 * kb;
                sacc = mfma32x32x16bf16(load_bf16x8(Kc + o), qreg[s], sacc);
                pacc = mfma32x32x16bf16(load_bf16x8(Vc + o), oreg[s], pacc);
            }
            // eight operand reads ahead of the products (d = 128: dQ 205-207 -> 203 us)
            if constexpr (D == 128) sched_reads_ahead<2 * NS, 2 * NS, 8, 2, 2, 2>();
            // dS^T = P^T (dP^T - D), P^T = exp2(S^T * scale*log2e - LSE*log2e);
            // the mask only in tiles that cross the diagonal or the key length
            auto softmax = [&](auto masked) {
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    float p = exp2_fast(fmaf(sacc[v], scale_log2, -lse2));
                    if (masked && 32 * kb + 8 * (v >> 2) + (v & 3) >= thr) p = 0.f;
                    pacc[v] *= p;
                }
            };
            if (full)
                softmax(std::false_type{});
            else
                softmax(std::true_type{});
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                const bf16x8 sb = pack_bf16_half(pacc, t);
                const int r0 = 32 * (32 * kb + 16 * t);
#pragma unroll
                for (int cb2 = 0; cb2 < NCB; ++cb2)
                    dqacc[cb2] = mfma32x32x16bf16(
                        load_tr_pair_at(Kc + klo + cb2 * BLK + r0, Kc + khi + cb2 * BLK + r0),
                        sb, dqacc[cb2]);
            }
            if constexpr (D == 128) sched_reads_ahead<4 * NCB, 2 * NCB, 8, 2, 1, 3>();
        }
        wait_vmcnt<0>();   // next K/V tile landed
        __syncthreads();   // it is visible; buffers (Kc, Vc) are free
    };
    if (ntiles > 0) fetch(0, Kr0, Vr0);
    wait_vmcnt<0>();
    __syncthreads();
    for (int kt = 0; kt < ntiles; kt += 2) {
        step(kt, Kr0, Vr0, Kr1, Vr1);
        if (kt + 1 < ntiles) step(kt + 1, Kr1, Vr1, Kr0, Vr0);
    }

    if (qi < Lq) {
        uint16_t *dqrow = dQ + qoff + (size_t)qi * D;
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
            for (int a = 0; a < 4; ++a)
                store_bf16x4(dqrow + 32 * cb + 8 * a + 4 * h,
                             f32x4{dqacc[cb][4 * a], dqacc[cb][4 * a + 1], dqacc[cb][4 * a + 2],
                                   dqacc[cb][4 * a + 3]} * scale);
    }
}

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

}  // namespace

// ---------------------------------------------------------------- launchers
hipError_t launch_fwd_bf16(const AttnProblem &p, const uint16_t *Q, const uint16_t *K,
                           const uint16_t *V, uint16_t *O, float *LSE, hipStream_t s) {
    const int BH = p.B * p.H;
    const int nqt = cdiv(p.Lq, kFwdRows);
    const dim3 grid(nqt * BH), block(kThreads);
    const float sl2 = p.scale * kLog2e;
    auto go = [&](auto kern) {
        const int ly = causal_rank_layer((const void *)kern, kThreads, grid.x, BH, p.causal);
        kern<<<grid, block, 0, s>>>(Q, K, V, O, LSE, p.key_len, p.H, p.Lq, p.Lk, p.causal, sl2,
                                    nqt, BH, ly);
    };
#define MG_FWD_BF16(KERN, DD) \
    (p.scale > 0.f ? go(KERN<DD, true>) : go(KERN<DD, false>))
    switch (p.d) {
    case 32: MG_FWD_BF16(attn_fwd_bf16_pipe, 32); break;
    case 64: MG_FWD_BF16(attn_fwd_bf16_pipe, 64); break;
    case 128: MG_FWD_BF16(attn_fwd_bf16, 128); break;
    default: return hipErrorInvalidValue;
    }
#undef MG_FWD_BF16
    return hipGetLastError();
}

hipError_t launch_bwd_dkdv_bf16(const AttnProblem &p, const uint16_t *Q, const uint16_t *K,
                                const uint16_t *V, const uint16_t *dO, const float *LSE,
                                const float *Dws, uint16_t *dK, uint16_t *dV, hipStream_t s) {
    const int BH = p.B * p.H;
    const float sl2 = p.scale * kLog2e;
    const dim3 grid(cdiv(p.Lk, kStatRows) * BH), block(kThreads);
    auto go = [&](auto kern) {
        const int ly = causal_rank_layer((const void *)kern, kThreads, grid.x, BH, p.causal);
        kern<<<grid, block, 0, s>>>(Q, K, V, dO, LSE, Dws, dK, dV, p.key_len, p.H, p.Lq, p.Lk,
                                    p.causal, p.scale, sl2, BH, ly);
    };
    switch (p.d) {
    case 32: go(attn_dkdv_bf16<32>); break;
    case 64: go(attn_dkdv_bf16<64>); break;
    case 128: go(attn_dkdv_bf16<128>); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_bwd_dq_bf16(const AttnProblem &p, const uint16_t *Q, const uint16_t *K,
                              const uint16_t *V, const uint16_t *O, const uint16_t *dO,
                              const float *LSE, float *Dws, uint16_t *dQ, hipStream_t s) {
    const int BH = p.B * p.H;
    const int nqt = cdiv(p.Lq, kFwdRows);
    const dim3 grid(nqt * BH), block(kThreads);
    const float sl2 = p.scale * kLog2e;
    auto go = [&](auto kern) {
        const int ly = causal_rank_layer((const void *)kern, kThreads, grid.x, BH, p.causal);
        kern<<<grid, block, 0, s>>>(Q, K, V, O, dO, LSE, Dws, dQ, p.key_len, p.H, p.Lq, p.Lk,
                                    p.causal, p.scale, sl2, nqt, BH, ly);
    };
    switch (p.d) {
    case 32: go(attn_dq_bf16<32, 64>); break;
    case 64: go(attn_dq_bf16<64, 64>); break;
    case 128: go(attn_dq_bf16<128, 64>); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace mg
