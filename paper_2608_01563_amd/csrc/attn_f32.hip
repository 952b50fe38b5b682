// attn_f32.hip -- strict-f32 attention kernels for gfx950 (f32 MFMA).
//
// The paper's attention archetype is three kernels: a tiled forward, a dQ
// kernel and a fused dK+dV kernel (Sec. 3.3; Sec. 8 makes the fused dK+dV
// kernel a compiler invariant; Sec. 7.3 profiles the backward pair).  Here:
//
//   attn_fwd_f32      query tile stationary, streams K/V tiles, online
//                     softmax in base 2, writes O and LSE (natural log).
//   attn_fwd_f32_ks2  the same for grids too small to spread evenly over
//                     the CUs: 32-row query tiles, whose key tiles are split
//                     between two halves of the workgroup; the halves merge
//                     their (max, sum, O) states through LDS at the end.
//   attn_rowdot_f32   D_i = sum_k dO_ik O_ik (HBM-bound row reduction).
//   attn_dkdv_f32     key tile stationary: recomputes P from LSE, then
//                     dV += P^T dO, dP = dO V^T, dS = P(dP - D), dK += dS^T Q.
//   attn_dkdvq_f32    attn_dkdv_f32 plus the dQ product of its key tile:
//                     dQ_part = dS K_tile goes to the workspace, one partial
//                     per (key tile, query row) (d <= 64).
//   attn_dq_reduce_f32  dQ = scale * sum of a row's partials, in key-tile
//                     order (fixed order: bitwise-reproducible, no atomics).
//   attn_dq_f32       query tile stationary: recomputes P and dS, then
//                     dQ += dS K (used when the partials do not fit: d = 128
//                     or a workspace above 1 GiB).
//
// Every product runs on v_mfma_f32_16x16x4_f32 (f32 inputs, f32 accumulate),
// which is what the strict contract permits (Sec. 4.2).  Each wave owns 16
// rows of the stationary tile (one per lane column l%16); the other operand
// is staged through LDS, 64 rows at a time, and shared by the waves of a
// workgroup.  The forward kernel copies its K and V tiles with gfx950's
// direct-to-LDS buffer loads (no staging registers) and fetches the next K
// tile during P V and the next V tile during S = K Q^T.  The backward
// kernels stage Q and dO through registers: the loads for the next tile are
// issued before the current one is consumed and written to LDS after it.
//
// Workgroup order: the 1-D grid is numbered rank-major over heads
// (id = slot * B*H + head) with rank 0 the tile that has the most work under
// a causal mask.  When the grid is larger than what the chip holds at once,
// slot = rank, so the longest tiles start first and the dispatcher hands the
// short ones to whichever CU frees up; when every workgroup is resident at
// once, layers of slots alternate direction (serpentine_rank) so that each
// CU holds a mix of long and short tiles.  With B*H a multiple of 8 every
// tile of a head lands on the same XCD (workgroups are dealt to the eight
// XCDs round-robin), so a head's K/V or Q/dO stay in one L2.
//
// Masking: an element's offset inside its tile is compared against one
// per-lane threshold (key length, causal diagonal); the forward kernel skips
// the comparison on tiles that hold no masked element.
#include <algorithm>
#include <climits>
#include <type_traits>

#include "device_common.h"
#include "launch.h"
#include "tiles_direct.h"
#include "tiles_f32.h"

// Per-kernel launch configuration: waves per workgroup, minimum waves per
// SIMD requested from the register allocator (0 = compiler default), and
// double-buffered LDS for the streamed tile of the backward kernels (the
// forward kernel always alternates its K and V fetches).  The defaults are
// the fastest of sweeps on MI355X at B8 H8 L1024 d64 and B16 H12 L512 d64
// (double buffering lost there: it halves the workgroups an LDS-heavy CU can
// hold); they can be overridden at build time.
#ifndef MG_FWD_CFG
#define MG_FWD_CFG 4, 3, false
#endif
#ifndef MG_DKDV_CFG
#define MG_DKDV_CFG 4, 3, false
#endif
#ifndef MG_DKDVQ_CAUSAL_CFG
#define MG_DKDVQ_CAUSAL_CFG 8, 4, false   // 128-key tiles: half the dQ partials
#endif
#ifndef MG_DQ_CFG
#define MG_DQ_CFG 8, 0, false
#endif
#ifndef MG_DKDVQ_CAUSAL_NIB
#define MG_DKDVQ_CAUSAL_NIB 2   // 16-row query blocks per step, 128-key fused kernel
#endif
#ifndef MG_DKDV_NIB
#define MG_DKDV_NIB 2   // 16-row query blocks per dK/dV step (d <= 64)
#endif

namespace mg {
namespace {

constexpr int kStream = 64;   // streamed rows per step
#ifndef MG_FWD_SPLIT_CFG
#define MG_FWD_SPLIT_CFG 2, 3, false
#endif
#ifndef MG_FWD_SPLIT_KS
#define MG_FWD_SPLIT_KS 32
#endif
#ifndef MG_FWD_SPLIT_BELOW
#define MG_FWD_SPLIT_BELOW 512   // forward grids below this split their key tiles in two
#endif
#ifndef MG_FWD_KS
#define MG_FWD_KS 64
#endif
#ifndef MG_FWD_SPLIT4_UPTO
#define MG_FWD_SPLIT4_UPTO 256     // 32-row grids up to this size split their keys four ways...
#endif
#ifndef MG_FWD_SPLIT4_MIN_KEYS
#define MG_FWD_SPLIT4_MIN_KEYS 256 // ...when each group still gets two or more 32-key tiles
#endif
constexpr int kFwdStream = MG_FWD_KS;   // keys per streamed forward tile

template <int NW_, int OCC_, bool DB_>
struct Cfg {
    static constexpr int NW = NW_;             // waves per workgroup
    static constexpr int NT = 64 * NW_;        // threads per workgroup
    static constexpr int ROWS = 16 * NW_;      // stationary rows per workgroup
    static constexpr int OCC = OCC_ > 0 ? OCC_ : 1;
    // the occupancy request only holds without spills for d <= 64
    template <int D> static constexpr int occ() { return D <= 64 ? OCC : 1; }
    static constexpr int NBUF = DB_ ? 2 : 1;   // LDS buffers for the streamed tile
};
using FwdCfg = Cfg<MG_FWD_CFG>;
using FwdSplitCfg = Cfg<MG_FWD_SPLIT_CFG>;   // 32-row tiles, keys split in two
using DkdvCfg = Cfg<MG_DKDV_CFG>;
using DkdvqCausalCfg = Cfg<MG_DKDVQ_CAUSAL_CFG>;
using DqCfg = Cfg<MG_DQ_CFG>;

// ---------------------------------- work-first order for key-padded grids
// In a non-causal problem with key padding, the key tiles at or past a
// batch's key length have no query work (their workgroups only write zero
// dK/dV rows).  Numbered in plain slot-major order such idle workgroups sit
// between the working ones and leave CU slots empty while working tiles wait,
// which measured 20-40 % slower than the same number of working tiles
// dispatched back to back.  Here every XCD x takes the heads h = x (mod 8)
// (workgroups are dealt to the eight XCDs round-robin, so block 8k + x runs
// on XCD x and a head's tiles share one L2), and its k-th block takes the
// k-th working (slot, head) of those heads in slot-major order, then the
// idle ones.  Needs B*H a multiple of 8 and at most 64 heads per XCD; the
// launcher checks both.  All lanes return the same slot and head.
__device__ __forceinline__ int nth_set_bit(uint64_t mask, int n) {
    for (int t = 0; t < n; ++t) mask &= mask - 1;   // drop the n lowest set bits
    return __builtin_ctzll(mask);
}

__device__ __forceinline__ void work_first_tile(int id, int nslots, int nsplit, int key_rows,
                                                int BH, int H, int Lk,
                                                const int32_t *__restrict__ key_len, int &slot,
                                                int &head) {
    const int lane = threadIdx.x & 63;
    const int x = id & 7, k = id >> 3;
    const int G = BH >> 3;                // heads of this XCD's group
    const bool valid = lane < G;
    const int klen = valid ? key_limit(key_len, (x + 8 * lane) / H, Lk) : 0;
    int before = 0;
    for (int pass = 0; pass < 2; ++pass) {   // working tiles, then idle ones
        for (int s = 0; s < nslots; ++s) {
            const bool works = (s / nsplit) * key_rows < klen;
            const uint64_t m = __ballot(valid && works == (pass == 0));
            const int c = __popcll(m);
            if (k < before + c) {
                slot = s;
                head = x + 8 * nth_set_bit(m, k - before);
                return;
            }
            before += c;
        }
    }
    slot = 0;   // not reached: the grid holds exactly nslots * B*H blocks
    head = x;
}

// The forward's version: every query tile of a non-causal key-padded head
// costs ceil(key length / key_rows) key tiles, so the k-th block of XCD x
// takes its heads' (slot, head) pairs by decreasing cost (head by head within
// one cost), and the short ones fill in at the end (a longest-first list
// schedule per XCD).  Same requirements as work_first_tile.
__device__ __forceinline__ void heavy_first_tile(int id, int nslots, int key_rows, int BH, int H,
                                                 int Lk, const int32_t *__restrict__ key_len,
                                                 int &slot, int &head) {
    const int lane = threadIdx.x & 63;
    const int x = id & 7, k = id >> 3;
    const int G = BH >> 3;
    const bool valid = lane < G;
    const int klen = valid ? key_limit(key_len, (x + 8 * lane) / H, Lk) : 0;
    const int cost = (klen + key_rows - 1) / key_rows;
    int before = 0;
    for (int v = (Lk + key_rows - 1) / key_rows; v >= 0; --v) {
        const uint64_t m = __ballot(valid && cost == v);
        const int c = __popcll(m) * nslots;
        if (k < before + c) {
            const int j = k - before;
            head = x + 8 * nth_set_bit(m, j / nslots);
            slot = j % nslots;
            return;
        }
        before += c;
    }
    slot = 0;   // not reached
    head = x;
}

// ---------------------------------------------------------------- forward --
// Query tile of C::ROWS rows stationary (16 per wave); K and V tiles of KS
// keys (64; 32 in the key-split form, one pair per half) stream through LDS
// by direct-to-LDS loads.  The next K tile is fetched
// while the softmax and P V of the current tile run, the next V tile while
// the next S = K Q^T runs, so each iteration has two barriers and no staging
// registers:
//   S(kt) from K | wait V(kt), barrier | fetch K(kt+1) | softmax, P V(kt)
//   | wait K(kt+1), barrier | fetch V(kt+1)
template <int D, class C, int KSPLIT>
__device__ __forceinline__ void fwd_f32_body(const float *__restrict__ Q, const float *__restrict__ K,
                  const float *__restrict__ V, float *__restrict__ O, float *__restrict__ LSE,
                  const int32_t *__restrict__ key_len, int H, int Lq, int Lk, int causal,
                  float scale_log2, int n_qtiles, int BH, int layer, int work_first) {
    // keys per streamed tile (the split form streams shorter tiles, so that
    // four of its workgroups fit in one CU's LDS)
    constexpr int KS = (KSPLIT > 1) ? MG_FWD_SPLIT_KS : kFwdStream;
    constexpr int DQ = D / 4;    // contraction values per lane in one S chain
    constexpr int NC = D / 16;   // 16-column blocks of the head dimension
    constexpr int NJB = KS / 16; // 16-key blocks per streamed tile
    using Tile = DirectTile<KS, D, C::NW>;
    static_assert(Tile::kEven, "the vmcnt waits below count kPerWave loads per fetch");
    constexpr int NL = Tile::kPerWave;   // vector-memory operations per tile fetch
    static_assert(KSPLIT == 1 || ((KSPLIT == 2 || KSPLIT == 4) && C::NW * NC * 256 <= KS * D),
                  "a key group's O must fit in its K tile");
    __shared__ __attribute__((aligned(16))) float Ks[KSPLIT][KS * D];
    __shared__ __attribute__((aligned(16))) float Vs[KSPLIT][KS * D];
    // key split: m, l of groups 1 .. KSPLIT-1
    __shared__ float xml[KSPLIT > 1 ? (KSPLIT - 1) * 2 * C::NW * 64 : 1];

    int slot, head;
    if (work_first) {
        heavy_first_tile(blockIdx.x, n_qtiles, KS, BH, H, Lk, key_len, slot, head);
    } else {
        slot = blockIdx.x / BH;
        head = blockIdx.x - slot * BH;
    }
    const int rank = serpentine_rank(slot, n_qtiles, layer);
    const int qt = causal ? (n_qtiles - 1 - rank) : rank;
    const int b = head / H;
    const float *Qh = Q + (size_t)head * Lq * D;
    const float *Kh = K + (size_t)head * Lk * D;
    const float *Vh = V + (size_t)head * Lk * D;
    const int diag = Lk - Lq;   // causal: row i sees keys j <= i + diag

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wg = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int hh = (KSPLIT > 1) ? wg / C::NW : 0;   // key group of this wave
    const int w = (KSPLIT > 1) ? wg - hh * C::NW : wg;   // row wave within its half
    const int il = lane & 15;
    const int g = lane >> 4;
    const int q0 = qt * C::ROWS;
    const int qw0 = q0 + 16 * w;   // first query row of this wave
    const int qi = qw0 + il;

    const int klen = key_limit(key_len, b, Lk);
    const int kend = causal ? min(klen, q0 + C::ROWS + diag) : klen;
    const int ntiles = (kend + KS - 1) / KS;
    // Key split: group h takes key tiles [h*m, min(n, (h+1)*m)) with
    // m = ceil(n/KSPLIT); every group runs m iterations so that every barrier
    // is reached by all waves (a group's surplus iterations only wait).
    const int iters = (KSPLIT > 1) ? (ntiles + KSPLIT - 1) / KSPLIT : ntiles;
    const int tbeg = hh * iters;
    const int tend = (KSPLIT > 1) ? min(ntiles, tbeg + iters) : ntiles;
    float *const Ksh = Ks[hh];
    float *const Vsh = Vs[hh];

    Tile tile;
    tile.init(w, lane);
    // LDS float offsets of this lane's operands in key block jb = 0; block jb
    // adds 16*jb*D (the chunk permutation repeats every 16 rows).
    int koff[DQ / 4], voffs[4][NC];
#pragma unroll
    for (int s4 = 0; s4 < DQ / 4; ++s4) koff[s4] = Tile::at(il, g * DQ + 4 * s4);
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < NC; ++c) voffs[r][c] = Tile::at(4 * g + r, 16 * c + il);
    if (tbeg < tend) {
        tile.issue(Ksh, Kh, tbeg * KS, Lk, w);
        tile.issue(Vsh, Vh, tbeg * KS, Lk, w);
    }

    // B operand of S^T = K Q^T: lane holds Q[qi][g*DQ + s] times
    // scale*log2(e), so that the product is the exponent in base 2.
    float qreg[DQ];
#pragma unroll
    for (int s4 = 0; s4 < DQ / 4; ++s4) {
        f32x4 v = (qi < Lq) ? *reinterpret_cast<const f32x4 *>(Qh + (size_t)qi * D + g * DQ + 4 * s4)
                           : zero4();
#pragma unroll
        for (int e = 0; e < 4; ++e) qreg[4 * s4 + e] = v[e] * scale_log2;
    }

    float m_run = -INFINITY;   // running max of this lane's row, base-2 units
    float l_run = 0.f;         // this lane's share of the row sum
    f32x4 oacc[NC];            // O^T[16c + 4g + r][qi]
#pragma unroll
    for (int c = 0; c < NC; ++c) oacc[c] = zero4();

    wait_vmcnt<NL>();   // K(0) landed (V(0) may still be in flight)
    __syncthreads();
    for (int it = 0; it < iters; ++it) {
        const int kt = tbeg + it;
        const bool act = (KSPLIT == 1) || kt < tend;   // uniform over the half
        // 16-key blocks of this tile that hold an allowed key for some row
        // of this wave (a prefix: keys past the key length, or past the
        // wave's last row under a causal mask, are masked for every row).
        // The products of the other blocks are skipped; their scores are
        // masked below and their probabilities are exactly zero.
        const int jt = kt * KS;
        const int kcut = causal ? min(klen, qw0 + 16 + diag) : klen;
        const int nlive = act ? min(NJB, (kcut - jt + 15) / 16) : 0;

        // S^T[16jb + 4g + r][qi] = sum_k K[j][k] Q[qi][k]
        f32x4 sacc[NJB];
#pragma unroll
        for (int jb = 0; jb < NJB; ++jb) sacc[jb] = zero4();
        if (nlive == NJB) {
#pragma unroll
            for (int s4 = 0; s4 < DQ / 4; ++s4) {
                f32x4 a[NJB];
#pragma unroll
                for (int jb = 0; jb < NJB; ++jb)
                    a[jb] = *reinterpret_cast<const f32x4 *>(&Ksh[koff[s4] + 16 * jb * D]);
#pragma unroll
                for (int e = 0; e < 4; ++e)
#pragma unroll
                    for (int jb = 0; jb < NJB; ++jb)
                        sacc[jb] = mfma16x16x4(a[jb][e], qreg[4 * s4 + e], sacc[jb]);
            }
        } else {
#pragma unroll
            for (int jb = 0; jb < NJB; ++jb) {
                if (jb >= nlive) break;
#pragma unroll
                for (int s4 = 0; s4 < DQ / 4; ++s4) {
                    const f32x4 a =
                        *reinterpret_cast<const f32x4 *>(&Ksh[koff[s4] + 16 * jb * D]);
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        sacc[jb] = mfma16x16x4(a[e], qreg[4 * s4 + e], sacc[jb]);
                }
            }
        }
        wait_vmcnt<0>();   // V(kt) landed
        __syncthreads();   // every wave is done with K(kt) and sees V(kt)
        if (kt + 1 < tend) tile.issue(Ksh, Kh, (kt + 1) * KS, Lk, w);

        if (act) {
            // Element (jb, r) holds key j0 + 16jb + r, allowed iff that offset is
            // below a per-lane threshold (key length; the query row if causal).
            // Only tiles that reach past the key length or past the wave's first
            // query row (causal) hold masked elements.
            if (jt + KS > klen || (causal && jt + KS - 1 > qw0 + diag)) {
                const int j0 = jt + 4 * g;
                const int thr = causal ? min(klen - j0, qi + diag - j0 + 1) : klen - j0;
    #pragma unroll
                for (int jb = 0; jb < NJB; ++jb)
    #pragma unroll
                    for (int r = 0; r < 4; ++r)
                        sacc[jb][r] = (16 * jb + r < thr) ? sacc[jb][r] : -INFINITY;
            }
            float mx = -INFINITY;
    #pragma unroll
            for (int jb = 0; jb < NJB; ++jb)
    #pragma unroll
                for (int r = 0; r < 4; ++r) mx = fmaxf(mx, sacc[jb][r]);
            mx = max_over_groups(mx);
            const float m_new = fmaxf(m_run, mx);
            const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
            // Rescaling by 2^(m_run - m_new) is a multiplication by one on every
            // lane whose maximum did not move; skip it when that holds wave-wide.
            if (__any(m_new != m_run)) {
                const float alpha = exp2_fast(m_run - m_use);
                l_run *= alpha;
    #pragma unroll
                for (int c = 0; c < NC; ++c) oacc[c] *= alpha;
            }
            m_run = m_new;
            float psum = 0.f;
    #pragma unroll
            for (int jb = 0; jb < NJB; ++jb)
    #pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const float p = exp2_fast(sacc[jb][r] - m_use);
                    sacc[jb][r] = p;
                    psum += p;
                }
            l_run += psum;

            // O^T[16c + 4g + r][qi] += sum_j V[j][16c + il'] P^T[j][qi]
    #pragma unroll
            for (int jb = 0; jb < NJB; ++jb) {
                if (jb >= nlive) break;
    #pragma unroll
                for (int r = 0; r < 4; ++r)
    #pragma unroll
                    for (int c = 0; c < NC; ++c)
                        oacc[c] = mfma16x16x4(Vsh[voffs[r][c] + 16 * jb * D], sacc[jb][r], oacc[c]);
            }
        }

        wait_vmcnt<0>();   // K(kt+1) landed
        __syncthreads();   // every wave is done with V(kt) and sees K(kt+1)
        if (kt + 1 < tend) tile.issue(Vsh, Vh, (kt + 1) * KS, Lk, w);
    }

    float l = sum_over_groups(l_run);
    if constexpr (KSPLIT > 1) {
        // Groups 1 .. KSPLIT-1 hand their (m, l, O) to group 0 through their
        // own K tiles, which no wave reads any more; group 0 merges the
        // online-softmax states in group order.
        if (hh > 0) {
            float *xo = Ks[hh];
            float *xm = xml + (hh - 1) * 2 * C::NW * 64, *xl = xm + C::NW * 64;
#pragma unroll
            for (int c = 0; c < NC; ++c)
                *reinterpret_cast<f32x4 *>(&xo[((w * NC + c) * 64 + lane) * 4]) = oacc[c];
            xm[w * 64 + lane] = m_run;
            xl[w * 64 + lane] = l;
        }
        __syncthreads();
        if (hh > 0) return;
        float mm = m_run;
#pragma unroll
        for (int h = 1; h < KSPLIT; ++h) mm = fmaxf(mm, xml[(h - 1) * 2 * C::NW * 64 + w * 64 + lane]);
        const float mu = (mm == -INFINITY) ? 0.f : mm;
        const float a0 = exp2_fast(m_run - mu);
        l *= a0;
#pragma unroll
        for (int c = 0; c < NC; ++c) oacc[c] *= a0;
#pragma unroll
        for (int h = 1; h < KSPLIT; ++h) {
            const float *xo = Ks[h];
            const float *xm = xml + (h - 1) * 2 * C::NW * 64, *xl = xm + C::NW * 64;
            const float ah = exp2_fast(xm[w * 64 + lane] - mu);
#pragma unroll
            for (int c = 0; c < NC; ++c)
                oacc[c] += *reinterpret_cast<const f32x4 *>(&xo[((w * NC + c) * 64 + lane) * 4]) * ah;
            l += xl[w * 64 + lane] * ah;
        }
        m_run = mm;
    }
    if (qi < Lq) {
        const float inv = (l > 0.f) ? 1.f / l : 0.f;
        float *orow = O + ((size_t)head * Lq + qi) * D;
#pragma unroll
        for (int c = 0; c < NC; ++c)
            *reinterpret_cast<f32x4 *>(orow + 16 * c + 4 * g) = oacc[c] * inv;
        if (g == 0)
            LSE[(size_t)head * Lq + qi] = (l > 0.f) ? (m_run + log2f(l)) * kLn2 : -INFINITY;
    }
}

// The kernels: one workgroup per (query tile, head); the _ks2 form splits
// the key tiles over two halves of the workgroup (grids too small to fill
// the chip).  Two named kernels over one device body: as one kernel template
// with the split as a third parameter, hipcc (ROCm 7.2) emitted the host
// launch stub of only one of the two instances per head size, and the
// library failed to link.
#define MG_FWD_F32_ARGS                                                                    \
    const float *__restrict__ Q, const float *__restrict__ K, const float *__restrict__ V, \
        float *__restrict__ O, float *__restrict__ LSE, const int32_t *__restrict__ key_len, \
        int H, int Lq, int Lk, int causal, float scale_log2, int n_qtiles, int BH, int layer, \
        int work_first
template <int D, class C>
__global__ __launch_bounds__(C::NT) __attribute__((amdgpu_waves_per_eu(C::template occ<D>(), 8)))
void attn_fwd_f32(MG_FWD_F32_ARGS) {
    fwd_f32_body<D, C, 1>(Q, K, V, O, LSE, key_len, H, Lq, Lk, causal, scale_log2, n_qtiles, BH,
                          layer, work_first);
}
template <int D, class C>
__global__ __launch_bounds__(2 * C::NT) __attribute__((amdgpu_waves_per_eu(C::template occ<D>(), 8)))
void attn_fwd_f32_ks2(MG_FWD_F32_ARGS) {
    fwd_f32_body<D, C, 2>(Q, K, V, O, LSE, key_len, H, Lq, Lk, causal, scale_log2, n_qtiles, BH,
                          layer, work_first);
}
template <int D, class C>
__global__ __launch_bounds__(4 * C::NT) __attribute__((amdgpu_waves_per_eu(C::template occ<D>(), 8)))
void attn_fwd_f32_ks4(MG_FWD_F32_ARGS) {
    fwd_f32_body<D, C, 4>(Q, K, V, O, LSE, key_len, H, Lq, Lk, causal, scale_log2, n_qtiles, BH,
                          layer, work_first);
}
#undef MG_FWD_F32_ARGS

// ------------------------------------------------- backward: D = rowsum(dO o O)
template <int D>
__global__ __launch_bounds__(256) void attn_rowdot_f32(const float *__restrict__ O,
                                                       const float *__restrict__ dO,
                                                       float *__restrict__ Dws, int rows) {
    constexpr int TPR = D / 4;   // threads per row, one 16-byte chunk each
    const int row = blockIdx.x * (256 / TPR) + threadIdx.x / TPR;
    const int c4 = threadIdx.x % TPR;
    float v = 0.f;
    if (row < rows) {
        const f32x4 o = *reinterpret_cast<const f32x4 *>(O + (size_t)row * D + 4 * c4);
        const f32x4 go = *reinterpret_cast<const f32x4 *>(dO + (size_t)row * D + 4 * c4);
        v = o[0] * go[0] + o[1] * go[1] + o[2] * go[2] + o[3] * go[3];
    }
#pragma unroll
    for (int m = TPR / 2; m >= 1; m >>= 1) v += xor_lanes(v, m);
    if (row < rows && c4 == 0) Dws[row] = v;
}

// ------------------------------------------------------- backward: dK, dV
// Key tile of C::ROWS keys stationary (16 per wave, one per lane column);
// query tiles of NIB*16 rows stream through LDS.
template <int D, int NIB, class C>
__global__ __launch_bounds__(C::NT) __attribute__((amdgpu_waves_per_eu(C::template occ<D>(), 8)))
void attn_dkdv_f32(const float *__restrict__ Q, const float *__restrict__ K,
                   const float *__restrict__ V, const float *__restrict__ dO,
                   const float *__restrict__ LSE, const float *__restrict__ Dws,
                   float *__restrict__ dK, float *__restrict__ dV,
                   const int32_t *__restrict__ key_len, int H, int Lq, int Lk, int causal, float scale,
                   float scale_log2, int BH, int layer) {
    constexpr int DQ = D / 4;
    constexpr int NC = D / 16;
    constexpr int BR = 16 * NIB;
    using Stager = F32TileStager<BR, D, C::NT>;
    constexpr int LD = Stager::kLd;
    __shared__ __attribute__((aligned(16))) float Qs[C::NBUF][BR][LD];
    __shared__ __attribute__((aligned(16))) float dOs[C::NBUF][BR][LD];
    __shared__ __attribute__((aligned(16))) float lse2s[C::NBUF][BR];
    __shared__ __attribute__((aligned(16))) float Ds[C::NBUF][BR];

    const int slot = blockIdx.x / BH;
    const int head = blockIdx.x - slot * BH;
    // low key tiles see the most queries under a causal mask
    const int kt = serpentine_rank(slot, (Lk + C::ROWS - 1) / C::ROWS, layer);
    const int b = head / H;
    const size_t qoff = (size_t)head * Lq * D, hoff = (size_t)head * Lk * D;
    const float *Qh = Q + qoff;
    const float *dOh = dO + qoff;
    const int diag = Lk - Lq;   // causal: row i sees keys j <= i + diag

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int il = lane & 15;
    const int g = lane >> 4;
    const int k0 = kt * C::ROWS;
    const int kj = k0 + 16 * (tid >> 6) + il;   // this lane's key

    const int klen = key_limit(key_len, b, Lk);
    const int nq = (Lq + BR - 1) / BR;
    // first query tile holding a row that sees key k0
    const int qstart = causal ? min(nq, max(0, k0 - diag) / BR) : 0;
    const int qstop = (k0 < klen) ? nq : qstart;   // a fully padded key tile does no work

    // B operands of S = Q K^T and dP = dO V^T: lane holds K[kj][g*DQ + s].
    float kreg[DQ], vreg[DQ];
#pragma unroll
    for (int s4 = 0; s4 < DQ / 4; ++s4) {
        const size_t off = hoff + (size_t)kj * D + g * DQ + 4 * s4;
        const f32x4 kv = (kj < Lk) ? *reinterpret_cast<const f32x4 *>(K + off) : zero4();
        const f32x4 vv = (kj < Lk) ? *reinterpret_cast<const f32x4 *>(V + off) : zero4();
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            kreg[4 * s4 + e] = kv[e];
            vreg[4 * s4 + e] = vv[e];
        }
    }

    f32x4 dkacc[NC], dvacc[NC];   // dK^T[16c + 4g + r][kj], dV^T likewise
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        dkacc[c] = zero4();
        dvacc[c] = zero4();
    }

    Stager qst, ost;
    float lse_pre = 0.f, d_pre = 0.f;
    auto load_rows = [&](int qt) {
        qst.load(Qh, qt * BR, Lq, tid);
        ost.load(dOh, qt * BR, Lq, tid);
        if (tid < BR) {
            const int row = qt * BR + tid;
            // natural log; scaled to base 2 at the LDS store so that nothing waits
            // for this load before the next tile's rows are consumed
            lse_pre = (row < Lq) ? LSE[(size_t)head * Lq + row] : 0.f;
            d_pre = (row < Lq) ? Dws[(size_t)head * Lq + row] : 0.f;
        }
    };
    auto store_rows = [&](int buf) {
        qst.store(Qs[buf], tid);
        ost.store(dOs[buf], tid);
        if (tid < BR) {
            lse2s[buf][tid] = lse_pre * kLog2e;
            Ds[buf][tid] = d_pre;
        }
    };
    if (qstart < qstop) {
        load_rows(qstart);
        if (C::NBUF == 2) {
            store_rows(0);
            __syncthreads();
        }
    }

    for (int qt = qstart; qt < qstop; ++qt) {
        const int cur = (C::NBUF == 2) ? ((qt - qstart) & 1) : 0;
        if (C::NBUF == 1) {
            __syncthreads();
            store_rows(0);
            __syncthreads();
        }
        if (qt + 1 < qstop) load_rows(qt + 1);

        // S[16ib + 4g + r][kj] and dP[..][kj]
        f32x4 sacc[NIB], pacc[NIB];
#pragma unroll
        for (int ib = 0; ib < NIB; ++ib) {
            sacc[ib] = zero4();
            pacc[ib] = zero4();
        }
#pragma unroll
        for (int s4 = 0; s4 < DQ / 4; ++s4) {
            f32x4 aq[NIB], ao[NIB];
#pragma unroll
            for (int ib = 0; ib < NIB; ++ib) {
                aq[ib] = *reinterpret_cast<const f32x4 *>(&Qs[cur][16 * ib + il][g * DQ + 4 * s4]);
                ao[ib] = *reinterpret_cast<const f32x4 *>(&dOs[cur][16 * ib + il][g * DQ + 4 * s4]);
            }
#pragma unroll
            for (int e = 0; e < 4; ++e)
#pragma unroll
                for (int ib = 0; ib < NIB; ++ib) {
                    sacc[ib] = mfma16x16x4(aq[ib][e], kreg[4 * s4 + e], sacc[ib]);
                    pacc[ib] = mfma16x16x4(ao[ib][e], vreg[4 * s4 + e], pacc[ib]);
                }
        }

        // P = exp(S - LSE), dS = P (dP - D).  Under a causal mask element
        // (ib, r) is query ibase + 16ib + r, allowed iff it is >= kj - diag.  Padded
        // keys (kj >= key length) are not masked here: their rows of dK and dV
        // are overwritten with zeros at the end.  Rows past Lq hold Q = dO = 0
        // and LSE = D = 0, so they contribute exactly nothing.
        const int ibase = qt * BR + 4 * g;
        const int thr = causal ? kj - diag - ibase : INT_MIN;
#pragma unroll
        for (int ib = 0; ib < NIB; ++ib) {
            const f32x4 l2 = *reinterpret_cast<const f32x4 *>(&lse2s[cur][16 * ib + 4 * g]);
            const f32x4 dd = *reinterpret_cast<const f32x4 *>(&Ds[cur][16 * ib + 4 * g]);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                float p = exp2_fast(sacc[ib][r] * scale_log2 - l2[r]);
                p = (16 * ib + r >= thr) ? p : 0.f;
                sacc[ib][r] = p;
                pacc[ib][r] = p * (pacc[ib][r] - dd[r]);
            }
        }

        // dV^T[16c + 4g + r][kj] += sum_i dO[i][16c + il'] P[i][kj]
        // dK^T[16c + 4g + r][kj] += sum_i  Q[i][16c + il'] dS[i][kj]
#pragma unroll
        for (int ib = 0; ib < NIB; ++ib)
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int c = 0; c < NC; ++c) {
                    dvacc[c] = mfma16x16x4(dOs[cur][16 * ib + 4 * g + r][16 * c + il],
                                           sacc[ib][r], dvacc[c]);
                    dkacc[c] = mfma16x16x4(Qs[cur][16 * ib + 4 * g + r][16 * c + il],
                                           pacc[ib][r], dkacc[c]);
                }

        if (C::NBUF == 2) {
            if (qt + 1 < qstop) store_rows(cur ^ 1);
            __syncthreads();
        }
    }

    if (kj < Lk) {
        const bool keep = kj < klen;   // padded keys get exact zeros
        float *dkrow = dK + hoff + (size_t)kj * D;
        float *dvrow = dV + hoff + (size_t)kj * D;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            *reinterpret_cast<f32x4 *>(dkrow + 16 * c + 4 * g) = keep ? dkacc[c] * scale : zero4();
            *reinterpret_cast<f32x4 *>(dvrow + 16 * c + 4 * g) = keep ? dvacc[c] : zero4();
        }
    }
}

// ---------------------------------------- backward: dK, dV and dQ partials
// The key-stationary kernel above, extended with the dQ product: after dS of
// a query tile is known, it goes through LDS and the workgroup multiplies it
// by its own key tile, dQ_part[i][:] = sum_{j in tile} dS[i][j] K[j][:].
// Each (key tile, query row) partial is written once to the workspace and
// attn_dq_reduce_f32 adds the partials of a row in key-tile order: no atomics,
// bitwise-reproducible, and no second recompute of S and dP.
//
// The Q and dO tiles, and the LSE and D values of their rows, reach LDS by
// row-wise direct-to-LDS loads (no staging registers, padded rows as in the
// kernel above); dQ partials leave through raw buffer stores whose
// descriptor ends at row Lq.  With two LDS buffers (C::NBUF == 2) the next tile is fetched
// during the whole current iteration; with one, during the dQ product.  A
// tile's dQ partials are stored at the start of the next iteration, so the
// wait for the next tile never waits on a just-issued store.
//
// Small grids (LOCALD): the O rows of each query tile arrive with its Q and
// dO rows, and the workgroup computes D_i = sum_k dO_ik O_ik in LDS before
// the softmax needs it, so no separate D launch precedes the kernel.  With a
// single key tile and no query split (direct_dq), the one partial of a row is
// its dQ: it is scaled and written to dQ (dQp points there), rows outside the
// tile's query range get zeros, and no reduction follows (LOCALD grids only,
// so that the large-grid instances carry none of this).
template <int D, int NIB, class C, bool LOCALD>
__global__ __launch_bounds__(C::NT) __attribute__((amdgpu_waves_per_eu(C::template occ<D>(), 8)))
void attn_dkdvq_f32(const float *__restrict__ Q, const float *__restrict__ K,
                    const float *__restrict__ V, const float *__restrict__ O,
                    const float *__restrict__ dO, const float *__restrict__ LSE,
                    const float *__restrict__ Dws, float *__restrict__ dK,
                    float *__restrict__ dV, float *__restrict__ dQp, float *__restrict__ dKVp,
                    const int32_t *__restrict__ key_len, int H, int Lq, int Lk, int causal,
                    float scale, float scale_log2, int BH, int nsplit, int nranks, int layer,
                    int work_first, int direct_dq) {
    constexpr int DQ = D / 4;
    constexpr int NC = D / 16;
    constexpr int BR = 16 * NIB;
    constexpr int KR = C::ROWS;                 // keys per workgroup
    constexpr int NBLK = NIB * NC;              // 16x16 blocks of a dQ partial tile
    constexpr int PER_WAVE = (NBLK + C::NW - 1) / C::NW;
    constexpr int NB = C::NBUF;
    constexpr int LD = D + 4;
    using Tile = RowDirectTile<BR, D, C::NW, LD>;
    __shared__ __attribute__((aligned(16))) float Qs[NB][BR][LD];
    __shared__ __attribute__((aligned(16))) float dOs[NB][BR][LD];
    __shared__ __attribute__((aligned(16))) float lse2s[NB][BR];    // LSE (natural log)
    __shared__ __attribute__((aligned(16))) float Ds[NB][BR];
    __shared__ __attribute__((aligned(16))) float Os[LOCALD ? NB : 1][LOCALD ? BR : 1][LD];
    __shared__ __attribute__((aligned(16))) float Kt[D][KR + 4];    // key tile, transposed
    __shared__ __attribute__((aligned(16))) float dSs[BR][KR + 4];  // dS of the query tile

    int slot, head;
    if (work_first) {
        work_first_tile(blockIdx.x, nranks, nsplit, C::ROWS, BH, H, Lk, key_len, slot, head);
    } else {
        slot = blockIdx.x / BH;
        head = blockIdx.x - slot * BH;
    }
    const int rank = serpentine_rank(slot, nranks, layer);
    const int kt = rank / nsplit;          // key tile
    const int split = rank - kt * nsplit;  // share of its query tiles
    const int b = head / H;
    const size_t qoff = (size_t)head * Lq * D, hoff = (size_t)head * Lk * D;
    const float *Qh = Q + qoff;
    const float *dOh = dO + qoff;
    const int diag = Lk - Lq;   // causal: row i sees keys j <= i + diag

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int il = lane & 15;
    const int g = lane >> 4;
    const int k0 = kt * KR;
    const int wkey0 = k0 + 16 * w;   // first key of this wave (wave-uniform)
    const int kj = wkey0 + il;

    const int klen = key_limit(key_len, b, Lk);
    const int nq = (Lq + BR - 1) / BR;
    // first query tile holding a row that sees key k0, and the end of the
    // range; split `split` of `nsplit` takes a contiguous share of it
    const int qfirst = causal ? min(nq, max(0, k0 - diag) / BR) : 0;
    const int qlast = (k0 < klen) ? nq : qfirst;
    const int qstart = qfirst + (int)((long)(qlast - qfirst) * split / nsplit);
    const int qstop = qfirst + (int)((long)(qlast - qfirst) * (split + 1) / nsplit);

    const Tile tile;

    // Direct-to-LDS loads of the Q and dO rows of query tile qt, and of their
    // LSE (wave 0) and D (the last wave) values, or with LOCALD of their O
    // rows instead of D; rows past Lq arrive as zeros.
    auto fetch = [&](int qt, int buf) {
        tile.issue(Qs[buf], Qh, qt * BR, Lq, w, lane);
        tile.issue(dOs[buf], dOh, qt * BR, Lq, w, lane);
        if constexpr (LOCALD) tile.issue(Os[buf], O + qoff, qt * BR, Lq, w, lane);
        if (w == 0 || (!LOCALD && w == C::NW - 1)) {
            const int row0 = qt * BR;
            const int rows = min(max(Lq - row0, 0), BR);
            const float *src = (w == 0 ? LSE : Dws) + (size_t)head * Lq + row0;
            const auto rsrc = buffer_rsrc(src, rows * 4);
            float *dst = (w == 0) ? lse2s[buf] : Ds[buf];
            if (lane < BR)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rsrc, (__attribute__((address_space(3))) void *)dst, 4, lane * 4, 0, 0, 0);
        }
    };
    if (qstart < qstop) fetch(qstart, 0);

    float kreg[DQ], vreg[DQ];
#pragma unroll
    for (int s4 = 0; s4 < DQ / 4; ++s4) {
        const size_t off = hoff + (size_t)kj * D + g * DQ + 4 * s4;
        const f32x4 kv = (kj < Lk) ? *reinterpret_cast<const f32x4 *>(K + off) : zero4();
        const f32x4 vv = (kj < Lk) ? *reinterpret_cast<const f32x4 *>(V + off) : zero4();
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            kreg[4 * s4 + e] = kv[e];
            vreg[4 * s4 + e] = vv[e];
        }
    }
    // The key tile, transposed, for the A operand of the dQ product.
    for (int f = tid; f < KR * (D / 4); f += C::NT) {
        const int row = f / (D / 4);
        const int c4 = f - row * (D / 4);
        const f32x4 v = (k0 + row < Lk)
            ? *reinterpret_cast<const f32x4 *>(K + hoff + (size_t)(k0 + row) * D + 4 * c4)
            : zero4();
#pragma unroll
        for (int e = 0; e < 4; ++e) Kt[4 * c4 + e][row] = v[e];
    }

    f32x4 dkacc[NC], dvacc[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        dkacc[c] = zero4();
        dvacc[c] = zero4();
    }

    // Under a causal mask element (ib, r) is query ibase + 16ib + r, allowed
    // iff it is >= kj - diag; a padded key (kj >= key length) is masked everywhere
    // so that it adds nothing to dQ.
    // (sentinels +-2^30 keep kthr - ibase free of overflow)
    constexpr int kNever = 1 << 30;
    const int kthr = (kj >= klen) ? kNever : (causal ? kj - diag : -kNever);

    // dQ partial blocks of this wave: consecutive blocks (same query rows,
    // shared dS reads) when they split evenly, else strided
    auto dq_block = [&](int bb) {
        return (NBLK % C::NW == 0) ? w * PER_WAVE + bb : w + bb * C::NW;
    };
    f32x4 dqacc[PER_WAVE];   // partials of the previous query tile, not yet stored
    // Raw buffer stores through a descriptor that covers the tile's rows below
    // Lq: stores of rows past Lq fall outside it and are dropped.
    float *dQp_head = dQp + ((size_t)kt * BH + head) * Lq * D;
    auto store_dq = [&](int qt) {
        const int row0 = qt * BR;
        const auto rsrc = buffer_rsrc(dQp_head + (size_t)row0 * D, min(Lq - row0, BR) * D * 4);
#pragma unroll
        for (int bb = 0; bb < PER_WAVE; ++bb) {
            const int blk = dq_block(bb);
            if (NBLK % C::NW != 0 && blk >= NBLK) break;
            const int ib = blk / NC;
            const int c = blk - ib * NC;
            __builtin_amdgcn_raw_buffer_store_b128(
                __builtin_bit_cast(u32x4, (LOCALD && direct_dq) ? dqacc[bb] * scale : dqacc[bb]),
                rsrc,
                ((16 * ib + il) * D + 16 * c + 4 * g) * 4, 0, 0);
        }
    };

    // D of the tile in buffer buf from its landed dO and O rows: TPR threads
    // per row, each summing every TPR-th 4-float chunk, then a butterfly.
    auto local_d = [&](int buf) {
        if constexpr (LOCALD) {
            constexpr int TPR = C::NT / BR;
            static_assert(C::NT % BR == 0 && (TPR & (TPR - 1)) == 0 && TPR <= 64,
                          "threads per row");
            const int row = tid / TPR, part = tid - (tid / TPR) * TPR;
            float acc = 0.f;
#pragma unroll
            for (int c4 = part; c4 < D / 4; c4 += TPR) {
                const f32x4 a = *reinterpret_cast<const f32x4 *>(&dOs[buf][row][4 * c4]);
                const f32x4 o = *reinterpret_cast<const f32x4 *>(&Os[buf][row][4 * c4]);
#pragma unroll
                for (int e = 0; e < 4; ++e) acc = fmaf(a[e], o[e], acc);
            }
#pragma unroll
            for (int m = TPR / 2; m >= 1; m >>= 1) acc += xor_lanes(acc, m);
            if (part == 0) Ds[buf][row] = acc;
        }
    };

    if (qstart < qstop) wait_vmcnt<0>();
    __syncthreads();   // first tile, its LSE/D and Kt visible
    if (LOCALD) {
        if (qstart < qstop) local_d(0);
        __syncthreads();   // its D visible
    }

    for (int qt = qstart; qt < qstop; ++qt) {
        const int cb = (NB == 2) ? ((qt - qstart) & 1) : 0;
        if (qt > qstart) store_dq(qt - 1);
        if (NB == 2 && qt + 1 < qstop) fetch(qt + 1, cb ^ 1);

        // A wave whose 16 keys are all masked for every row of this query
        // tile (padded keys, or keys past the tile's last row under a causal
        // mask) contributes nothing but its zero block of dS.
        const bool live = wkey0 < klen && (!causal || wkey0 - diag <= qt * BR + BR - 1);
        if (live) {
            f32x4 sacc[NIB], pacc[NIB];
#pragma unroll
            for (int ib = 0; ib < NIB; ++ib) {
                sacc[ib] = zero4();
                pacc[ib] = zero4();
            }
            // S = Q K^T, then dP = dO V^T: one product at a time keeps one
            // set of A operands live, so the kernel fits in 128 VGPRs (four
            // waves per SIMD, two 8-wave workgroups per CU).
#pragma unroll
            for (int s4 = 0; s4 < DQ / 4; ++s4) {
                f32x4 aq[NIB];
#pragma unroll
                for (int ib = 0; ib < NIB; ++ib)
                    aq[ib] = *reinterpret_cast<const f32x4 *>(&Qs[cb][16 * ib + il][g * DQ + 4 * s4]);
#pragma unroll
                for (int e = 0; e < 4; ++e)
#pragma unroll
                    for (int ib = 0; ib < NIB; ++ib)
                        sacc[ib] = mfma16x16x4(aq[ib][e], kreg[4 * s4 + e], sacc[ib]);
            }
#pragma unroll
            for (int s4 = 0; s4 < DQ / 4; ++s4) {
                f32x4 ao[NIB];
#pragma unroll
                for (int ib = 0; ib < NIB; ++ib)
                    ao[ib] = *reinterpret_cast<const f32x4 *>(&dOs[cb][16 * ib + il][g * DQ + 4 * s4]);
#pragma unroll
                for (int e = 0; e < 4; ++e)
#pragma unroll
                    for (int ib = 0; ib < NIB; ++ib)
                        pacc[ib] = mfma16x16x4(ao[ib][e], vreg[4 * s4 + e], pacc[ib]);
            }

            const int ibase = qt * BR + 4 * g;
            const int thr = kthr - ibase;
#pragma unroll
            for (int ib = 0; ib < NIB; ++ib) {
                const f32x4 l2 = *reinterpret_cast<const f32x4 *>(&lse2s[cb][16 * ib + 4 * g]) * kLog2e;
                const f32x4 dd = *reinterpret_cast<const f32x4 *>(&Ds[cb][16 * ib + 4 * g]);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    float p = exp2_fast(sacc[ib][r] * scale_log2 - l2[r]);
                    p = (16 * ib + r >= thr) ? p : 0.f;
                    sacc[ib][r] = p;
                    pacc[ib][r] = p * (pacc[ib][r] - dd[r]);
                    dSs[16 * ib + 4 * g + r][16 * w + il] = pacc[ib][r];
                }
            }

#pragma unroll
            for (int ib = 0; ib < NIB; ++ib)
#pragma unroll
                for (int r = 0; r < 4; ++r)
#pragma unroll
                    for (int c = 0; c < NC; ++c) {
                        dvacc[c] = mfma16x16x4(dOs[cb][16 * ib + 4 * g + r][16 * c + il],
                                               sacc[ib][r], dvacc[c]);
                        dkacc[c] = mfma16x16x4(Qs[cb][16 * ib + 4 * g + r][16 * c + il],
                                               pacc[ib][r], dkacc[c]);
                    }
        } else {
#pragma unroll
            for (int ib = 0; ib < NIB; ++ib)
#pragma unroll
                for (int r = 0; r < 4; ++r) dSs[16 * ib + 4 * g + r][16 * w + il] = 0.f;
        }

        __syncthreads();   // dS complete (and, single-buffered, Q/dO consumed)
        if (NB == 1 && qt + 1 < qstop) fetch(qt + 1, 0);

        // dQ_part^T[16c + 4g + r][16ib + il] = sum_j K^T[16c + il'][j] dS^T[j][16ib + il]
        // over the 16-key blocks that hold an allowed key for some row of the
        // tile (the rest of dS is zero: past the key length, or past the
        // tile's last row under a causal mask)
        int qblocks = min(KR / 16, (klen - k0 + 15) / 16);
        if (causal) qblocks = min(qblocks, max(0, qt * BR + BR - 1 + diag - k0) / 16 + 1);
        // (full tiles keep a loop without exits, which the compiler schedules freely)
        auto dq_product = [&](auto full) {
#pragma unroll
            for (int bb = 0; bb < PER_WAVE; ++bb) {
                const int blk = dq_block(bb);
                if (NBLK % C::NW != 0 && blk >= NBLK) break;
                const int ib = blk / NC;
                const int c = blk - ib * NC;
                f32x4 acc = zero4();
#pragma unroll
                for (int q = 0; q < KR / 16; ++q) {
                    if (!decltype(full)::value && q >= qblocks) break;
                    const f32x4 bv = *reinterpret_cast<const f32x4 *>(&dSs[16 * ib + il][16 * q + 4 * g]);
                    const f32x4 av = *reinterpret_cast<const f32x4 *>(&Kt[16 * c + il][16 * q + 4 * g]);
#pragma unroll
                    for (int e = 0; e < 4; ++e) acc = mfma16x16x4(av[e], bv[e], acc);
                }
                dqacc[bb] = acc;
            }
        };
        if (qblocks == KR / 16)
            dq_product(std::true_type{});
        else
            dq_product(std::false_type{});

        if (qt + 1 < qstop) wait_vmcnt<0>();   // next Q/dO tile and its LSE/D landed
        __syncthreads();   // next tile visible; dS and this tile's buffer free
        if (LOCALD) {
            if (qt + 1 < qstop) local_d(NB == 2 ? (cb ^ 1) : 0);
            __syncthreads();   // its D visible
        }
    }
    if (qstart < qstop) store_dq(qstop - 1);
    if (LOCALD && direct_dq) {
        // rows no query tile of this workgroup wrote (none see a key) get zeros
        float *dqh = dQp + (size_t)head * Lq * D;
        const int r0 = min(qstart * BR, Lq), r1 = min(qstop * BR, Lq);
        const int nz = (r0 + (Lq - r1)) * (D / 4);
        for (int f = tid; f < nz; f += C::NT) {
            const int rr = f / (D / 4);
            const int row = rr < r0 ? rr : r1 + (rr - r0);
            *reinterpret_cast<f32x4 *>(dqh + (size_t)row * D + 4 * (f - rr * (D / 4))) = zero4();
        }
    }

    // One split writes dK and dV directly; several write partials laid out
    // [dK, dV][split][B*H][Lk][d] (every split writes its rows, zeros for an
    // empty share) for attn_bwd_reduce_f32.
    if (kj < Lk) {
        const bool keep = kj < klen;
        const size_t row = hoff + (size_t)kj * D;
        const size_t part = (size_t)BH * Lk * D;
        float *dkrow = (nsplit == 1) ? dK + row : dKVp + (size_t)split * part + row;
        float *dvrow = (nsplit == 1) ? dV + row : dKVp + (size_t)(nsplit + split) * part + row;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            *reinterpret_cast<f32x4 *>(dkrow + 16 * c + 4 * g) = keep ? dkacc[c] * scale : zero4();
            *reinterpret_cast<f32x4 *>(dvrow + 16 * c + 4 * g) = keep ? dvacc[c] : zero4();
        }
    }
}

// dK and dV from the per-split partials of attn_dkdvq_f32, added in
// increasing split order (a fixed order).  n4 = B*H*Lk*d / 4; idx runs over
// the 2*n4 16-byte chunks of dK then dV.
__device__ __forceinline__ void dkdv_reduce_at(long idx, const float *__restrict__ dKVp,
                                               float *__restrict__ dK, float *__restrict__ dV,
                                               int nsplit, long n4) {
    if (idx >= 2 * n4) return;
    const int t = idx >= n4;           // 0: dK, 1: dV
    const long e4 = idx - t * n4;
    const f32x4 *src = reinterpret_cast<const f32x4 *>(dKVp) + (long)t * nsplit * n4 + e4;
    f32x4 sum = zero4();
    for (int s = 0; s < nsplit; ++s) sum += src[(long)s * n4];
    reinterpret_cast<f32x4 *>(t ? dV : dK)[e4] = sum;
}

// dQ[i] = scale * sum over key tiles kt that hold an allowed key for row i of
// dQ_part[kt][i], added in increasing kt (a fixed order).  Partials are laid
// out [key tile][B*H][Lq][d].
template <int D>
__device__ __forceinline__ void dq_reduce_at(size_t idx, const float *__restrict__ dQp,
                                             float *__restrict__ dQ,
                                             const int32_t *__restrict__ key_len, int H, int Lq,
                                             int Lk, int causal, float scale, int BH,
                                             int key_rows) {
    constexpr int C4 = D / 4;
    const size_t total = (size_t)BH * Lq * C4;
    if (idx >= total) return;
    const size_t rowg = idx / C4;              // head * Lq + i
    const int head = (int)(rowg / Lq);
    const int i = (int)(rowg - (size_t)head * Lq);
    const int klen = key_limit(key_len, head / H, Lk);
    const int nk = (klen + key_rows - 1) / key_rows;
    // causal: row i sees keys j <= i + Lk - Lq, i.e. key tiles up to that key's
    const int last = i + Lk - Lq;
    const int kmax = causal ? (last < 0 ? 0 : min(nk, last / key_rows + 1)) : nk;
    const size_t stride = (size_t)BH * Lq * D;
    const float *src = dQp + idx * 4;
    f32x4 sum = zero4();
    for (int kt = 0; kt < kmax; ++kt)
        sum += *reinterpret_cast<const f32x4 *>(src + (size_t)kt * stride);
    *reinterpret_cast<f32x4 *>(dQ + idx * 4) = sum * scale;
}

template <int D>
__global__ __launch_bounds__(256) void attn_dq_reduce_f32(const float *__restrict__ dQp,
                                                          float *__restrict__ dQ,
                                                          const int32_t *__restrict__ key_len,
                                                          int H, int Lq, int Lk, int causal,
                                                          float scale, int BH, int key_rows) {
    dq_reduce_at<D>((size_t)blockIdx.x * 256 + threadIdx.x, dQp, dQ, key_len, H, Lq, Lk, causal,
                    scale, BH, key_rows);
}

// Both reductions of a query-split fused backward in one launch: the first
// nb_kv workgroups add the dK/dV partials, the rest the dQ partials.
template <int D>
__global__ __launch_bounds__(256) void attn_bwd_reduce_f32(
    const float *__restrict__ dKVp, float *__restrict__ dK, float *__restrict__ dV, int nsplit,
    long n4, unsigned nb_kv, const float *__restrict__ dQp, float *__restrict__ dQ,
    const int32_t *__restrict__ key_len, int H, int Lq, int Lk, int causal, float scale, int BH,
    int key_rows) {
    if (blockIdx.x < nb_kv)
        dkdv_reduce_at((long)blockIdx.x * 256 + threadIdx.x, dKVp, dK, dV, nsplit, n4);
    else
        dq_reduce_at<D>((size_t)(blockIdx.x - nb_kv) * 256 + threadIdx.x, dQp, dQ, key_len, H,
                        Lq, Lk, causal, scale, BH, key_rows);
}

// ------------------------------------------------------------ backward: dQ
// Query tile of C::ROWS rows stationary (16 per wave); key tiles stream.
template <int D, class C>
__global__ __launch_bounds__(C::NT) __attribute__((amdgpu_waves_per_eu(C::template occ<D>(), 8)))
void attn_dq_f32(const float *__restrict__ Q, const float *__restrict__ K,
                 const float *__restrict__ V, const float *__restrict__ dO,
                 const float *__restrict__ LSE, const float *__restrict__ Dws,
                 float *__restrict__ dQ, const int32_t *__restrict__ key_len, int H, int Lq,
                 int Lk, int causal, float scale, float scale_log2, int n_qtiles, int BH, int layer) {
    constexpr int DQ = D / 4;
    constexpr int NC = D / 16;
    using Stager = F32TileStager<kStream, D, C::NT>;
    constexpr int LD = Stager::kLd;
    __shared__ __attribute__((aligned(16))) float Ks[C::NBUF][kStream][LD];
    __shared__ __attribute__((aligned(16))) float Vs[C::NBUF][kStream][LD];

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
    const int il = lane & 15;
    const int g = lane >> 4;
    const int q0 = qt * C::ROWS;
    const int qi = q0 + 16 * (tid >> 6) + il;

    const int klen = key_limit(key_len, b, Lk);
    const int kend = causal ? min(klen, q0 + C::ROWS + diag) : klen;
    const int ntiles = (kend + kStream - 1) / kStream;

    float qreg[DQ], oreg[DQ];
#pragma unroll
    for (int s4 = 0; s4 < DQ / 4; ++s4) {
        const size_t off = qoff + (size_t)qi * D + g * DQ + 4 * s4;
        const f32x4 qv = (qi < Lq) ? *reinterpret_cast<const f32x4 *>(Q + off) : zero4();
        const f32x4 ov = (qi < Lq) ? *reinterpret_cast<const f32x4 *>(dO + off) : zero4();
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            qreg[4 * s4 + e] = qv[e];
            oreg[4 * s4 + e] = ov[e];
        }
    }
    const float lse2 = (qi < Lq) ? LSE[(size_t)head * Lq + qi] * kLog2e : 0.f;
    const float Di = (qi < Lq) ? Dws[(size_t)head * Lq + qi] : 0.f;

    f32x4 dqacc[NC];   // dQ^T[16c + 4g + r][qi]
#pragma unroll
    for (int c = 0; c < NC; ++c) dqacc[c] = zero4();

    Stager kst, vst;
    if (ntiles > 0) {
        kst.load(Kh, 0, Lk, tid);
        vst.load(Vh, 0, Lk, tid);
        if (C::NBUF == 2) {
            kst.store(Ks[0], tid);
            vst.store(Vs[0], tid);
            __syncthreads();
        }
    }
    for (int kt = 0; kt < ntiles; ++kt) {
        const int cur = (C::NBUF == 2) ? (kt & 1) : 0;
        if (C::NBUF == 1) {
            __syncthreads();
            kst.store(Ks[0], tid);
            vst.store(Vs[0], tid);
            __syncthreads();
        }
        if (kt + 1 < ntiles) {
            kst.load(Kh, (kt + 1) * kStream, Lk, tid);
            vst.load(Vh, (kt + 1) * kStream, Lk, tid);
        }

        // S^T[j][qi] and dP^T[j][qi], j = 16jb + 4g + r
        f32x4 sacc[4], pacc[4];
#pragma unroll
        for (int jb = 0; jb < 4; ++jb) {
            sacc[jb] = zero4();
            pacc[jb] = zero4();
        }
#pragma unroll
        for (int s4 = 0; s4 < DQ / 4; ++s4) {
            f32x4 ak[4], av[4];
#pragma unroll
            for (int jb = 0; jb < 4; ++jb) {
                ak[jb] = *reinterpret_cast<const f32x4 *>(&Ks[cur][16 * jb + il][g * DQ + 4 * s4]);
                av[jb] = *reinterpret_cast<const f32x4 *>(&Vs[cur][16 * jb + il][g * DQ + 4 * s4]);
            }
#pragma unroll
            for (int e = 0; e < 4; ++e)
#pragma unroll
                for (int jb = 0; jb < 4; ++jb) {
                    sacc[jb] = mfma16x16x4(ak[jb][e], qreg[4 * s4 + e], sacc[jb]);
                    pacc[jb] = mfma16x16x4(av[jb][e], oreg[4 * s4 + e], pacc[jb]);
                }
        }

        // Element (jb, r) holds key j0 + 16jb + r; same threshold as forward.
        const int j0 = kt * kStream + 4 * g;
        const int thr = causal ? min(klen - j0, qi + diag - j0 + 1) : klen - j0;
#pragma unroll
        for (int jb = 0; jb < 4; ++jb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                float p = exp2_fast(sacc[jb][r] * scale_log2 - lse2);
                p = (16 * jb + r < thr) ? p : 0.f;
                pacc[jb][r] = p * (pacc[jb][r] - Di);
            }

        // dQ^T[16c + 4g + r][qi] += sum_j K[j][16c + il'] dS^T[j][qi]
#pragma unroll
        for (int jb = 0; jb < 4; ++jb)
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int c = 0; c < NC; ++c)
                    dqacc[c] = mfma16x16x4(Ks[cur][16 * jb + 4 * g + r][16 * c + il],
                                           pacc[jb][r], dqacc[c]);

        if (C::NBUF == 2) {
            if (kt + 1 < ntiles) {
                kst.store(Ks[cur ^ 1], tid);
                vst.store(Vs[cur ^ 1], tid);
            }
            __syncthreads();
        }
    }

    if (qi < Lq) {
        float *dqrow = dQ + qoff + (size_t)qi * D;
#pragma unroll
        for (int c = 0; c < NC; ++c)
            *reinterpret_cast<f32x4 *>(dqrow + 16 * c + 4 * g) = dqacc[c] * scale;
    }
}

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

// Key-padded non-causal grids take the XCD-grouped work orders
// (heavy_first_tile, work_first_tile) when the heads split evenly over the
// eight XCDs, at most 64 per XCD, and the per-workgroup search (one ballot
// per key tile) stays short: at most 1024 key tiles.
inline int padded_work_order(const AttnProblem &p) {
    const int BH = p.B * p.H;
    return (p.key_len != nullptr && !p.causal && BH % 8 == 0 && BH <= 512 &&
            p.Lk <= 1024 * 64) ? 1 : 0;
}

}  // namespace

// ---------------------------------------------------------------- launchers
namespace {
template <class C, class Kern>
void launch_fwd_f32_as(Kern kern, int ksplit, const AttnProblem &p, const float *Q,
                       const float *K, const float *V, float *O, float *LSE, hipStream_t s) {
    const int BH = p.B * p.H;
    const int nqt = cdiv(p.Lq, C::ROWS);
    const dim3 grid(nqt * BH), block(C::NT * ksplit);
    const int ly = causal_rank_layer((const void *)kern, block.x, grid.x, BH, p.causal);
    kern<<<grid, block, 0, s>>>(Q, K, V, O, LSE, p.key_len, p.H, p.Lq, p.Lk, p.causal,
                                p.scale * kLog2e, nqt, BH, ly, padded_work_order(p));
}
}  // namespace

hipError_t launch_fwd_f32(const AttnProblem &p, const float *Q, const float *K,
                          const float *V, float *O, float *LSE, hipStream_t s) {
    // Grids of fewer than MG_FWD_SPLIT_BELOW workgroups of 64 rows fall
    // unevenly on the CUs (288 of them on 256 CUs put two on 32 CUs, which
    // then set the kernel's time).  There the query tiles shrink to 32 rows
    // and each workgroup splits its key tiles over two halves: four times
    // the workgroups, each a quarter of the work (d <= 64, two or more key tiles).
    // When even the 32-row grid leaves most CUs without a workgroup and the
    // key side is long, the key tiles go to four groups instead of two.
    const long grid = (long)cdiv(p.Lq, FwdCfg::ROWS) * p.B * p.H;
    const bool split = p.d <= 64 && grid < MG_FWD_SPLIT_BELOW && p.Lk > kFwdStream;
    const bool split4 = split && (long)cdiv(p.Lq, FwdSplitCfg::ROWS) * p.B * p.H <=
                                     MG_FWD_SPLIT4_UPTO && p.Lk >= MG_FWD_SPLIT4_MIN_KEYS;
    switch (p.d) {
    case 32:
        if (split4)
            launch_fwd_f32_as<FwdSplitCfg>(attn_fwd_f32_ks4<32, FwdSplitCfg>, 4, p, Q, K, V, O,
                                           LSE, s);
        else if (split)
            launch_fwd_f32_as<FwdSplitCfg>(attn_fwd_f32_ks2<32, FwdSplitCfg>, 2, p, Q, K, V, O,
                                           LSE, s);
        else
            launch_fwd_f32_as<FwdCfg>(attn_fwd_f32<32, FwdCfg>, 1, p, Q, K, V, O, LSE, s);
        break;
    case 64:
        if (split4)
            launch_fwd_f32_as<FwdSplitCfg>(attn_fwd_f32_ks4<64, FwdSplitCfg>, 4, p, Q, K, V, O,
                                           LSE, s);
        else if (split)
            launch_fwd_f32_as<FwdSplitCfg>(attn_fwd_f32_ks2<64, FwdSplitCfg>, 2, p, Q, K, V, O,
                                           LSE, s);
        else
            launch_fwd_f32_as<FwdCfg>(attn_fwd_f32<64, FwdCfg>, 1, p, Q, K, V, O, LSE, s);
        break;
    case 128: launch_fwd_f32_as<FwdCfg>(attn_fwd_f32<128, FwdCfg>, 1, p, Q, K, V, O, LSE, s); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_bwd_rowdot_f32(const AttnProblem &p, const float *O, const float *dO,
                                 float *Dws, hipStream_t s) {
    const int rows = p.B * p.H * p.Lq;
    const dim3 block(256);
    switch (p.d) {
    case 32: attn_rowdot_f32<32><<<dim3(cdiv(rows, 256 / 8)), block, 0, s>>>(O, dO, Dws, rows); break;
    case 64: attn_rowdot_f32<64><<<dim3(cdiv(rows, 256 / 16)), block, 0, s>>>(O, dO, Dws, rows); break;
    case 128: attn_rowdot_f32<128><<<dim3(cdiv(rows, 256 / 32)), block, 0, s>>>(O, dO, Dws, rows); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_bwd_dkdv_f32(const AttnProblem &p, const float *Q, const float *K,
                               const float *V, const float *dO, const float *LSE,
                               const float *Dws, float *dK, float *dV, hipStream_t s) {
    using C = DkdvCfg;
    const int BH = p.B * p.H;
    const dim3 grid(cdiv(p.Lk, C::ROWS) * BH), block(C::NT);
    const float sl2 = p.scale * kLog2e;
    auto go = [&](auto kern) {
        const int ly = causal_rank_layer((const void *)kern, C::NT, grid.x, BH, p.causal);
        kern<<<grid, block, 0, s>>>(Q, K, V, dO, LSE, Dws, dK, dV, p.key_len, p.H, p.Lq, p.Lk,
                                    p.causal, p.scale, sl2, BH, ly);
    };
    switch (p.d) {
    case 32: go(attn_dkdv_f32<32, MG_DKDV_NIB, C>); break;
    case 64: go(attn_dkdv_f32<64, MG_DKDV_NIB, C>); break;
    case 128: go(attn_dkdv_f32<128, 2, C>); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// Fused dQ: causal problems with enough work use 128-key tiles (heavy-first
// ordering keeps the fewer workgroups balanced, and the partials halve);
// the rest keep 64-key tiles, which measured faster there.
bool wide_key_tiles(const AttnProblem &p) {
    return p.causal && (long)cdiv(p.Lk, DkdvqCausalCfg::ROWS) * p.B * p.H >= 512;
}
int fused_dq_key_rows(const AttnProblem &p) {
    return wide_key_tiles(p) ? DkdvqCausalCfg::ROWS : DkdvCfg::ROWS;
}

// Few keys (a short context, few heads) leave the key-stationary grid far
// smaller than the chip: below MG_DKDV_SPLIT_BELOW workgroups, each key
// tile's query tiles are split over up to ceil(MG_DKDV_SPLIT_TARGET / grid)
// workgroups, keeping at least MG_DKDV_SPLIT_MIN_TILES query tiles each.
#ifndef MG_DKDV_SPLIT_BELOW
#define MG_DKDV_SPLIT_BELOW 512
#endif
#ifndef MG_DKDV_SPLIT_TARGET
#define MG_DKDV_SPLIT_TARGET 1024
#endif
#ifndef MG_DKDV_SPLIT_MIN_TILES
#define MG_DKDV_SPLIT_MIN_TILES 4
#endif
int fused_dq_query_splits(const AttnProblem &p) {
    const long grid = (long)cdiv(p.Lk, fused_dq_key_rows(p)) * p.B * p.H;
    if (grid >= MG_DKDV_SPLIT_BELOW) return 1;
    const int br = 16 * (wide_key_tiles(p) ? MG_DKDVQ_CAUSAL_NIB : MG_DKDV_NIB);
    const long by_grid = (MG_DKDV_SPLIT_TARGET + grid - 1) / grid;
    // short query sides (at most 8 tiles) split down to 2 tiles per share:
    // each share is then latency-bound, and finer shares measured faster
    const int nqt = cdiv(p.Lq, br);
    const long by_tiles = nqt / (nqt <= 8 ? 2 : MG_DKDV_SPLIT_MIN_TILES);
    return (int)std::max(1L, std::min(by_grid, by_tiles));
}

// Small fused grids compute D in the kernel (LOCALD): at most this many key
// tiles per head, so that each query tile's O rows are read a few times, and
// a grid below MG_DKDV_SPLIT_BELOW workgroups.
#ifndef MG_LOCAL_D_MAX_KEY_TILES
#define MG_LOCAL_D_MAX_KEY_TILES 4
#endif
bool fused_local_d(const AttnProblem &p) {
    const long nkt = cdiv(p.Lk, fused_dq_key_rows(p));
    return nkt <= MG_LOCAL_D_MAX_KEY_TILES && nkt * p.B * p.H < MG_DKDV_SPLIT_BELOW;
}
bool fused_direct_dq(const AttnProblem &p) {
    return fused_local_d(p) && cdiv(p.Lk, fused_dq_key_rows(p)) == 1 &&
           fused_dq_query_splits(p) == 1;
}

template <class C, int NIB>
static hipError_t launch_dkdvq(const AttnProblem &p, const float *Q, const float *K,
                               const float *V, const float *O, const float *dO,
                               const float *LSE, const float *Dws, float *dK, float *dV,
                               float *dQp, float *dKVp, hipStream_t s) {
    const int BH = p.B * p.H;
    const int ns = fused_dq_query_splits(p);
    const int nr = cdiv(p.Lk, C::ROWS) * ns;   // ranks: key tile x split
    const dim3 grid(nr * BH), block(C::NT);
    const float sl2 = p.scale * kLog2e;
    const int direct = fused_direct_dq(p) ? 1 : 0;
    auto go = [&](auto kern) {
        const int ly = causal_rank_layer((const void *)kern, C::NT, grid.x, BH, p.causal);
        kern<<<grid, block, 0, s>>>(Q, K, V, O, dO, LSE, Dws, dK, dV, dQp, dKVp, p.key_len,
                                    p.H, p.Lq, p.Lk, p.causal, p.scale, sl2, BH, ns, nr, ly,
                                    padded_work_order(p), direct);
    };
    // Local D only in the 64-key form: grids small enough for it never take
    // the 128-key tiles, which need at least 512 workgroups.
    constexpr bool kLocalForm = !std::is_same<C, DkdvqCausalCfg>::value;
    const bool local = kLocalForm && fused_local_d(p);
    auto pick = [&](auto plain, auto with_local) {
        if constexpr (kLocalForm) {
            if (local) return go(with_local);
        }
        go(plain);
    };
    switch (p.d) {
    case 32: pick(attn_dkdvq_f32<32, NIB, C, false>, attn_dkdvq_f32<32, NIB, C, kLocalForm>); break;
    case 64: pick(attn_dkdvq_f32<64, NIB, C, false>, attn_dkdvq_f32<64, NIB, C, kLocalForm>); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_bwd_dkdvq_f32(const AttnProblem &p, const float *Q, const float *K,
                                const float *V, const float *O, const float *dO,
                                const float *LSE, const float *Dws, float *dK, float *dV,
                                float *dQp, float *dKVp, hipStream_t s) {
    if (fused_dq_query_splits(p) > 1 && dKVp == nullptr) return hipErrorInvalidValue;
    return wide_key_tiles(p)
        ? launch_dkdvq<DkdvqCausalCfg, MG_DKDVQ_CAUSAL_NIB>(p, Q, K, V, O, dO, LSE, Dws, dK, dV,
                                                            dQp, dKVp, s)
        : launch_dkdvq<DkdvCfg, MG_DKDV_NIB>(p, Q, K, V, O, dO, LSE, Dws, dK, dV, dQp, dKVp, s);
}

hipError_t launch_bwd_reduce_f32(const AttnProblem &p, const float *dKVp, float *dK,
                                 float *dV, const float *dQp, float *dQ, hipStream_t s) {
    const int BH = p.B * p.H;
    const long n4 = (long)BH * p.Lk * p.d / 4;
    const unsigned nb_kv = (unsigned)((2 * n4 + 255) / 256);
    const size_t total = (size_t)BH * p.Lq * (p.d / 4);
    const dim3 grid(nb_kv + (unsigned)((total + 255) / 256)), block(256);
    const int ns = fused_dq_query_splits(p), kr = fused_dq_key_rows(p);
    switch (p.d) {
    case 32: attn_bwd_reduce_f32<32><<<grid, block, 0, s>>>(dKVp, dK, dV, ns, n4, nb_kv, dQp, dQ, p.key_len, p.H, p.Lq, p.Lk, p.causal, p.scale, BH, kr); break;
    case 64: attn_bwd_reduce_f32<64><<<grid, block, 0, s>>>(dKVp, dK, dV, ns, n4, nb_kv, dQp, dQ, p.key_len, p.H, p.Lq, p.Lk, p.causal, p.scale, BH, kr); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_bwd_dq_reduce_f32(const AttnProblem &p, const float *dQp, float *dQ,
                                    hipStream_t s) {
    const int BH = p.B * p.H;
    const size_t total = (size_t)BH * p.Lq * (p.d / 4);
    const dim3 grid((unsigned)((total + 255) / 256)), block(256);
    const int kr = fused_dq_key_rows(p);
    switch (p.d) {
    case 32: attn_dq_reduce_f32<32><<<grid, block, 0, s>>>(dQp, dQ, p.key_len, p.H, p.Lq, p.Lk, p.causal, p.scale, BH, kr); break;
    case 64: attn_dq_reduce_f32<64><<<grid, block, 0, s>>>(dQp, dQ, p.key_len, p.H, p.Lq, p.Lk, p.causal, p.scale, BH, kr); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_bwd_dq_f32(const AttnProblem &p, const float *Q, const float *K,
                             const float *V, const float *dO, const float *LSE,
                             const float *Dws, float *dQ, hipStream_t s) {
    using C = DqCfg;
    const int BH = p.B * p.H;
    const int nqt = cdiv(p.Lq, C::ROWS);
    const dim3 grid(nqt * BH), block(C::NT);
    const float sl2 = p.scale * kLog2e;
    auto go = [&](auto kern) {
        const int ly = causal_rank_layer((const void *)kern, C::NT, grid.x, BH, p.causal);
        kern<<<grid, block, 0, s>>>(Q, K, V, dO, LSE, Dws, dQ, p.key_len, p.H, p.Lq, p.Lk,
                                    p.causal, p.scale, sl2, nqt, BH, ly);
    };
    switch (p.d) {
    case 32: go(attn_dq_f32<32, C>); break;
    case 64: go(attn_dq_f32<64, C>); break;
    case 128: go(attn_dq_f32<128, C>); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace mg
