// device_common.h -- device helpers shared by the gfx950 attention kernels.
//
// Matrix-core conventions used throughout (CDNA3/CDNA4 MFMA, wave64):
//
//   v_mfma_f32_16x16x4_f32   C[16x16] += A[16x4] * B[4x16]
//     lane l holds A[l%16][l/16], B[l/16][l%16] (one f32 each) and
//     C[4*(l/16) + r][l%16] in accumulator register r = 0..3.
//
//   v_mfma_f32_16x16x32_bf16 C[16x16] += A[16x32] * B[32x16]
//     lane l holds 8 bf16 of A row l%16 and 8 bf16 of B column l%16; the
//     eight contraction indices a lane holds are the same set for A and B,
//     and C has the layout above.
//
// Because a contraction index only has to mean the same thing in A and B,
// each kernel picks the contraction order that makes its loads contiguous.
// An accumulator C[x][y] (x by lane group and register, y = lane%16) can
// feed the next product directly as its B operand (contraction over x,
// output columns y), which is how P and dS reach the second GEMM of each
// pass without a trip through LDS.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mg {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
// Online-softmax slack (base 2): a forward may keep a running maximum up to
// this far below the true one, so probabilities stay at most 2^kSlack.
constexpr float kSlack = 8.f;
constexpr float kLn2 = 0.69314718055994531f;

__device__ __forceinline__ f32x4 mfma16x16x4(float a, float b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x4 mfma16x16x32bf16(bf16x8 a, bf16x8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// v_mfma_f32_32x32x16_bf16: C[32x32] += A[32x16] * B[16x32]; lane l holds 8
// bf16 of A row l%32 and of B column l%32 (the same 8 contraction indices
// for both), and C[8*(v/4) + 4*(l/32) + v%4][l%32] in register v = 0..15.
__device__ __forceinline__ f32x16 mfma32x32x16bf16(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Scheduling request for the region (basic block) in which it is placed:
// PRE of its NREADS LDS reads first, then groups of MPG matrix products and
// RPG reads in turn, then the remaining products.  A wave then keeps about
// PRE operand reads in flight ahead of the products that consume them,
// instead of the one or two the default schedule issues when registers are
// tight.  (Mask 0x100: LDS reads; 0x008: matrix instructions.)
// (PRE is capped at NREADS for small regions.)
template <int NREADS, int NMFMA, int PRE_, int RPG, int MPG, int ID>
__device__ __forceinline__ void sched_reads_ahead() {
    constexpr int PRE = PRE_ < NREADS ? PRE_ : NREADS;
    constexpr int NG = (NREADS - PRE) / RPG;
    static_assert((NREADS - PRE) % RPG == 0 && MPG * NG <= NMFMA,
                  "read and product counts of the region");
    __builtin_amdgcn_sched_group_barrier(0x100, PRE, ID);
#pragma unroll
    for (int u = 0; u < NG; ++u) {
        __builtin_amdgcn_sched_group_barrier(0x008, MPG, ID);
        __builtin_amdgcn_sched_group_barrier(0x100, RPG, ID);
    }
    if constexpr (NMFMA > MPG * NG)
        __builtin_amdgcn_sched_group_barrier(0x008, NMFMA - MPG * NG, ID);
}

__device__ __forceinline__ f32x16 zero16() {
    f32x16 z;
#pragma unroll
    for (int i = 0; i < 16; ++i) z[i] = 0.f;
    return z;
}

// 2^x on the transcendental unit (v_exp_f32); 2^-inf = 0.
__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float xor_lanes(float v, int mask) { return __shfl_xor(v, mask, 64); }
// max(a, b, c) as one v_max3_f32.  Written out because in IEEE mode the
// compiler must quiet a possible signalling NaN before each fmaxf, and for
// values it cannot prove canonical (matrix-core results) it spends one
// v_max per input on that; the row maxima here are taken over MFMA results
// and -inf, which are never signalling NaNs.
__device__ __forceinline__ float max3_f32(float a, float b, float c) {
    float r;
    asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
    return r;
}


// Cross-row exchanges on the VALU (no LDS crossbar round trip).  For
// v_permlane16_swap(x, x) every lane receives {x of the even 16-lane row,
// x of the odd row} of its row pair, in that order; v_permlane32_swap does the
// same for the two 32-lane halves.  Combining the pair therefore yields the
// same value, bit for bit, on both partners.
__device__ __forceinline__ float max_xor16(float v) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float max_xor32(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_xor16(float v) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float sum_xor32(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Reductions across the four 16-lane groups that share one column l%16.
__device__ __forceinline__ float max_over_groups(float v) { return max_xor32(max_xor16(v)); }
__device__ __forceinline__ float sum_over_groups(float v) { return sum_xor32(sum_xor16(v)); }

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

// f32 -> bf16 bits, round to nearest even (finite inputs; NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float x) {
    uint32_t u = __float_as_uint(x);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(((uint32_t)b) << 16);
}

// Word 3 of a gfx9-family buffer descriptor: 32-bit data format, every other
// field zero (no swizzle, no index stride); untyped dword loads need a
// non-zero data format.
constexpr int kBufferWord3 = 0x00020000;

// Descriptor of `bytes` bytes starting at `base` (stride 0: offsets are plain
// byte offsets; loads at offsets >= bytes return zero).  Both arguments must
// be the same on every lane of the wave; they are read from the first active
// lane so that the descriptor lives in scalar registers.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void *base, int bytes) {
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
    void *p = reinterpret_cast<void *>(((uint64_t)hi << 32) | lo);
    return __builtin_amdgcn_make_buffer_rsrc(p, (short)0, __builtin_amdgcn_readfirstlane(bytes),
                                             kBufferWord3);
}

__device__ __forceinline__ f32x4 buffer_load_f32x4(__amdgpu_buffer_rsrc_t r, int byte_offset) {
    return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, byte_offset, 0, 0));
}

// s_waitcnt immediate that waits until at most `N` vector-memory operations
// of this wave are outstanding (gfx9 encoding: vmcnt bits 3:0 in bits 3:0 and
// bits 5:4 in bits 15:14; expcnt and lgkmcnt left at their maxima, i.e. not
// waited for).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}

// Rank of the tile a workgroup takes.  Workgroups are dealt to the chip's
// compute units in layers (one workgroup slot on every CU per layer of
// `layer` ranks, `layer` * B*H workgroups); reversing the rank order in every
// other layer puts a heavy causal tile and a light one on the same CU.
// layer <= 0 keeps the plain order.
__device__ __forceinline__ int serpentine_rank(int rho, int nranks, int layer) {
    if (layer <= 0) return rho;
    const int s = rho / layer;
    if ((s & 1) == 0) return rho;
    const int base = s * layer;
    const int len = min(layer, nranks - base);
    return base + len - 1 - (rho - base);
}

// Clamp a per-batch key length to [0, L]; L when no padding is given.
__device__ __forceinline__ int key_limit(const int32_t *key_len, int b, int L) {
    if (key_len == nullptr) return L;
    int n = key_len[b];
    return n < 0 ? 0 : (n > L ? L : n);
}

}  // namespace mg
