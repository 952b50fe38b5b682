// tiles_bf16.h -- cooperative global->LDS staging of bf16 row tiles, in
// row-major and/or transposed layout.
//
// bf16 MFMA (16x16x32) takes 8 contraction values per lane.  Products that
// contract over the head dimension read a tile row-major (8 consecutive d
// values = one 16-byte LDS read); products that contract over the streamed
// rows read it transposed (two runs of 4 consecutive rows = two 8-byte LDS
// reads).  Both layouts are written from one pass over global memory.
//
// Work unit: a quad = 4 consecutive rows x one 8-column chunk.  When a
// transposed copy is written, quads are numbered row-group fastest so the
// transposed 8-byte writes of a wave fall on consecutive LDS words; a
// row-major-only tile numbers them chunk fastest, so global reads and LDS
// writes of a wave are contiguous along each row.  Rows at or beyond L are
// zero-filled.
//
//   row-major  R[ROWS][D + 8]   (row stride 16-byte aligned; D+8 u16 words
//                                is 4 words past a multiple of 64 banks)
//   transposed T[D][ROWS + 4]   (row stride 8-byte aligned)
#pragma once

#include "device_common.h"

namespace mg {

template <int ROWS, int D, int NTHREADS, bool ROW_MAJOR, bool TRANSPOSED>
struct Bf16TileStager {
    static constexpr int kLdR = D + 8;
    static constexpr int kLdT = ROWS + 4;
    static constexpr int kGroups = ROWS / 4;          // row groups of 4
    static constexpr int kChunks = D / 8;             // 8-column chunks per row
    static constexpr int kQuads = kGroups * kChunks;
    static constexpr int kIters = (kQuads + NTHREADS - 1) / NTHREADS;
    static_assert(ROWS % 4 == 0 && D % 8 == 0, "tile shape");

    u32x4 buf[kIters][4];

    __device__ __forceinline__ void load(const uint16_t *__restrict__ src, int row0, int L,
                                         int tid) {
#pragma unroll
        for (int it = 0; it < kIters; ++it) {
            const int q = tid + it * NTHREADS;
            const int rg = TRANSPOSED ? q % kGroups : q / kChunks;
            const int c8 = TRANSPOSED ? q / kGroups : q % kChunks;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int row = row0 + 4 * rg + k;
                buf[it][k] = (q < kQuads && row < L)
                    ? *reinterpret_cast<const u32x4 *>(src + (size_t)row * D + 8 * c8)
                    : u32x4{0u, 0u, 0u, 0u};
            }
        }
    }

    __device__ __forceinline__ void store(uint16_t (*R)[kLdR], uint16_t (*T)[kLdT],
                                          int tid) const {
#pragma unroll
        for (int it = 0; it < kIters; ++it) {
            const int q = tid + it * NTHREADS;
            if (q >= kQuads) continue;
            const int rg = TRANSPOSED ? q % kGroups : q / kChunks;
            const int c8 = TRANSPOSED ? q / kGroups : q % kChunks;
            if constexpr (ROW_MAJOR) {
#pragma unroll
                for (int k = 0; k < 4; ++k)
                    *reinterpret_cast<u32x4 *>(&R[4 * rg + k][8 * c8]) = buf[it][k];
            }
            if constexpr (TRANSPOSED) {
                // column 8*c8 + e of rows 4rg..4rg+3 -> T[8*c8 + e][4rg..4rg+3]
#pragma unroll
                for (int m = 0; m < 4; ++m) {
                    const uint32_t w0 = buf[it][0][m], w1 = buf[it][1][m];
                    const uint32_t w2 = buf[it][2][m], w3 = buf[it][3][m];
                    // even element 2m: low halves; odd element 2m+1: high halves
                    const uint32_t lo01 = (w0 & 0xffffu) | (w1 << 16);
                    const uint32_t lo23 = (w2 & 0xffffu) | (w3 << 16);
                    const uint32_t hi01 = (w0 >> 16) | (w1 & 0xffff0000u);
                    const uint32_t hi23 = (w2 >> 16) | (w3 & 0xffff0000u);
                    *reinterpret_cast<uint64_t *>(&T[8 * c8 + 2 * m][4 * rg]) =
                        (uint64_t)lo01 | ((uint64_t)lo23 << 32);
                    *reinterpret_cast<uint64_t *>(&T[8 * c8 + 2 * m + 1][4 * rg]) =
                        (uint64_t)hi01 | ((uint64_t)hi23 << 32);
                }
            }
        }
    }
};

// Eight bf16 from 16 bytes of LDS or global memory.
__device__ __forceinline__ bf16x8 load_bf16x8(const uint16_t *p) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(p));
}

// Eight bf16 from two 8-byte runs (contraction positions 0..3 and 4..7).
__device__ __forceinline__ bf16x8 load_bf16x4x2(const uint16_t *lo, const uint16_t *hi) {
    typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
    const u32x2 a = *reinterpret_cast<const u32x2 *>(lo);
    const u32x2 b = *reinterpret_cast<const u32x2 *>(hi);
    return __builtin_bit_cast(bf16x8, u32x4{a[0], a[1], b[0], b[1]});
}

// Round two accumulator blocks (4 values each) to bf16 as one B operand:
// positions 0..3 from `a`, 4..7 from `b` (nearest-even rounding).
__device__ __forceinline__ bf16x8 pack_bf16(f32x4 a, f32x4 b) {
    bf16x8 v;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        v[r] = (__bf16)a[r];
        v[4 + r] = (__bf16)b[r];
    }
    return v;
}

// Accumulator registers [8t, 8t+8) of a 32x32 block, rounded to bf16 (nearest
// even), as the B operand of a 32x32x16 product contracting over its rows.
__device__ __forceinline__ bf16x8 pack_bf16_half(const f32x16 &a, int t) {
    bf16x8 v;
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = (__bf16)a[8 * t + e];
    return v;
}

// Four f32 -> four bf16 (nearest even) stored as 8 bytes.
__device__ __forceinline__ void store_bf16x4(uint16_t *dst, f32x4 v) {
    typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
    bf16x4 b;
#pragma unroll
    for (int r = 0; r < 4; ++r) b[r] = (__bf16)v[r];
    *reinterpret_cast<uint64_t *>(dst) = __builtin_bit_cast(uint64_t, b);
}

}  // namespace mg
