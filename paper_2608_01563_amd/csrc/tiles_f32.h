// tiles_f32.h -- cooperative global->LDS staging of f32 row tiles.
//
// A tile is `ROWS` consecutive rows of one head's [L][D] matrix.  Every
// thread of the workgroup moves `kPerThread` 16-byte chunks: global reads are
// fully coalesced (consecutive threads read consecutive 16-byte chunks of a
// row) and land in a row-padded LDS array with stride D+4 floats, which keeps
// both the row-fragment reads (16 lanes on 16 rows, 16 bytes each) and the
// column reads (16 lanes along one row, 4 rows apart) free of bank conflicts.
// Rows at or beyond L are filled with zeros, so nothing past the tensor is
// read and masked rows stay finite.
#pragma once

#include "device_common.h"

namespace mg {

template <int ROWS, int D, int NTHREADS>
struct F32TileStager {
    static constexpr int kChunksPerRow = D / 4;
    static constexpr int kChunks = ROWS * kChunksPerRow;
    static constexpr int kPerThread = (kChunks + NTHREADS - 1) / NTHREADS;
    static constexpr bool kExact = kChunks % NTHREADS == 0;   // no idle threads
    static constexpr int kLd = D + 4;

    f32x4 buf[kPerThread];

    // Issue the global loads of rows [row0, row0+ROWS) of `src` (one head).
    __device__ __forceinline__ void load(const float *__restrict__ src, int row0, int L,
                                         int tid) {
#pragma unroll
        for (int u = 0; u < kPerThread; ++u) {
            const int f = tid + u * NTHREADS;
            const int r = f / kChunksPerRow;
            const int c4 = f - r * kChunksPerRow;
            const int row = row0 + r;
            buf[u] = ((kExact || f < kChunks) && row < L)
                ? *reinterpret_cast<const f32x4 *>(src + (size_t)row * D + 4 * c4)
                : zero4();
        }
    }

    // Write the loaded chunks into dst[ROWS][D+4].
    __device__ __forceinline__ void store(float (*dst)[kLd], int tid) const {
#pragma unroll
        for (int u = 0; u < kPerThread; ++u) {
            const int f = tid + u * NTHREADS;
            if (!kExact && f >= kChunks) continue;
            const int r = f / kChunksPerRow;
            const int c4 = f - r * kChunksPerRow;
            *reinterpret_cast<f32x4 *>(&dst[r][4 * c4]) = buf[u];
        }
    }
};

}  // namespace mg

namespace mg {

// Quad staging: each thread moves a 4-row x 4-column block of an f32 tile and
// writes it row-major R[ROWS][D+4] and/or transposed T[D][ROWS+4], both with
// 16-byte LDS stores (the 4x4 transpose happens in registers).  Quads are
// numbered row-group fastest, so a wave's transposed stores are contiguous.
// The transposed copy lets a lane read four consecutive rows of one column
// (the B-operand order of an accumulator) with a single 16-byte read.
template <int ROWS, int D, int NTHREADS, bool ROW_MAJOR, bool TRANSPOSED>
struct F32QuadStager {
    static constexpr int kLdR = D + 4;
    static constexpr int kLdT = ROWS + 4;
    static constexpr int kGroups = ROWS / 4;
    static constexpr int kQuads = kGroups * (D / 4);
    static constexpr int kIters = (kQuads + NTHREADS - 1) / NTHREADS;
    static_assert(ROWS % 4 == 0 && D % 4 == 0, "tile shape");

    f32x4 buf[kIters][4];

    __device__ __forceinline__ void load(const float *__restrict__ src, int row0, int L,
                                         int tid) {
#pragma unroll
        for (int it = 0; it < kIters; ++it) {
            const int q = tid + it * NTHREADS;
            const int rg = q % kGroups;
            const int c4 = q / kGroups;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int row = row0 + 4 * rg + k;
                buf[it][k] = (q < kQuads && row < L)
                    ? *reinterpret_cast<const f32x4 *>(src + (size_t)row * D + 4 * c4)
                    : zero4();
            }
        }
    }

    __device__ __forceinline__ void store(float (*R)[kLdR], float (*T)[kLdT], int tid) const {
#pragma unroll
        for (int it = 0; it < kIters; ++it) {
            const int q = tid + it * NTHREADS;
            if (kQuads % NTHREADS != 0 && q >= kQuads) continue;
            const int rg = q % kGroups;
            const int c4 = q / kGroups;
            if constexpr (ROW_MAJOR) {
#pragma unroll
                for (int k = 0; k < 4; ++k)
                    *reinterpret_cast<f32x4 *>(&R[4 * rg + k][4 * c4]) = buf[it][k];
            }
            if constexpr (TRANSPOSED) {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    *reinterpret_cast<f32x4 *>(&T[4 * c4 + e][4 * rg]) =
                        f32x4{buf[it][0][e], buf[it][1][e], buf[it][2][e], buf[it][3][e]};
            }
        }
    }
};

}  // namespace mg
