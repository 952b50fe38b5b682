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
    static_assert(kChunks % NTHREADS == 0, "tile must split evenly over threads");
    static constexpr int kPerThread = kChunks / NTHREADS;
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
            buf[u] = (row < L)
                ? *reinterpret_cast<const f32x4 *>(src + (size_t)row * D + 4 * c4)
                : zero4();
        }
    }

    // Write the loaded chunks into dst[ROWS][D+4].
    __device__ __forceinline__ void store(float (*dst)[kLd], int tid) const {
#pragma unroll
        for (int u = 0; u < kPerThread; ++u) {
            const int f = tid + u * NTHREADS;
            const int r = f / kChunksPerRow;
            const int c4 = f - r * kChunksPerRow;
            *reinterpret_cast<f32x4 *>(&dst[r][4 * c4]) = buf[u];
        }
    }
};

}  // namespace mg
