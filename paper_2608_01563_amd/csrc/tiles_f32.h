// tiles_f32.h -- register-staged global->LDS copies of f32 row tiles.
//
// A tile is `ROWS` consecutive rows of one head's [L][D] matrix.  Every
// thread of the workgroup moves `kPerThread` 16-byte chunks: global reads are
// fully coalesced (consecutive threads read consecutive 16-byte chunks of a
// row) and land in a row-padded LDS array with stride D+4 floats, which keeps
// both the row-fragment reads (16 lanes on 16 rows, 16 bytes each) and the
// column reads (16 lanes along one row, 4 rows apart) free of bank conflicts.
//
// The reads are raw buffer loads through a descriptor that covers exactly the
// tile's rows below L: a chunk past the end reads as zero without touching
// memory, so the tail tile needs neither a branch nor a per-lane bounds test,
// and the only per-lane address is the thread's fixed byte offset in the tile.
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

    // Issue the global loads of rows [row0, row0+ROWS) of `src` (one head);
    // rows at or beyond L read as zero.  Chunk f of the tile sits at byte
    // 16*f from the tile's first row, because tile rows are contiguous.
    __device__ __forceinline__ void load(const float *__restrict__ src, int row0, int L,
                                         int tid) {
        const int rows = min(max(L - row0, 0), ROWS);
        const auto rsrc = buffer_rsrc(src + (size_t)row0 * D, rows * D * 4);
#pragma unroll
        for (int u = 0; u < kPerThread; ++u)
            buf[u] = buffer_load_f32x4(rsrc, 16 * (tid + u * NTHREADS));
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
