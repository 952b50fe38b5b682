// tiles_direct.h -- global->LDS tile copies that use gfx950's direct-to-LDS
// buffer loads (buffer_load_dword/dwordx4 ... lds): the loaded data is
// written to LDS by the load itself, so no staging registers and no LDS
// store instructions are needed.  Completion is tracked by the issuing
// wave's vmcnt; a barrier then makes the tile visible to the workgroup.
#pragma once

#include "device_common.h"

namespace mg {

// Chunk permutation for DirectTile (a function of the row index, values in
// [0, D/4)): chunk c of row r at c ^ (r mod 16) (d = 32: c ^ (r/2 mod 8)).
// Conflict-free for 16-byte reads of 16 consecutive rows at one chunk
// position and for 4-byte reads of rows {4g + r : g < 4} x 16 columns.
template <int D> struct RowXor {
    __host__ __device__ static constexpr int f(int row) { return D == 32 ? ((row >> 1) & 7) : (row & 15); }
};

// A [ROWS][D] f32 tile copied from global memory straight into LDS with
// 16-byte buffer loads that write LDS themselves (no staging registers, no
// LDS store instructions).  One such load moves 64 chunks of 16 bytes, one
// per lane, into 1 KB of contiguous LDS, so rows cannot be padded; instead
// the 16-byte chunks of a row are permuted (chunk c of row r is stored at
// position c ^ SW::f(r)), chosen so that the operand reads of the kernel that
// uses the tile are bank-conflict free for d = 64 and 128.
// The lane -> chunk assignment is fixed per thread, so each lane's global
// offset is computed once.  Rows at or beyond L arrive as zeros.
template <int ROWS, int D, int NW, class SW = RowXor<D>>
struct DirectTile {
    static constexpr int kCpr = D / 4;                  // chunks per row
    static constexpr int kWaveLoads = ROWS * kCpr / 64; // 1 KB loads per tile
    static constexpr int kPerWave = (kWaveLoads + NW - 1) / NW;
    // every wave issues exactly kPerWave loads per tile (else some issue fewer)
    static constexpr bool kEven = kWaveLoads % NW == 0;
    static_assert(ROWS * kCpr % 64 == 0, "tile must be a whole number of 1 KB loads");

    __host__ __device__ static constexpr int swz(int row) { return SW::f(row); }
    // Float offset of logical element (row, col) inside the tile.
    __host__ __device__ static constexpr int at(int row, int col) {
        return row * D + 4 * ((col >> 2) ^ swz(row)) + (col & 3);
    }

    int voff[kPerWave];   // byte offset, relative to the tile's first row

    __device__ __forceinline__ void init(int w, int lane) {
#pragma unroll
        for (int u = 0; u < kPerWave; ++u) {
            const int pos = (u * NW + w) * 64 + lane;   // chunk position in LDS
            const int row = pos / kCpr;
            const int chunk = (pos % kCpr) ^ swz(row);   // logical chunk stored there
            voff[u] = (row * D + 4 * chunk) * 4;
        }
    }

    // Issue this wave's share of the copy of rows [row0, row0 + ROWS) of
    // `src` into `dst` (float[ROWS * D] in LDS).  Completion is tracked by
    // the wave's vmcnt: kPerWave operations per call when kEven, at most
    // that many otherwise.  `w` is the wave index (wave-uniform).
    __device__ __forceinline__ void issue(float *dst, const float *__restrict__ src, int row0,
                                          int L, int w) const {
        const int rows = min(max(L - row0, 0), ROWS);
        const auto rsrc = buffer_rsrc(src + (size_t)row0 * D, rows * D * 4);
#pragma unroll
        for (int u = 0; u < kPerWave; ++u)
            if (kEven || u * NW + w < kWaveLoads)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rsrc, (__attribute__((address_space(3))) void *)(dst + (u * NW + w) * 256),
                    16, voff[u], 0, 0, 0);
    }
};

}  // namespace mg

namespace mg {

// A [ROWS][D] f32 tile copied row by row straight into a padded LDS array
// dst[ROWS][LD]: one wave-wide 4-byte direct-to-LDS buffer load moves 64
// consecutive floats of a row (256 bytes, fully coalesced), so every row
// keeps the padded stride and all operand reads keep immediate offsets from
// one per-lane base.  For D = 32 the upper half of the wave stays idle.  Rows
// at or beyond L arrive as zeros.  Loads are dealt to the waves round-robin.
template <int ROWS, int D, int NW, int LD>
struct RowDirectTile {
    static constexpr int kPart = D < 64 ? D : 64;       // floats per load
    static constexpr int kParts = D / kPart;            // loads per row
    static constexpr int kLoads = ROWS * kParts;        // loads per tile
    static constexpr int kPerWave = (kLoads + NW - 1) / NW;
    static constexpr bool kEven = kLoads % NW == 0;
    static_assert(D % kPart == 0 && LD >= D, "row shape");

    __device__ __forceinline__ void issue(float (*dst)[LD], const float *__restrict__ src,
                                          int row0, int L, int w, int lane) const {
        const int rows = min(max(L - row0, 0), ROWS);
        const auto rsrc = buffer_rsrc(src + (size_t)row0 * D, rows * D * 4);
#pragma unroll
        for (int u = 0; u < kPerWave; ++u) {
            const int t = u * NW + w;
            if (!kEven && t >= kLoads) break;
            const int row = t / kParts;
            const int part = t - row * kParts;
            if (kPart == 64 || lane < kPart)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rsrc, (__attribute__((address_space(3))) void *)&dst[row][kPart * part], 4,
                    (row * D + kPart * part + lane) * 4, 0, 0, 0);
        }
    }
};

}  // namespace mg
