// tiles_bf16.h -- LDS layout of bf16 row tiles and the LDS reads that feed
// bf16 MFMA operands (the tiles themselves arrive by the direct-to-LDS row
// loads of tiles_direct.h).
//
// A streamed tile is stored row-major only.  Products that contract over the
// head dimension read 8 consecutive d values of a row (one 16-byte read);
// products that contract over the streamed rows read 4 consecutive rows of
// one column with gfx950's 16-bit transpose read (ds_read_b64_tr_b16): in
// each 16-lane group, lane i receives element i%4 of the 8-byte chunks that
// lanes i/4, i/4+4, i/4+8 and i/4+12 address, so when lane j addresses row
// j/4, columns 4*(j%4)..+3 of a 4 x 16 block, lane i gets rows 0..3 of
// column i.  No transposed copy of any tile is needed.
//
// Row stride (u16): the smallest padding for which both the 16-row 16-byte
// reads and the 4-row transpose reads of a 16-lane group hit 16 distinct
// 4-bank groups: d=32 -> 56, d=64 -> 72, d=128 -> 152.  Rows at or beyond L
// arrive as zeros.
#pragma once

#include "device_common.h"

namespace mg {

template <int D> struct Bf16Ld;
template <> struct Bf16Ld<32> { static constexpr int value = 56; };
template <> struct Bf16Ld<64> { static constexpr int value = 72; };
template <> struct Bf16Ld<128> { static constexpr int value = 152; };

// Row stride (u16) of a streamed tile that is only ever read by 4-row
// transpose reads feeding 32x32x16 products (the V tile of the forward): a
// stride of 0 bytes modulo 64 serves them without conflicts (the strides
// above, which also serve 16-byte reads of 32 rows, cost such a read twice
// the minimum).
template <int D> struct Bf16LdTr;
template <> struct Bf16LdTr<32> { static constexpr int value = 32; };
template <> struct Bf16LdTr<64> { static constexpr int value = 96; };
template <> struct Bf16LdTr<128> { static constexpr int value = 160; };

// Row stride (u16) of the streamed tiles of the 16-key dK/dV kernel, whose
// reads are 16 rows x 4 chunks (16-byte, 16x16x32 operands) and 4-row
// transpose reads: a stride of 32 bytes modulo 64 serves both without
// conflicts (the strides above serve the 32-row reads of the 32x32x16
// kernels and conflict here).
template <int D> struct Bf16LdKV;
template <> struct Bf16LdKV<32> { static constexpr int value = 48; };
template <> struct Bf16LdKV<64> { static constexpr int value = 80; };
template <> struct Bf16LdKV<128> { static constexpr int value = 144; };

// A [ROWS][D] bf16 tile stored as D/W column blocks of [ROWS][W] (rows of
// 2W bytes), the 16-byte chunks of row r permuted by j -> j ^ swz(r) with
// swz(r) = ((r >> SS) & SM) * SK.  It arrives by 16-byte direct-to-LDS
// loads: one load fills 1 KB, 512/W rows of one block, from 2W-byte pieces
// of as many global rows; a compute unit moves two to three times the bytes
// per clock this way than with the 4-byte row loads of tiles_direct.h (more
// with longer pieces).  The swizzle spreads the rows that one read
// instruction touches over all 64 banks; the kernels pick, per tile, one
// under which each of their read patterns runs at the LDS's minimum cycles
// per instruction (measured: 16-byte reads of 16 rows x 4 chunks or 32 rows
// x 2 chunks, 4-row transpose reads of 16 rows x 32 bytes or 8 rows x 64
// bytes).  The chunk a swizzle moves depends only on bits of the row that a
// lane's read pattern fixes, so every read is one of a few per-lane bases
// plus a compile-time offset, and a load's lane offsets are the same for
// every load of the tile.  Rows at or beyond L arrive as zeros.
template <int ROWS, int D, int NW, int W, int SS, int SM, int SK>
struct Bf16Tile {
    static constexpr int kRowsPerLoad = 512 / W;
    static_assert((W == 32 || W == 64) && D % W == 0 && ROWS % kRowsPerLoad == 0, "tile shape");
    static_assert(SM * SK < W / 8 && (kRowsPerLoad >> SS) % (SM + 1) == 0,
                  "the swizzle stays inside a row and repeats every load");
    static constexpr int kBlock = ROWS * W;     // u16 per column block
    static constexpr int kSize = ROWS * D;      // u16 per tile
    static constexpr int kLoads = kSize / 512;  // 1 KB loads per tile
    static constexpr int kPerWave = kLoads / NW;
    static_assert(kLoads % NW == 0, "every wave issues the same number of loads");

    __host__ __device__ static constexpr int swz(int r) { return ((r >> SS) & SM) * SK; }
    // u16 offset of element (r, e) in the tile
    __host__ __device__ static constexpr int at(int r, int e) {
        return (e / W) * kBlock + r * W + 8 * (((e % W) >> 3) ^ swz(r)) + (e & 7);
    }

    int voff;   // this lane's byte offset within the rows of one load

    __device__ __forceinline__ void init(int lane) {
        // LDS chunk `lane` of a load is row lane / (W/8) of the load, chunk
        // position lane % (W/8), which holds logical chunk position ^ swz(row)
        const int r = lane / (W / 8), j = lane % (W / 8);
        voff = r * D * 2 + 16 * (j ^ swz(r));
    }

    // This wave's share of rows [row0, row0 + ROWS) of src (row-major, D
    // bf16 per row) into dst (kSize u16 of LDS); kPerWave loads, tracked by
    // the wave's vmcnt.  A load's row and block offset goes into the vector
    // offset, the one the buffer's range check sees.
    __device__ __forceinline__ void issue(uint16_t *dst, const uint16_t *__restrict__ src,
                                          int row0, int L, int w) const {
        const int rows = min(max(L - row0, 0), ROWS);
        const auto rsrc = buffer_rsrc(src + (size_t)row0 * D, rows * D * 2);
#pragma unroll
        for (int uu = 0; uu < kPerWave; ++uu) {
            const int u = uu * NW + w;
            const int r0 = (kRowsPerLoad * u) % ROWS, blk = (kRowsPerLoad * u) / ROWS;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rsrc, (__attribute__((address_space(3))) void *)(dst + 512 * u), 16,
                voff + r0 * D * 2 + 2 * W * blk, 0, 0, 0);
        }
    }
};

typedef short s16x4 __attribute__((ext_vector_type(4)));

// Transpose read (see above): `p` is this lane's 8-byte chunk address.
__device__ __forceinline__ s16x4 lds_read_tr16(const uint16_t *p) {
    typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)p);
}

// A operand of a product contracting over the rows of row-major tile X:
// positions 0..3 are rows r0..r0+3 and 4..7 rows r1..r1+3 of column col0 + i
// (i = lane%16); `jr`, `jc` are this lane's row / column offsets in its
// 4 x 16 transpose block (lane%16 / 4 and 4*(lane%4)).
template <int LD>
__device__ __forceinline__ bf16x8 load_tr_pair(const uint16_t (*X)[LD], int r0, int r1,
                                               int col0, int jr, int jc) {
    const s16x4 lo = lds_read_tr16(&X[r0 + jr][col0 + jc]);
    const s16x4 hi = lds_read_tr16(&X[r1 + jr][col0 + jc]);
    return __builtin_bit_cast(bf16x8, (short __attribute__((ext_vector_type(8)))){
        lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]});
}

// A operand from two transpose reads at lane addresses `lo` and `hi`
// (positions 0..3 and 4..7).
__device__ __forceinline__ bf16x8 load_tr_pair_at(const uint16_t *lo, const uint16_t *hi) {
    const s16x4 a = lds_read_tr16(lo);
    const s16x4 b = lds_read_tr16(hi);
    return __builtin_bit_cast(bf16x8, (short __attribute__((ext_vector_type(8)))){
        a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]});
}

// Eight bf16 from 16 bytes of LDS or global memory.
__device__ __forceinline__ bf16x8 load_bf16x8(const uint16_t *p) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(p));
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
