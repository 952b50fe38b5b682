// lds_probe.hip -- LDS read cost of the attention kernels' access patterns
// (mg_lds_probe in mg_attn.h).
//
// The kernels choose the row stride of every LDS tile so that their operand
// reads are free of bank conflicts.  Which strides achieve that for a given
// lane -> address pattern is a property of the LDS hardware (how it groups
// the lanes of a 16-byte or transposed read into bank cycles), so it is
// measured rather than derived: this kernel issues one pattern's reads back
// to back from every wave of two workgroups per CU and reports the LDS clocks
// one read instruction costs a CU.  The patterns are the exact lane maps the
// kernels use, applied to rows of `row_bytes` bytes.
#include <vector>

#include "device_common.h"
#include "host_runtime.h"
#include "tiles_bf16.h"
#include "tiles_direct.h"

namespace mg {

// Written only when the reads produced a value no fill can produce; external
// linkage, so the reads cannot be dropped as dead.
__device__ unsigned g_lds_probe_sink;

constexpr int kProbeMaxWaves = 4096;   // two 4-wave workgroups on up to 512 CUs
// Clock counts of the probe's waves (a fixed array: the call allocates nothing).
__device__ unsigned long long g_lds_probe_cycles[kProbeMaxWaves];

namespace {

constexpr int kProbeWgThreads = 256;
constexpr int kProbeWords = 16384;   // 64 KB of LDS per workgroup
constexpr int kReadsPerStep = 8;

// The bf16 kernels' tile layouts ([64 rows][128 columns] in column blocks),
// and the same blocks without the chunk swizzle.
using KvTile = Bf16Tile<64, 128, 4, 32, 1, 3, 1>;      // dK/dV: Q, dO
using RowTile = Bf16Tile<64, 128, 4, 32, 2, 3, 1>;     // forward K, dQ K and V
using TrTile = Bf16Tile<64, 128, 4, 64, 1, 1, 4>;      // forward V
using Plain32 = Bf16Tile<64, 128, 4, 32, 0, 0, 0>;
using Plain64 = Bf16Tile<64, 128, 4, 64, 0, 0, 0>;
// The strict f32 forward's K and V tiles at d = 64 (rows of 256 bytes, the
// 16-byte chunks of row r permuted by j -> j ^ (r % 16)).
using F32FwdTile = DirectTile<64, 64, 4>;

// Row and column that lane l reads in the block-layout patterns (7..16).
__host__ __device__ inline int block_row(int p, int l) {
    switch ((p - 7) % 5) {
    case 0: return l & 15;                                 // 16 rows x 4 chunks
    case 1: return 4 * (l >> 4) + ((l & 15) >> 2);          // 16-row transpose
    case 2: return l & 31;                                 // 32 rows x 2 chunks
    default: return 4 * (l >> 5) + ((l & 15) >> 2);         // 32x32 transpose
    }
}
__host__ __device__ inline int block_col(int p, int l) {
    switch ((p - 7) % 5) {
    case 0: return 8 * (l >> 4);
    case 1: return 4 * (l & 3);
    case 2: return 8 * (l >> 5);
    default: return 16 * ((l >> 4) & 1) + 4 * (l & 3);
    }
}

// Byte offset of lane `l`'s read in pattern `p` for rows of `rb` bytes.
__host__ __device__ inline int probe_offset(int p, int l, int rb) {
    const int il = l & 15, g = l >> 4, jr = il >> 2, jc = 4 * (il & 3);
    if (p == 17) return 4 * F32FwdTile::at(il, 16 * g);     // K: row l%16, group l/16
    if (p == 18) return 4 * F32FwdTile::at(4 * g, il);      // V: row 4(l/16), word l%16
    if (p >= 7) {
        const int r = block_row(p, l), e = block_col(p, l);
        switch (p) {
        case 7: case 8: return 2 * KvTile::at(r, e);
        case 9: case 10: return 2 * RowTile::at(r, e);
        case 11: return 2 * TrTile::at(r, e);
        case 16: return 2 * Plain64::at(r, e);
        default: return 2 * Plain32::at(r, e);
        }
    }
    switch (p) {
    case 0: return il * rb + 16 * g;                               // 16 rows x 4 adjacent chunks
    case 1: return il * rb + 64 * g;                               // 16 rows x 4 chunks 64 B apart
    case 2: return (l & 31) * rb + 16 * (l >> 5);                  // 32 rows x 2 chunks
    case 3: return (4 * g + jr) * rb + 2 * jc;                     // transpose, 16-key dK/dV
    case 4: return (4 * (l >> 5) + jr) * rb + 2 * (16 * ((l >> 4) & 1) + jc);   // transpose, 32x32
    case 5: return 16 * l;                                         // contiguous 1 KB
    case 6: return (4 * g) * rb + 4 * il;                          // 4 rows x 16 words
    default: return 0;
    }
}

// 0: 16-byte reads, 1: 8-byte transpose reads, 2: 4-byte reads
__host__ __device__ constexpr int probe_kind(int p) {
    return (p == 3 || p == 4 || p == 8 || p == 10 || p == 11 || p == 13 || p == 15 || p == 16)
               ? 1
               : ((p == 6 || p == 18) ? 2 : 0);
}

// Row length (bytes) of the fixed-layout patterns' tiles (7..18).
__host__ __device__ constexpr int block_row_bytes(int p) {
    return p >= 17 ? 256 : ((p == 11 || p == 16) ? 128 : 64);
}

typedef unsigned u32x2 __attribute__((ext_vector_type(2)));

template <int KIND>
__global__ __launch_bounds__(kProbeWgThreads) void lds_probe(int pattern, int rb, int iters) {
    __shared__ __attribute__((aligned(16))) unsigned buf[kProbeWords];
    for (int i = threadIdx.x; i < kProbeWords; i += kProbeWgThreads) buf[i] = i * 2654435761u;
    __syncthreads();
    const int lane = threadIdx.x & 63;
    const unsigned base = (unsigned)(uintptr_t)(&buf[0]) + probe_offset(pattern, lane, rb);
    unsigned acc = 0;
    const unsigned long long t0 = clock64();
    for (int it = 0; it < iters; ++it) {
        // 4 KB steps leave every bank mapping unchanged; the eight reads of a
        // step sit 8 KB and 1 KB apart (also mapping-neutral)
        const unsigned a = base + ((it & 3) << 12);
        if (KIND == 0) {
            u32x4 v0, v1, v2, v3, v4, v5, v6, v7;
            asm volatile(
                "ds_read_b128 %0, %8 offset:0\n ds_read_b128 %1, %8 offset:8192\n"
                "ds_read_b128 %2, %8 offset:16384\n ds_read_b128 %3, %8 offset:24576\n"
                "ds_read_b128 %4, %8 offset:1024\n ds_read_b128 %5, %8 offset:9216\n"
                "ds_read_b128 %6, %8 offset:17408\n ds_read_b128 %7, %8 offset:25600\n"
                "s_waitcnt lgkmcnt(0)"
                : "=v"(v0), "=v"(v1), "=v"(v2), "=v"(v3), "=v"(v4), "=v"(v5), "=v"(v6), "=v"(v7)
                : "v"(a));
            acc ^= v0.x ^ v1.y ^ v2.z ^ v3.w ^ v4.x ^ v5.y ^ v6.z ^ v7.w;
        } else if (KIND == 1) {
            u32x2 v0, v1, v2, v3, v4, v5, v6, v7;
            asm volatile(
                "ds_read_b64_tr_b16 %0, %8 offset:0\n ds_read_b64_tr_b16 %1, %8 offset:8192\n"
                "ds_read_b64_tr_b16 %2, %8 offset:16384\n ds_read_b64_tr_b16 %3, %8 offset:24576\n"
                "ds_read_b64_tr_b16 %4, %8 offset:1024\n ds_read_b64_tr_b16 %5, %8 offset:9216\n"
                "ds_read_b64_tr_b16 %6, %8 offset:17408\n ds_read_b64_tr_b16 %7, %8 offset:25600\n"
                "s_waitcnt lgkmcnt(0)"
                : "=v"(v0), "=v"(v1), "=v"(v2), "=v"(v3), "=v"(v4), "=v"(v5), "=v"(v6), "=v"(v7)
                : "v"(a));
            acc ^= v0.x ^ v1.y ^ v2.x ^ v3.y ^ v4.x ^ v5.y ^ v6.x ^ v7.y;
        } else {
            unsigned v0, v1, v2, v3, v4, v5, v6, v7;
            asm volatile(
                "ds_read_b32 %0, %8 offset:0\n ds_read_b32 %1, %8 offset:8192\n"
                "ds_read_b32 %2, %8 offset:16384\n ds_read_b32 %3, %8 offset:24576\n"
                "ds_read_b32 %4, %8 offset:1024\n ds_read_b32 %5, %8 offset:9216\n"
                "ds_read_b32 %6, %8 offset:17408\n ds_read_b32 %7, %8 offset:25600\n"
                "s_waitcnt lgkmcnt(0)"
                : "=v"(v0), "=v"(v1), "=v"(v2), "=v"(v3), "=v"(v4), "=v"(v5), "=v"(v6), "=v"(v7)
                : "v"(a));
            acc ^= v0 ^ v1 ^ v2 ^ v3 ^ v4 ^ v5 ^ v6 ^ v7;
        }
    }
    const unsigned long long t1 = clock64();
    if (lane == 0)
        g_lds_probe_cycles[blockIdx.x * (kProbeWgThreads / 64) + (threadIdx.x >> 6)] = t1 - t0;
    if (acc == 0x9e3779b9u) g_lds_probe_sink = acc;
}

// Largest byte offset any lane of any pattern reads, for row strides up to
// `rb`: base offset + 3 * 4 KB + 25600 + 16 must stay inside the 64 KB array.
constexpr int kMaxRowBytes = 480;
static_assert(31 * kMaxRowBytes + 16 + 3 * 4096 + 25600 + 16 <= 4 * kProbeWords,
              "probe reads must stay inside the LDS array");
// The block-layout tiles are 16 KB, the f32 forward tile 16 KB.
static_assert(2 * KvTile::kSize + 3 * 4096 + 25600 <= 4 * kProbeWords &&
                  4 * 64 * 64 + 3 * 4096 + 25600 <= 4 * kProbeWords,
              "fixed-layout reads must stay inside the LDS array");

}  // namespace
}  // namespace mg

using namespace mg;
using namespace mg::host;

extern "C" mg_status_t mg_lds_probe(int pattern, int row_bytes, int iters, double *clocks,
                                    hipStream_t stream) {
    if (pattern < 0 || pattern > 18)
        return fail(MG_ERR_INVALID_ARGUMENT, "pattern %d outside [0, 18]", pattern);
    if (pattern >= 7 && row_bytes != block_row_bytes(pattern))
        return fail(MG_ERR_INVALID_ARGUMENT, "pattern %d reads %d-byte tile rows, not %d",
                    pattern, block_row_bytes(pattern), row_bytes);
    if (row_bytes < 16 || row_bytes > kMaxRowBytes || row_bytes % 16 != 0)
        return fail(MG_ERR_INVALID_ARGUMENT,
                    "row_bytes %d must be a multiple of 16 in [16, %d]", row_bytes, kMaxRowBytes);
    if (iters < 1 || iters > (1 << 20))
        return fail(MG_ERR_INVALID_ARGUMENT, "iters %d outside [1, 2^20]", iters);
    if (clocks == nullptr) return fail(MG_ERR_INVALID_ARGUMENT, "clocks is NULL");
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return fail(MG_ERR_HIP, "device query failed");
    // two 4-wave workgroups per CU: eight waves share each CU's LDS
    const int grid = 2 * cus;
    const int waves = grid * (kProbeWgThreads / 64);
    if (waves > kProbeMaxWaves) return fail(MG_ERR_UNSUPPORTED, "%d CUs: too many for the probe", cus);
    auto launch = [&](int n) {
        switch (probe_kind(pattern)) {
        case 0: lds_probe<0><<<grid, kProbeWgThreads, 0, stream>>>(pattern, row_bytes, n); break;
        case 1: lds_probe<1><<<grid, kProbeWgThreads, 0, stream>>>(pattern, row_bytes, n); break;
        default: lds_probe<2><<<grid, kProbeWgThreads, 0, stream>>>(pattern, row_bytes, n); break;
        }
        return hipGetLastError();
    };
    hipError_t err = launch(iters > 8 ? iters / 8 : 1);   // warm-up
    if (err == hipSuccess) err = launch(iters);
    std::vector<unsigned long long> host(waves);
    if (err == hipSuccess)
        err = hipMemcpyFromSymbolAsync(host.data(), HIP_SYMBOL(g_lds_probe_cycles),
                                       waves * sizeof(unsigned long long), 0,
                                       hipMemcpyDeviceToHost, stream);
    if (err == hipSuccess) err = hipStreamSynchronize(stream);
    if (err != hipSuccess) return fail(MG_ERR_HIP, "lds probe: %s", hipGetErrorString(err));
    double mean = 0.0;
    for (unsigned long long c : host) mean += (double)c;
    mean /= waves;
    // waves of a CU share its LDS: clocks per read instruction per CU
    *clocks = mean / ((double)kReadsPerStep * iters * 2 * (kProbeWgThreads / 64));
    return ok();
}
