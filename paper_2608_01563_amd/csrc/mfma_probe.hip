// mfma_probe.hip -- sustained matrix-core throughput of the running device
// (mg_mfma_peak in mg_attn.h).
//
// The published MI355X peaks assume every SIMD issues one matrix instruction
// back to back at 2.4 GHz.  A roofline fraction read against what the chip
// actually sustains needs that figure measured: this kernel keeps NCH
// independent accumulator chains per wave busy for `iters` steps, with no
// memory traffic, eight waves per SIMD, on every CU.  Operands come from
// registers and vary per lane; the accumulators are consumed by a store that
// only a NaN result would take, so no product can be dropped.
#include "device_common.h"
#include "host_runtime.h"

namespace mg {

// Written only if a chain produced NaN; external linkage, so the stores (and
// the products behind them) cannot be dropped as dead.
__device__ float g_probe_sink;

namespace {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

constexpr int kProbeThreads = 256;

template <int KIND>
__global__ __launch_bounds__(kProbeThreads) void mfma_probe(int iters) {
    const int lane = threadIdx.x & 63;
    const float a0 = 1.f + 1e-3f * lane, b0 = 1.f - 1e-3f * lane;
    float total = 0.f;
    if (KIND == 0) {   // v_mfma_f32_16x16x4_f32: 2048 flop
        constexpr int NCH = 8;
        f32x4 acc[NCH];
#pragma unroll
        for (int c = 0; c < NCH; ++c) acc[c] = zero4();
        for (int it = 0; it < iters; ++it)
#pragma unroll
            for (int c = 0; c < NCH; ++c) acc[c] = mfma16x16x4(a0 + c, b0, acc[c]);
#pragma unroll
        for (int c = 0; c < NCH; ++c) total += acc[c][0] + acc[c][3];
    } else {           // v_mfma_f32_32x32x16_{bf16,f16}: 32768 flop
        constexpr int NCH = 4;
        f32x16 acc[NCH];
#pragma unroll
        for (int c = 0; c < NCH; ++c) acc[c] = zero16();
        if (KIND == 1) {
            bf16x8 a, b;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                a[e] = (__bf16)(a0 + e);
                b[e] = (__bf16)(b0 - e);
            }
            for (int it = 0; it < iters; ++it)
#pragma unroll
                for (int c = 0; c < NCH; ++c) acc[c] = mfma32x32x16bf16(a, b, acc[c]);
        } else {
            f16x8 a, b;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                a[e] = (_Float16)(a0 + e);
                b[e] = (_Float16)(b0 - e);
            }
            for (int it = 0; it < iters; ++it)
#pragma unroll
                for (int c = 0; c < NCH; ++c)
                    acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, acc[c], 0, 0, 0);
        }
#pragma unroll
        for (int c = 0; c < NCH; ++c) total += acc[c][0] + acc[c][15];
    }
    if (total != total) g_probe_sink = total;
}

}  // namespace
}  // namespace mg

using namespace mg;
using namespace mg::host;

extern "C" mg_status_t mg_mfma_peak(int kind, int iters, double *tflops, hipStream_t stream) {
    if (kind < 0 || kind > 2) return fail(MG_ERR_INVALID_ARGUMENT, "kind %d is not 0, 1 or 2", kind);
    if (iters < 1 || iters > (1 << 24))
        return fail(MG_ERR_INVALID_ARGUMENT, "iters %d outside [1, 2^24]", iters);
    if (tflops == nullptr) return fail(MG_ERR_INVALID_ARGUMENT, "tflops is NULL");
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return fail(MG_ERR_HIP, "device query failed");
    // eight 4-wave workgroups per CU: eight waves per SIMD
    const dim3 grid(8 * cus), block(kProbeThreads);
    const double per_mfma = kind == 0 ? 2048.0 : 32768.0;
    const double chains = kind == 0 ? 8.0 : 4.0;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    hipError_t err = hipEventCreate(&e0);
    if (err == hipSuccess) err = hipEventCreate(&e1);
    auto launch = [&](int n) {
        switch (kind) {
        case 0: mfma_probe<0><<<grid, block, 0, stream>>>(n); break;
        case 1: mfma_probe<1><<<grid, block, 0, stream>>>(n); break;
        default: mfma_probe<2><<<grid, block, 0, stream>>>(n); break;
        }
        return hipGetLastError();
    };
    if (err == hipSuccess) err = launch(iters > 8 ? iters / 8 : 1);   // warm-up
    if (err == hipSuccess) err = hipEventRecord(e0, stream);
    if (err == hipSuccess) err = launch(iters);
    if (err == hipSuccess) err = hipEventRecord(e1, stream);
    if (err == hipSuccess) err = hipEventSynchronize(e1);
    float ms = 0.f;
    if (err == hipSuccess) err = hipEventElapsedTime(&ms, e0, e1);
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
    if (err != hipSuccess) return fail(MG_ERR_HIP, "mfma probe: %s", hipGetErrorString(err));
    const double flop = (double)grid.x * (kProbeThreads / 64) * iters * chains * per_mfma;
    *tflops = flop / (ms * 1e-3) / 1e12;
    return ok();
}
