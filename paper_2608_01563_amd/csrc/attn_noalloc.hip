// attn_noalloc.hip -- mg_attn_bwd_noalloc: the attention backward with its
// workspace in a fixed device array of the library instead of caller
// memory, for callers that cannot allocate (graph capture, serving loops).
//
// The array, `scratch`, is a file-scope device variable: the runtime places
// one copy on every device that loads this code object and keeps it until
// the process ends.  Host code never uses its name as an address (on the
// host the name is only a stand-in for the symbol); the device address is
// looked up once per device with hipGetSymbolAddress and kept.  The kernels
// and their launch sequence are those of mg_attn_bwd_cross; only where the
// workspace lives differs.  Nothing in the workspace needs to start at zero:
// D and every partial are written before they are read in the same call.
#include <hip/hip_runtime.h>

#include <mutex>

#include "attn_bwd.h"
#include "host_runtime.h"
#include "mg_attn.h"

namespace {

using mg::host::fail;

static_assert(MG_ATTN_NOALLOC_SCRATCH_BYTES % 256 == 0, "scratch size");
static __device__ __align__(256) unsigned char scratch[MG_ATTN_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void *g_scratch[kMaxDevices];   // device address of `scratch`, per device

// The scratch array's address on the current device (looked up on the
// first call there, with that device current).
mg_status_t scratch_address(void **out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();
        return fail(MG_ERR_HIP, "hipGetDevice failed");
    }
    if (dev < 0 || dev >= kMaxDevices)
        return fail(MG_ERR_UNSUPPORTED, "device %d beyond the %d the scratch table holds", dev,
                    kMaxDevices);
    std::lock_guard<std::mutex> g(g_mu);
    if (g_scratch[dev] == nullptr) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || p == nullptr) {
            (void)hipGetLastError();
            return fail(MG_ERR_HIP, "hipGetSymbolAddress of the scratch array failed: %s",
                        hipGetErrorString(e));
        }
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return MG_OK;
}

}  // namespace

extern "C" mg_status_t mg_attn_bwd_noalloc(const void *Q, const void *K, const void *V,
                                           const void *O, const float *LSE, const void *dO,
                                           void *dQ, void *dK, void *dV,
                                           const int32_t *key_len, int B, int H, int Lq,
                                           int Lk, int d, int causal, float scale,
                                           mg_contract_t contract, hipStream_t stream) {
    MG_TRY(mg::attn_bwd_check_shape(B, H, Lq, Lk, d, scale, contract));
    constexpr size_t cap = MG_ATTN_NOALLOC_SCRATCH_BYTES;
    // the caller-workspace layout when it fits, else D alone (separate dQ pass)
    size_t limit = mg::attn_bwd_partial_limit();
    if (mg::attn_bwd_workspace(B, H, Lq, Lk, d, causal, contract, limit) > cap) limit = 0;
    const size_t need = mg::attn_bwd_workspace(B, H, Lq, Lk, d, causal, contract, limit);
    if (need > cap)
        return fail(MG_ERR_WORKSPACE,
                    "B*H*Lq = %lld query rows need %zu bytes of workspace; the static "
                    "scratch holds %zu",
                    (long long)B * H * Lq, need, cap);
    MG_TRY(mg::attn_bwd_check_args(Q, K, V, O, LSE, dO, dQ, dK, dV, key_len, nullptr));
    void *ws = nullptr;
    MG_TRY(scratch_address(&ws));
    return mg::attn_bwd_enqueue(Q, K, V, O, LSE, dO, dQ, dK, dV, key_len, B, H, Lq, Lk, d,
                                causal, scale, contract, ws, limit, stream);
}
