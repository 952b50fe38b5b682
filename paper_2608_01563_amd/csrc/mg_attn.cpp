// mg_attn.cpp -- C ABI of the attention library: argument validation,
// selection of the kernel instance, and launch on the caller's stream.
//
// Validation runs entirely on the host before anything is enqueued, so a
// rejected call has no effect on the device.  The kernel instance and its
// launch geometry are chosen together by the per-kernel launchers.
#include "mg_attn.h"

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <string>

#include "attn_bwd.h"
#include "host_runtime.h"
#include "launch.h"

namespace {

using mg::host::fail;
using mg::host::ok;
using mg::host::round256;
using mg::host::run_kernel;

constexpr int64_t kMaxElems = INT32_MAX;

mg_status_t check_shape(int B, int H, int Lq, int Lk, int d, float scale,
                        mg_contract_t contract) {
    if (contract != MG_CONTRACT_STRICT_F32 && contract != MG_CONTRACT_FAST_BF16 &&
        contract != MG_CONTRACT_ACCELERATED)
        return fail(MG_ERR_INVALID_ARGUMENT, "unknown contract %d", (int)contract);
    if (B < 1 || H < 1 || Lq < 1 || Lk < 1 || d < 1)
        return fail(MG_ERR_INVALID_ARGUMENT,
                    "sizes must be >= 1 (B=%d H=%d Lq=%d Lk=%d d=%d)", B, H, Lq, Lk, d);
    if (d != 32 && d != 64 && d != 128)
        return fail(MG_ERR_UNSUPPORTED, "head dimension d=%d not in {32, 64, 128}", d);
    const int64_t n = (int64_t)B * H * std::max(Lq, Lk) * d;
    if (n > kMaxElems)
        return fail(MG_ERR_INVALID_ARGUMENT, "B*H*max(Lq,Lk)*d = %lld exceeds 2^31-1",
                    (long long)n);
    if (!std::isfinite(scale)) return fail(MG_ERR_INVALID_ARGUMENT, "scale is not finite");
    return MG_OK;
}

mg_status_t check_tensors(std::initializer_list<mg::host::NamedPtr> ptrs) {
    return mg::host::check_device_ptrs(ptrs, 16);
}

// key_len's alignment is a host-only check, so it runs with the other
// pointers' null and alignment checks, before any pointer reaches the
// runtime's device-memory query.
mg_status_t check_key_len_alignment(const int32_t *key_len) {
    if (key_len != nullptr && reinterpret_cast<uintptr_t>(key_len) % 4 != 0)
        return fail(MG_ERR_MISALIGNED, "key_len is not 4-byte aligned");
    return MG_OK;
}

mg_status_t check_key_len(const int32_t *key_len) {
    return mg::host::check_optional_device_ptr(key_len, "key_len", 4);
}

const char *kernel_name(const char *stage, mg_contract_t c, int d) {
    const char *suffix = c == MG_CONTRACT_STRICT_F32 ? "f32"
                         : c == MG_CONTRACT_FAST_BF16 ? "bf16" : "accel";
    char buf[96];
    snprintf(buf, sizeof buf, "%s_%s_d%d", stage, suffix, d);
    return mg::host::intern_name(buf);
}

// The accelerated contract's backward is the strict-f32 backward (its
// tensors are f32 and its backward matrices stay f32).
mg_contract_t backward_contract(mg_contract_t c) {
    return c == MG_CONTRACT_ACCELERATED ? MG_CONTRACT_STRICT_F32 : c;
}

// Strict f32 with d <= 64 fuses dQ into the key-stationary kernel when its
// per-key-tile partials fit under this many bytes; otherwise (and for bf16)
// a separate query-stationary dQ kernel recomputes what it needs.
constexpr size_t kFusedPartialLimit = size_t(1) << 30;

size_t dq_partial_bytes(int B, int H, int Lq, int Lk, int d, int causal) {
    const mg::AttnProblem p{B, H, Lq, Lk, d, causal ? 1 : 0, 1.0f, nullptr};
    const int kr = mg::fused_dq_key_rows(p);
    return (size_t)((Lk + kr - 1) / kr) * B * H * Lq * d * sizeof(float);
}

bool use_fused_dq(int B, int H, int Lq, int Lk, int d, int causal, mg_contract_t contract,
                  size_t partial_limit) {
    return contract == MG_CONTRACT_STRICT_F32 && d <= 64 &&
           dq_partial_bytes(B, H, Lq, Lk, d, causal) <= partial_limit;
}

// dK/dV partials of a fused backward whose query tiles are split (zero
// bytes with one split).
size_t dkdv_partial_bytes(int B, int H, int Lq, int Lk, int d, int causal) {
    const mg::AttnProblem p{B, H, Lq, Lk, d, causal ? 1 : 0, 1.0f, nullptr};
    const int ns = mg::fused_dq_query_splits(p);
    return ns > 1 ? (size_t)2 * ns * B * H * Lk * d * sizeof(float) : 0;
}

}  // namespace

namespace mg {

// Layout: D (f32 per query row) first; when fused, the dQ partials, then
// (256-byte aligned) the dK/dV partials of a split backward.
size_t attn_bwd_workspace(int B, int H, int Lq, int Lk, int d, int causal,
                          mg_contract_t contract, size_t partial_limit) {
    contract = backward_contract(contract);
    size_t n = round256((size_t)B * H * Lq * sizeof(float));
    if (use_fused_dq(B, H, Lq, Lk, d, causal, contract, partial_limit)) {
        n += dq_partial_bytes(B, H, Lq, Lk, d, causal);
        const size_t kv = dkdv_partial_bytes(B, H, Lq, Lk, d, causal);
        if (kv > 0) n = round256(n) + kv;
    }
    return n;
}

size_t attn_bwd_partial_limit() { return kFusedPartialLimit; }

mg_status_t attn_bwd_check_args(const void *Q, const void *K, const void *V, const void *O,
                                const float *LSE, const void *dO, void *dQ, void *dK,
                                void *dV, const int32_t *key_len, const void *workspace) {
    MG_TRY(check_key_len_alignment(key_len));
    if (workspace != nullptr)
        MG_TRY(check_tensors({{Q, "Q"}, {K, "K"}, {V, "V"}, {O, "O"}, {LSE, "LSE"},
                              {dO, "dO"}, {dQ, "dQ"}, {dK, "dK"}, {dV, "dV"},
                              {workspace, "workspace"}}));
    else
        MG_TRY(check_tensors({{Q, "Q"}, {K, "K"}, {V, "V"}, {O, "O"}, {LSE, "LSE"},
                              {dO, "dO"}, {dQ, "dQ"}, {dK, "dK"}, {dV, "dV"}}));
    return check_key_len(key_len);
}

mg_status_t attn_bwd_check_shape(int B, int H, int Lq, int Lk, int d, float scale,
                                 mg_contract_t contract) {
    return check_shape(B, H, Lq, Lk, d, scale, contract);
}

mg_status_t attn_bwd_enqueue(const void *Q, const void *K, const void *V, const void *O,
                             const float *LSE, const void *dO, void *dQ, void *dK, void *dV,
                             const int32_t *key_len, int B, int H, int Lq, int Lk, int d,
                             int causal, float scale, mg_contract_t contract, void *workspace,
                             size_t partial_limit, hipStream_t stream) {
    const mg::AttnProblem p{B, H, Lq, Lk, d, causal ? 1 : 0, scale, key_len};
    float *Dws = (float *)workspace;
    contract = backward_contract(contract);
    if (contract == MG_CONTRACT_STRICT_F32) {
        const float *q = (const float *)Q, *k = (const float *)K, *v = (const float *)V;
        const float *o = (const float *)O, *go = (const float *)dO;
        const bool fused = use_fused_dq(B, H, Lq, Lk, d, causal, contract, partial_limit);
        // small fused grids compute D in the kernel itself
        if (!fused || !mg::fused_local_d(p))
            MG_TRY(run_kernel(kernel_name("attn_rowdot", contract, d), stream,
                              [&] { return mg::launch_bwd_rowdot_f32(p, o, go, Dws, stream); }));
        if (fused) {
            char *base = (char *)workspace;
            float *dQp = (float *)(base + round256((size_t)B * H * Lq * sizeof(float)));
            float *dKVp = dkdv_partial_bytes(B, H, Lq, Lk, d, causal) == 0 ? nullptr
                : (float *)((char *)dQp + round256(dq_partial_bytes(B, H, Lq, Lk, d, causal)));
            // one key tile and no split: the kernel writes dQ itself
            const bool direct = mg::fused_direct_dq(p);
            MG_TRY(run_kernel(kernel_name("attn_dkdvq", contract, d), stream, [&] {
                return mg::launch_bwd_dkdvq_f32(p, q, k, v, o, go, LSE, Dws, (float *)dK,
                                                (float *)dV, direct ? (float *)dQ : dQp, dKVp,
                                                stream);
            }));
            if (dKVp != nullptr)
                MG_TRY(run_kernel(kernel_name("attn_bwdreduce", contract, d), stream, [&] {
                    return mg::launch_bwd_reduce_f32(p, dKVp, (float *)dK, (float *)dV, dQp,
                                                     (float *)dQ, stream);
                }));
            else if (!direct)
                MG_TRY(run_kernel(kernel_name("attn_dqreduce", contract, d), stream, [&] {
                    return mg::launch_bwd_dq_reduce_f32(p, dQp, (float *)dQ, stream);
                }));
            return ok();
        }
        MG_TRY(run_kernel(kernel_name("attn_dkdv", contract, d), stream, [&] {
            return mg::launch_bwd_dkdv_f32(p, q, k, v, go, LSE, Dws, (float *)dK, (float *)dV,
                                           stream);
        }));
        MG_TRY(run_kernel(kernel_name("attn_dq", contract, d), stream, [&] {
            return mg::launch_bwd_dq_f32(p, q, k, v, go, LSE, Dws, (float *)dQ, stream);
        }));
    } else {
        const uint16_t *q = (const uint16_t *)Q, *k = (const uint16_t *)K,
                       *v = (const uint16_t *)V;
        const uint16_t *o = (const uint16_t *)O, *go = (const uint16_t *)dO;
        // The dQ kernel computes D for its query rows on the way (it holds
        // each row's dO already) and writes it for the dK/dV kernel.
        MG_TRY(run_kernel(kernel_name("attn_dq", contract, d), stream, [&] {
            return mg::launch_bwd_dq_bf16(p, q, k, v, o, go, LSE, Dws, (uint16_t *)dQ, stream);
        }));
        MG_TRY(run_kernel(kernel_name("attn_dkdv", contract, d), stream, [&] {
            return mg::launch_bwd_dkdv_bf16(p, q, k, v, go, LSE, Dws, (uint16_t *)dK,
                                            (uint16_t *)dV, stream);
        }));
    }
    return ok();
}

}  // namespace mg

extern "C" {

mg_status_t mg_attn_fwd_cross(const void *Q, const void *K, const void *V, void *O, float *LSE,
                              const int32_t *key_len, int B, int H, int Lq, int Lk, int d,
                              int causal, float scale, mg_contract_t contract,
                              hipStream_t stream) {
    MG_TRY(check_shape(B, H, Lq, Lk, d, scale, contract));
    MG_TRY(check_key_len_alignment(key_len));
    MG_TRY(check_tensors({{Q, "Q"}, {K, "K"}, {V, "V"}, {O, "O"}, {LSE, "LSE"}}));
    MG_TRY(check_key_len(key_len));
    const mg::AttnProblem p{B, H, Lq, Lk, d, causal ? 1 : 0, scale, key_len};
    if (contract == MG_CONTRACT_STRICT_F32) {
        MG_TRY(run_kernel(kernel_name("attn_fwd", contract, d), stream, [&] {
            return mg::launch_fwd_f32(p, (const float *)Q, (const float *)K, (const float *)V,
                                      (float *)O, LSE, stream);
        }));
    } else if (contract == MG_CONTRACT_ACCELERATED) {
        MG_TRY(run_kernel(kernel_name("attn_fwd", contract, d), stream, [&] {
            return mg::launch_fwd_accel(p, (const float *)Q, (const float *)K, (const float *)V,
                                        (float *)O, LSE, stream);
        }));
    } else {
        MG_TRY(run_kernel(kernel_name("attn_fwd", contract, d), stream, [&] {
            return mg::launch_fwd_bf16(p, (const uint16_t *)Q, (const uint16_t *)K,
                                       (const uint16_t *)V, (uint16_t *)O, LSE, stream);
        }));
    }
    return ok();
}

size_t mg_attn_bwd_cross_workspace_bytes(int B, int H, int Lq, int Lk, int d, int causal,
                                         mg_contract_t contract) {
    const std::string saved = mg::host::saved_detail();
    mg_status_t st = check_shape(B, H, Lq, Lk, d, 1.0f, contract);
    mg::host::restore_detail(saved);
    if (st != MG_OK) return 0;
    return mg::attn_bwd_workspace(B, H, Lq, Lk, d, causal, contract, kFusedPartialLimit);
}

mg_status_t mg_attn_bwd_cross(const void *Q, const void *K, const void *V, const void *O,
                              const float *LSE, const void *dO, void *dQ, void *dK, void *dV,
                              const int32_t *key_len, int B, int H, int Lq, int Lk, int d,
                              int causal, float scale, mg_contract_t contract, void *workspace,
                              size_t ws_bytes, hipStream_t stream) {
    MG_TRY(check_shape(B, H, Lq, Lk, d, scale, contract));
    const size_t need =
        mg::attn_bwd_workspace(B, H, Lq, Lk, d, causal, contract, kFusedPartialLimit);
    if (workspace == nullptr || ws_bytes < need)
        return fail(MG_ERR_WORKSPACE, "workspace of %zu bytes given, %zu needed",
                    workspace ? ws_bytes : (size_t)0, need);
    MG_TRY(mg::attn_bwd_check_args(Q, K, V, O, LSE, dO, dQ, dK, dV, key_len, workspace));
    return mg::attn_bwd_enqueue(Q, K, V, O, LSE, dO, dQ, dK, dV, key_len, B, H, Lq, Lk, d,
                                causal, scale, contract, workspace, kFusedPartialLimit, stream);
}

mg_status_t mg_attn_fwd(const void *Q, const void *K, const void *V, void *O, float *LSE,
                        const int32_t *key_len, int B, int H, int L, int d, int causal,
                        float scale, mg_contract_t contract, hipStream_t stream) {
    return mg_attn_fwd_cross(Q, K, V, O, LSE, key_len, B, H, L, L, d, causal, scale, contract,
                             stream);
}

size_t mg_attn_bwd_workspace_bytes(int B, int H, int L, int d, int causal,
                                   mg_contract_t contract) {
    return mg_attn_bwd_cross_workspace_bytes(B, H, L, L, d, causal, contract);
}

mg_status_t mg_attn_bwd(const void *Q, const void *K, const void *V, const void *O,
                        const float *LSE, const void *dO, void *dQ, void *dK, void *dV,
                        const int32_t *key_len, int B, int H, int L, int d, int causal,
                        float scale, mg_contract_t contract, void *workspace,
                        size_t ws_bytes, hipStream_t stream) {
    return mg_attn_bwd_cross(Q, K, V, O, LSE, dO, dQ, dK, dV, key_len, B, H, L, L, d, causal,
                             scale, contract, workspace, ws_bytes, stream);
}

}  // extern "C"
