// mg_attn.cpp -- C ABI of the attention library: argument validation,
// selection of the kernel instance, and launch on the caller's stream.
//
// Validation runs entirely on the host before anything is enqueued, so a
// rejected call has no effect on the device.  The kernel instance and its
// launch geometry are chosen together by the per-kernel launchers.
#include "mg_attn.h"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <initializer_list>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "launch.h"

namespace {

thread_local std::string g_detail;

mg_status_t fail(mg_status_t st, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
mg_status_t fail(mg_status_t st, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_detail = buf;
    return st;
}

mg_status_t ok() {
    g_detail.clear();
    return MG_OK;
}

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

struct NamedPtr {
    const void *ptr;
    const char *name;
};

// Required tensor pointers: non-null and 16-byte aligned (checked for all of
// them first, without touching the runtime), then device-accessible.
mg_status_t check_tensors(std::initializer_list<NamedPtr> ptrs) {
    for (const NamedPtr &p : ptrs) {
        if (p.ptr == nullptr) return fail(MG_ERR_INVALID_ARGUMENT, "%s is NULL", p.name);
        if (reinterpret_cast<uintptr_t>(p.ptr) % 16 != 0)
            return fail(MG_ERR_MISALIGNED, "%s is not 16-byte aligned", p.name);
    }
    for (const NamedPtr &p : ptrs) {
        hipPointerAttribute_t attr;
        hipError_t e = hipPointerGetAttributes(&attr, p.ptr);
        if (e != hipSuccess) {
            (void)hipGetLastError();   // keep the lookup error out of the caller's state
            return fail(MG_ERR_INVALID_ARGUMENT, "%s is not a device pointer (%s)", p.name,
                        hipGetErrorString(e));
        }
        if (attr.type != hipMemoryTypeDevice && attr.type != hipMemoryTypeManaged)
            return fail(MG_ERR_INVALID_ARGUMENT, "%s is not device memory", p.name);
    }
    return MG_OK;
}

mg_status_t check_key_len(const int32_t *key_len) {
    if (key_len == nullptr) return MG_OK;
    if (reinterpret_cast<uintptr_t>(key_len) % 4 != 0)
        return fail(MG_ERR_MISALIGNED, "key_len is not 4-byte aligned");
    hipPointerAttribute_t attr;
    hipError_t e = hipPointerGetAttributes(&attr, key_len);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(MG_ERR_INVALID_ARGUMENT, "key_len is not a device pointer (%s)",
                    hipGetErrorString(e));
    }
    if (attr.type != hipMemoryTypeDevice && attr.type != hipMemoryTypeManaged)
        return fail(MG_ERR_INVALID_ARGUMENT, "key_len is not device memory");
    return MG_OK;
}

#define MG_TRY(expr)                         \
    do {                                     \
        mg_status_t st_ = (expr);            \
        if (st_ != MG_OK) return st_;        \
    } while (0)

// ------------------------------------------------------------- profiling --
struct ProfRecord {
    const char *name;
    hipEvent_t start, stop;
};

struct Profiler {
    std::mutex mu;
    bool enabled = false;
    std::vector<hipEvent_t> pool;
    std::vector<ProfRecord> pending;
    std::map<std::string, std::pair<int64_t, double>> totals;
    std::vector<const char *> order;   // names in first-seen order (static storage)

    hipError_t take(hipEvent_t *ev) {
        if (!pool.empty()) {
            *ev = pool.back();
            pool.pop_back();
            return hipSuccess;
        }
        return hipEventCreate(ev);
    }
};

Profiler &prof() {
    static Profiler p;
    return p;
}

// Launch one kernel, bracketed by events when profiling is enabled.
template <typename F>
mg_status_t run_kernel(const char *name, hipStream_t stream, F &&launch) {
    Profiler &p = prof();
    ProfRecord rec{name, nullptr, nullptr};
    bool timed = false;
    {
        std::lock_guard<std::mutex> g(p.mu);
        if (p.enabled) {
            if (p.take(&rec.start) != hipSuccess || p.take(&rec.stop) != hipSuccess)
                return fail(MG_ERR_HIP, "hipEventCreate failed for %s", name);
            timed = true;
        }
    }
    if (timed && hipEventRecord(rec.start, stream) != hipSuccess)
        return fail(MG_ERR_HIP, "hipEventRecord failed before %s", name);
    hipError_t e = launch();
    if (e != hipSuccess)
        return fail(MG_ERR_HIP, "launch of %s failed: %s", name, hipGetErrorString(e));
    if (timed) {
        if (hipEventRecord(rec.stop, stream) != hipSuccess)
            return fail(MG_ERR_HIP, "hipEventRecord failed after %s", name);
        std::lock_guard<std::mutex> g(p.mu);
        p.pending.push_back(rec);
    }
    return MG_OK;
}

const char *kernel_name(const char *stage, mg_contract_t c, int d) {
    // Static storage: one name per (stage, contract, d).
    static std::mutex mu;
    static std::map<std::string, std::string> names;
    char buf[96];
    const char *suffix = c == MG_CONTRACT_STRICT_F32 ? "f32"
                         : c == MG_CONTRACT_FAST_BF16 ? "bf16" : "accel";
    snprintf(buf, sizeof buf, "%s_%s_d%d", stage, suffix, d);
    std::lock_guard<std::mutex> g(mu);
    auto it = names.find(buf);
    if (it == names.end()) it = names.emplace(buf, buf).first;
    return it->second.c_str();
}

size_t round256(size_t n) { return (n + 255) / 256 * 256; }

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

bool use_fused_dq(int B, int H, int Lq, int Lk, int d, int causal, mg_contract_t contract) {
    return contract == MG_CONTRACT_STRICT_F32 && d <= 64 &&
           dq_partial_bytes(B, H, Lq, Lk, d, causal) <= kFusedPartialLimit;
}

// dK/dV partials of a fused backward whose query tiles are split (zero
// bytes with one split).
size_t dkdv_partial_bytes(int B, int H, int Lq, int Lk, int d, int causal) {
    const mg::AttnProblem p{B, H, Lq, Lk, d, causal ? 1 : 0, 1.0f, nullptr};
    const int ns = mg::fused_dq_query_splits(p);
    return ns > 1 ? (size_t)2 * ns * B * H * Lk * d * sizeof(float) : 0;
}

// Layout: D (f32 per query row) first; when fused, the dQ partials, then
// (256-byte aligned) the dK/dV partials of a split backward.
size_t workspace_bytes(int B, int H, int Lq, int Lk, int d, int causal,
                       mg_contract_t contract) {
    contract = backward_contract(contract);
    size_t n = round256((size_t)B * H * Lq * sizeof(float));
    if (use_fused_dq(B, H, Lq, Lk, d, causal, contract)) {
        n += dq_partial_bytes(B, H, Lq, Lk, d, causal);
        const size_t kv = dkdv_partial_bytes(B, H, Lq, Lk, d, causal);
        if (kv > 0) n = round256(n) + kv;
    }
    return n;
}

}  // namespace

extern "C" {

mg_status_t mg_attn_fwd_cross(const void *Q, const void *K, const void *V, void *O, float *LSE,
                              const int32_t *key_len, int B, int H, int Lq, int Lk, int d,
                              int causal, float scale, mg_contract_t contract,
                              hipStream_t stream) {
    MG_TRY(check_shape(B, H, Lq, Lk, d, scale, contract));
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
    std::string saved = g_detail;
    mg_status_t st = check_shape(B, H, Lq, Lk, d, 1.0f, contract);
    g_detail = saved;
    if (st != MG_OK) return 0;
    return workspace_bytes(B, H, Lq, Lk, d, causal, contract);
}

mg_status_t mg_attn_bwd_cross(const void *Q, const void *K, const void *V, const void *O,
                              const float *LSE, const void *dO, void *dQ, void *dK, void *dV,
                              const int32_t *key_len, int B, int H, int Lq, int Lk, int d,
                              int causal, float scale, mg_contract_t contract, void *workspace,
                              size_t ws_bytes, hipStream_t stream) {
    MG_TRY(check_shape(B, H, Lq, Lk, d, scale, contract));
    const size_t need = workspace_bytes(B, H, Lq, Lk, d, causal, contract);
    if (workspace == nullptr || ws_bytes < need)
        return fail(MG_ERR_WORKSPACE, "workspace of %zu bytes given, %zu needed",
                    workspace ? ws_bytes : (size_t)0, need);
    MG_TRY(check_tensors({{Q, "Q"}, {K, "K"}, {V, "V"}, {O, "O"}, {LSE, "LSE"}, {dO, "dO"},
                          {dQ, "dQ"}, {dK, "dK"}, {dV, "dV"}, {workspace, "workspace"}}));
    MG_TRY(check_key_len(key_len));
    const mg::AttnProblem p{B, H, Lq, Lk, d, causal ? 1 : 0, scale, key_len};
    float *Dws = (float *)workspace;
    contract = backward_contract(contract);
    if (contract == MG_CONTRACT_STRICT_F32) {
        const float *q = (const float *)Q, *k = (const float *)K, *v = (const float *)V;
        const float *o = (const float *)O, *go = (const float *)dO;
        MG_TRY(run_kernel(kernel_name("attn_rowdot", contract, d), stream,
                          [&] { return mg::launch_bwd_rowdot_f32(p, o, go, Dws, stream); }));
        if (use_fused_dq(B, H, Lq, Lk, d, causal, contract)) {
            char *base = (char *)workspace;
            float *dQp = (float *)(base + round256((size_t)B * H * Lq * sizeof(float)));
            float *dKVp = dkdv_partial_bytes(B, H, Lq, Lk, d, causal) == 0 ? nullptr
                : (float *)((char *)dQp + round256(dq_partial_bytes(B, H, Lq, Lk, d, causal)));
            MG_TRY(run_kernel(kernel_name("attn_dkdvq", contract, d), stream, [&] {
                return mg::launch_bwd_dkdvq_f32(p, q, k, v, go, LSE, Dws, (float *)dK,
                                                (float *)dV, dQp, dKVp, stream);
            }));
            if (dKVp != nullptr)
                MG_TRY(run_kernel(kernel_name("attn_dkdvreduce", contract, d), stream, [&] {
                    return mg::launch_bwd_dkdv_reduce_f32(p, dKVp, (float *)dK, (float *)dV,
                                                          stream);
                }));
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
        MG_TRY(run_kernel(kernel_name("attn_rowdot", contract, d), stream,
                          [&] { return mg::launch_bwd_rowdot_bf16(p, o, go, Dws, stream); }));
        MG_TRY(run_kernel(kernel_name("attn_dkdv", contract, d), stream, [&] {
            return mg::launch_bwd_dkdv_bf16(p, q, k, v, go, LSE, Dws, (uint16_t *)dK,
                                            (uint16_t *)dV, stream);
        }));
        MG_TRY(run_kernel(kernel_name("attn_dq", contract, d), stream, [&] {
            return mg::launch_bwd_dq_bf16(p, q, k, v, go, LSE, Dws, (uint16_t *)dQ, stream);
        }));
    }
    return ok();
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

const char *mg_status_string(mg_status_t s) {
    switch (s) {
    case MG_OK: return "MG_OK";
    case MG_ERR_INVALID_ARGUMENT: return "MG_ERR_INVALID_ARGUMENT";
    case MG_ERR_UNSUPPORTED: return "MG_ERR_UNSUPPORTED";
    case MG_ERR_MISALIGNED: return "MG_ERR_MISALIGNED";
    case MG_ERR_WORKSPACE: return "MG_ERR_WORKSPACE";
    case MG_ERR_HIP: return "MG_ERR_HIP";
    }
    return "MG_ERR_UNKNOWN";
}

const char *mg_last_error_detail(void) { return g_detail.c_str(); }

mg_status_t mg_profile_enable(int enable) {
    Profiler &p = prof();
    std::lock_guard<std::mutex> g(p.mu);
    p.enabled = enable != 0;
    return ok();
}

int mg_profile_collect(const char **names, int64_t *launches, double *total_ms,
                       int max_entries) {
    Profiler &p = prof();
    std::lock_guard<std::mutex> g(p.mu);
    for (const ProfRecord &r : p.pending) {
        float ms = 0.f;
        if (hipEventSynchronize(r.stop) != hipSuccess ||
            hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess) {
            fail(MG_ERR_HIP, "event wait failed for %s", r.name);
            return -1;
        }
        auto it = p.totals.find(r.name);
        if (it == p.totals.end()) {
            it = p.totals.emplace(r.name, std::make_pair((int64_t)0, 0.0)).first;
            p.order.push_back(r.name);
        }
        it->second.first += 1;
        it->second.second += ms;
        p.pool.push_back(r.start);
        p.pool.push_back(r.stop);
    }
    p.pending.clear();
    const int n = (int)p.order.size();
    for (int i = 0; i < n && i < max_entries; ++i) {
        const auto &t = p.totals[p.order[i]];
        if (names) names[i] = p.order[i];
        if (launches) launches[i] = t.first;
        if (total_ms) total_ms[i] = t.second;
    }
    return n;
}

void mg_profile_reset(void) {
    Profiler &p = prof();
    std::lock_guard<std::mutex> g(p.mu);
    p.totals.clear();
    p.order.clear();
}

}  // extern "C"
