// host_runtime.cpp -- the shared host plumbing of host_runtime.h and the
// library-wide C entry points that report on it (status strings, the last
// error detail, per-launch event timing), plus the launch-order query of
// launch.h (causal_rank_layer).
#include "host_runtime.h"
#include "launch.h"

#include <cstdarg>
#include <cstdio>
#include <map>
#include <mutex>
#include <tuple>

namespace mg {
namespace host {
namespace {
thread_local std::string g_detail;
}

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

std::string saved_detail() { return g_detail; }
void restore_detail(const std::string &s) { g_detail = s; }

static mg_status_t check_device(const void *ptr, const char *name) {
    hipPointerAttribute_t attr;
    hipError_t e = hipPointerGetAttributes(&attr, ptr);
    if (e != hipSuccess) {
        (void)hipGetLastError();   // keep the lookup error out of the caller's state
        return fail(MG_ERR_INVALID_ARGUMENT, "%s is not a device pointer (%s)", name,
                    hipGetErrorString(e));
    }
    if (attr.type != hipMemoryTypeDevice && attr.type != hipMemoryTypeManaged)
        return fail(MG_ERR_INVALID_ARGUMENT, "%s is not device memory", name);
    return MG_OK;
}

mg_status_t check_device_ptrs(std::initializer_list<NamedPtr> ptrs, int align) {
    for (const NamedPtr &p : ptrs) {
        if (p.ptr == nullptr) return fail(MG_ERR_INVALID_ARGUMENT, "%s is NULL", p.name);
        if (reinterpret_cast<uintptr_t>(p.ptr) % align != 0)
            return fail(MG_ERR_MISALIGNED, "%s is not %d-byte aligned", p.name, align);
    }
    for (const NamedPtr &p : ptrs) MG_TRY(check_device(p.ptr, p.name));
    return MG_OK;
}

mg_status_t check_optional_device_ptr(const void *ptr, const char *name, int align) {
    if (ptr == nullptr) return MG_OK;
    if (reinterpret_cast<uintptr_t>(ptr) % align != 0)
        return fail(MG_ERR_MISALIGNED, "%s is not %d-byte aligned", name, align);
    return check_device(ptr, name);
}

const char *intern_name(const std::string &name) {
    static std::mutex mu;
    static std::map<std::string, std::string> names;
    std::lock_guard<std::mutex> g(mu);
    auto it = names.find(name);
    if (it == names.end()) it = names.emplace(name, name).first;
    return it->second.c_str();
}

size_t round256(size_t n) { return (n + 255) / 256 * 256; }

hipError_t Profiler::take(hipEvent_t *ev) {
    if (!pool.empty()) {
        *ev = pool.back();
        pool.pop_back();
        return hipSuccess;
    }
    return hipEventCreate(ev);
}

Profiler &profiler() {
    static Profiler p;
    return p;
}

}  // namespace host
}  // namespace mg

namespace mg {

int causal_rank_layer(const void *kernel, int block, long grid, int BH, int causal) {
    if (!causal || BH <= 0) return 0;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();
        return 0;
    }
    // (kernel, block, device) -> (CUs, resident workgroups per CU)
    static std::mutex mu;
    static std::map<std::tuple<const void *, int, int>, std::pair<int, int>> cache;
    std::pair<int, int> res;
    {
        std::lock_guard<std::mutex> g(mu);
        auto key = std::make_tuple(kernel, block, dev);
        auto it = cache.find(key);
        if (it == cache.end()) {
            int cus = 0, per_cu = 0;
            if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                    hipSuccess ||
                hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, block, 0) !=
                    hipSuccess) {
                (void)hipGetLastError();
                cus = per_cu = 0;
            }
            it = cache.emplace(key, std::make_pair(cus, per_cu)).first;
        }
        res = it->second;
    }
    const int cus = res.first, per_cu = res.second;
    if (cus <= 0 || per_cu <= 0 || grid > (long)cus * per_cu || cus % BH != 0) return 0;
    return cus / BH;
}

}  // namespace mg

using namespace mg::host;

extern "C" {

const char *mg_status_string(mg_status_t s) {
    switch (s) {
    case MG_OK: return "MG_OK";
    case MG_ERR_INVALID_ARGUMENT: return "MG_ERR_INVALID_ARGUMENT";
    case MG_ERR_UNSUPPORTED: return "MG_ERR_UNSUPPORTED";
    case MG_ERR_MISALIGNED: return "MG_ERR_MISALIGNED";
    case MG_ERR_WORKSPACE: return "MG_ERR_WORKSPACE";
    case MG_ERR_HIP: return "MG_ERR_HIP";
    default: break;
    }
    return "MG_ERR_UNKNOWN";
}

const char *mg_last_error_detail(void) { return g_detail.c_str(); }

mg_status_t mg_profile_enable(int enable) {
    Profiler &p = profiler();
    std::lock_guard<std::mutex> g(p.mu);
    p.enabled = enable != 0;
    return ok();
}

int mg_profile_collect(const char **names, int64_t *launches, double *total_ms,
                       int max_entries) {
    Profiler &p = profiler();
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
    Profiler &p = profiler();
    std::lock_guard<std::mutex> g(p.mu);
    p.totals.clear();
    p.order.clear();
}

}  // extern "C"
