// host_runtime.h -- host-side plumbing shared by the library's C entry points:
// the per-thread error detail, pointer validation, kernel-name interning and
// the optional per-launch event timing behind mg_profile_*.
//
// Nothing here touches the device except hipPointerGetAttributes (pointer
// validation) and, while profiling is enabled, event creation and recording.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <initializer_list>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "mg_attn.h"

namespace mg {
namespace host {

// Record a formatted error detail for mg_last_error_detail() and return `st`.
mg_status_t fail(mg_status_t st, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
// Clear the detail and return MG_OK.
mg_status_t ok();
// Keep the current detail across a call that may overwrite it.
std::string saved_detail();
void restore_detail(const std::string &s);

struct NamedPtr {
    const void *ptr;
    const char *name;
};

// Required pointers: non-null and `align`-byte aligned (checked for all of
// them first, without touching the runtime), then device-accessible.
mg_status_t check_device_ptrs(std::initializer_list<NamedPtr> ptrs, int align = 16);
// An optional pointer: null is fine, otherwise aligned device memory.
mg_status_t check_optional_device_ptr(const void *ptr, const char *name, int align);

// "<stage>_<suffix>" with static storage (one string per distinct name).
const char *intern_name(const std::string &name);

size_t round256(size_t n);

// ---- per-launch event timing (mg_profile_enable / collect / reset)
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

    hipError_t take(hipEvent_t *ev);
};

Profiler &profiler();

// Launch one kernel, bracketed by events on `stream` when profiling is on.
template <typename F>
mg_status_t run_kernel(const char *name, hipStream_t stream, F &&launch) {
    Profiler &p = profiler();
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

}  // namespace host
}  // namespace mg

#define MG_TRY(expr)                         \
    do {                                     \
        mg_status_t st_ = (expr);            \
        if (st_ != MG_OK) return st_;        \
    } while (0)
