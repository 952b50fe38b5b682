// abi_host_check.cpp -- host-side checks of the C ABI, built together with
// the library's sources under AddressSanitizer and UndefinedBehaviorSanitizer
// (host code only) by tests/test_abi_sanitized_cpu.py.
//
// Every call below is rejected on the host (bad sizes, contract, scale,
// pointers, workspace), or only queries sizes, strings and the profiler, so
// the program needs no GPU; the pointers it passes are never dereferenced.
// Host memory passed as a tensor goes through the runtime's pointer query,
// which must refuse it whether or not a device is present.  The sanitizers
// watch the validation code, the workspace arithmetic, the per-thread error
// detail and the profiler's bookkeeping; any report aborts the program.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <limits>
#include <string>
#include <thread>
#include <vector>

#include "mg_attn.h"
#include "mg_conv.h"

namespace {

int g_failures = 0;

void expect(bool ok, const char *what, int line) {
    if (!ok) {
        std::fprintf(stderr, "FAIL line %d: %s (detail: %s)\n", line, what,
                     mg_last_error_detail());
        ++g_failures;
    }
}
#define EXPECT(cond) expect((cond), #cond, __LINE__)

void *fake(uintptr_t a) { return reinterpret_cast<void *>(a); }

const mg_contract_t kStrict = MG_CONTRACT_STRICT_F32;

mg_status_t fwd(std::vector<void *> p, int B = 1, int H = 1, int L = 8, int d = 64,
                float scale = 0.125f, int contract = 0) {
    return mg_attn_fwd(p[0], p[1], p[2], p[3], static_cast<float *>(p[4]), nullptr, B, H, L, d,
                       1, scale, static_cast<mg_contract_t>(contract), nullptr);
}

std::vector<void *> good5() {
    return {fake(0x1000), fake(0x2000), fake(0x3000), fake(0x4000), fake(0x5000)};
}

void attention_checks() {
    // sizes, head dimension, scale, contract, element count
    EXPECT(fwd(good5(), 0) == MG_ERR_INVALID_ARGUMENT);
    EXPECT(fwd(good5(), 1, -1) == MG_ERR_INVALID_ARGUMENT);
    EXPECT(fwd(good5(), 1, 1, 0) == MG_ERR_INVALID_ARGUMENT);
    EXPECT(fwd(good5(), 1, 1, 8, 0) == MG_ERR_INVALID_ARGUMENT);
    EXPECT(fwd(good5(), 1, 1, 8, 48) == MG_ERR_UNSUPPORTED);
    EXPECT(fwd(good5(), 1, 1, 8, 256) == MG_ERR_UNSUPPORTED);
    EXPECT(fwd(good5(), 1, 1, 8, 64, std::numeric_limits<float>::infinity()) ==
           MG_ERR_INVALID_ARGUMENT);
    EXPECT(fwd(good5(), 1, 1, 8, 64, std::nanf("")) == MG_ERR_INVALID_ARGUMENT);
    EXPECT(fwd(good5(), 1, 1, 8, 64, 0.125f, 5) == MG_ERR_INVALID_ARGUMENT);
    EXPECT(fwd(good5(), 1 << 12, 1 << 10, 1 << 10, 64) == MG_ERR_INVALID_ARGUMENT);
    EXPECT(std::strstr(mg_last_error_detail(), "2^31") != nullptr);
    EXPECT(mg_attn_fwd_cross(fake(0x1000), fake(0x2000), fake(0x3000), fake(0x4000),
                             static_cast<float *>(fake(0x5000)), nullptr, 16, 2, 1 << 22, 4, 64,
                             1, 0.125f, kStrict, nullptr) == MG_ERR_INVALID_ARGUMENT);
    // null and misaligned pointers, each position
    for (int k = 0; k < 5; ++k) {
        std::vector<void *> p = good5();
        p[k] = nullptr;
        EXPECT(fwd(p) == MG_ERR_INVALID_ARGUMENT);
        p[k] = fake(0x1000 * (k + 1) + 4);
        EXPECT(fwd(p) == MG_ERR_MISALIGNED);
    }
    const int32_t *bad_kl = static_cast<const int32_t *>(fake(0x6002));
    EXPECT(mg_attn_fwd(fake(0x1000), fake(0x2000), fake(0x3000), fake(0x4000),
                       static_cast<float *>(fake(0x5000)), bad_kl, 1, 1, 8, 64, 0, 0.125f,
                       kStrict, nullptr) == MG_ERR_MISALIGNED);
    // host memory is not device memory
    std::vector<std::vector<unsigned char>> host(5, std::vector<unsigned char>(4096 + 16));
    std::vector<void *> hp;
    for (auto &b : host)
        hp.push_back(fake((reinterpret_cast<uintptr_t>(b.data()) + 15) / 16 * 16));
    EXPECT(fwd(hp) == MG_ERR_INVALID_ARGUMENT);
    EXPECT(std::strstr(mg_last_error_detail(), "device") != nullptr);

    // backward: workspace checked before any pointer reaches the runtime
    void *p9[9];
    for (int k = 0; k < 9; ++k) p9[k] = fake(0x1000 * (k + 1));
    auto bwd = [&](void *ws, size_t bytes, int contract, int L = 8) {
        return mg_attn_bwd(p9[0], p9[1], p9[2], p9[3], static_cast<const float *>(p9[4]), p9[5],
                           p9[6], p9[7], p9[8], nullptr, 1, 1, L, 64, 1, 0.125f,
                           static_cast<mg_contract_t>(contract), ws, bytes, nullptr);
    };
    EXPECT(bwd(nullptr, 0, 0) == MG_ERR_WORKSPACE);
    EXPECT(bwd(fake(0xa000), 16, 0) == MG_ERR_WORKSPACE);
    EXPECT(bwd(nullptr, 0, 9) == MG_ERR_INVALID_ARGUMENT);
    const size_t need = mg_attn_bwd_workspace_bytes(1, 1, 8, 64, 1, kStrict);
    EXPECT(need > 0);
    EXPECT(bwd(fake(0xa004), need, 0) == MG_ERR_MISALIGNED);

    // the static-scratch backward: sizes first, then the rows D needs, then
    // pointers; nothing here reaches the device
    auto noalloc = [&](void *q, int Lq, int d, int contract) {
        return mg_attn_bwd_noalloc(q, p9[1], p9[2], p9[3], static_cast<const float *>(p9[4]),
                                   p9[5], p9[6], p9[7], p9[8], nullptr, 1, 1, Lq, 64, d, 1,
                                   0.125f, static_cast<mg_contract_t>(contract), nullptr);
    };
    EXPECT(noalloc(p9[0], 8, 48, 0) == MG_ERR_UNSUPPORTED);
    EXPECT(noalloc(p9[0], 8, 64, 4) == MG_ERR_INVALID_ARGUMENT);
    const int too_many = (int)(MG_ATTN_NOALLOC_SCRATCH_BYTES / 4 + 1);
    EXPECT(noalloc(p9[0], too_many, 32, 0) == MG_ERR_WORKSPACE);
    EXPECT(std::strstr(mg_last_error_detail(), "scratch") != nullptr);
    EXPECT(noalloc(p9[0], too_many, 32, 1) == MG_ERR_WORKSPACE);
    EXPECT(noalloc(nullptr, 8, 64, 0) == MG_ERR_INVALID_ARGUMENT);
    EXPECT(noalloc(fake(0x1008), 8, 64, 0) == MG_ERR_MISALIGNED);

    // workspace queries: D rounded to 256 bytes plus the dQ partials
    const size_t rows = 8 * 8 * 1024;
    EXPECT(mg_attn_bwd_workspace_bytes(8, 8, 1024, 64, 1, kStrict) ==
           rows * 4 + 8 * rows * 64 * 4);
    EXPECT(mg_attn_bwd_workspace_bytes(8, 8, 1024, 64, 1, MG_CONTRACT_FAST_BF16) == rows * 4);
    EXPECT(mg_attn_bwd_workspace_bytes(8, 8, 8192, 64, 0, kStrict) == 8 * 8 * 8192 * 4);
    EXPECT(mg_attn_bwd_workspace_bytes(1, 1, 3, 48, 0, kStrict) == 0);
    EXPECT(mg_attn_bwd_workspace_bytes(0, 1, 3, 32, 0, kStrict) == 0);
    EXPECT(mg_attn_bwd_cross_workspace_bytes(1, 1, 3, 0, 32, 0, kStrict) == 0);
    EXPECT(mg_attn_bwd_cross_workspace_bytes(4, 8, 1024, 77, 64, 0, MG_CONTRACT_ACCELERATED) ==
           mg_attn_bwd_cross_workspace_bytes(4, 8, 1024, 77, 64, 0, kStrict));
    // a sweep of shapes through the size arithmetic (split and tile rules)
    for (int L : {1, 2, 63, 64, 65, 127, 128, 129, 1000, 1500, 4096})
        for (int d : {32, 64, 128})
            for (int c = 0; c < 3; ++c)
                for (int causal = 0; causal < 2; ++causal) {
                    const size_t n = mg_attn_bwd_cross_workspace_bytes(
                        2, 3, L, L / 2 + 1, d, causal, static_cast<mg_contract_t>(c));
                    EXPECT(n >= (size_t)2 * 3 * L * 4);
                }
}

mg_conv2d_shape_t shape(int N = 1, int H = 8, int W = 8, int C = 4, int K = 8, int R = 3,
                        int S = 3, int sh = 1, int sw = 1, int ph = 1, int pw = 1) {
    mg_conv2d_shape_t s;
    s.N = N; s.H = H; s.W = W; s.C = C; s.K = K; s.R = R; s.S = S;
    s.stride_h = sh; s.stride_w = sw; s.pad_h = ph; s.pad_w = pw;
    return s;
}

void conv_checks() {
    const float *a = static_cast<const float *>(fake(0x1000));
    const float *b = static_cast<const float *>(fake(0x2000));
    float *c = static_cast<float *>(fake(0x3000));
    float *e = static_cast<float *>(fake(0x4000));
    auto data = [&](const mg_conv2d_shape_t *s, int k) {
        return mg_conv2d_bwd_data(a, b, c, s, static_cast<mg_contract_t>(k), nullptr, 0, nullptr);
    };
    mg_conv2d_shape_t s = shape();
    EXPECT(data(&s, 1) == MG_ERR_UNSUPPORTED);
    EXPECT(data(&s, 7) == MG_ERR_INVALID_ARGUMENT);
    EXPECT(data(nullptr, 0) == MG_ERR_INVALID_ARGUMENT);
    for (mg_conv2d_shape_t bad : {shape(0), shape(1, 8, 8, -1), shape(1, 8, 8, 4, 8, 0),
                                  shape(1, 8, 8, 4, 8, 3, 3, 0), shape(1, 8, 8, 4, 8, 3, 3, 1, 1, 1, -1),
                                  shape(1, 2, 8, 4, 8, 5, 3, 1, 1, 1, 1),
                                  shape(64, 512, 512, 64)})
        EXPECT(data(&bad, 0) == MG_ERR_INVALID_ARGUMENT);
    EXPECT(mg_conv2d_bwd_data(nullptr, b, c, &s, kStrict, nullptr, 0, nullptr) ==
           MG_ERR_INVALID_ARGUMENT);
    EXPECT(mg_conv2d_bwd_data(static_cast<const float *>(fake(0x1004)), b, c, &s, kStrict,
                              nullptr, 0, nullptr) == MG_ERR_MISALIGNED);
    mg_conv2d_shape_t s7 = shape(4, 7, 7, 512, 512, 3, 3, 1, 1, 1, 1);
    EXPECT(mg_conv2d_bwd_data_workspace_bytes(&s7, kStrict) == (size_t)18 * 196 * 512 * 4);
    EXPECT(data(&s7, 0) == MG_ERR_WORKSPACE);
    mg_conv2d_shape_t big = shape(4, 224, 224, 3, 64, 7, 7, 2, 2, 3, 3);
    EXPECT(mg_conv2d_bwd_filter_workspace_bytes(&big, kStrict) == (size_t)196 * 64 * 147 * 4);
    EXPECT(mg_conv2d_bwd_filter(a, b, c, &big, kStrict, nullptr, 0, nullptr) == MG_ERR_WORKSPACE);
    EXPECT(mg_conv2d_bwd(a, b, a, c, e, &s, MG_CONTRACT_FAST_BF16, nullptr, 0, nullptr) ==
           MG_ERR_UNSUPPORTED);
    EXPECT(mg_conv2d_bwd(a, b, a, nullptr, e, &s, kStrict, nullptr, 0, nullptr) ==
           MG_ERR_INVALID_ARGUMENT);
    EXPECT(mg_conv2d_bwd(a, b, a, c, e, &s7, kStrict, nullptr, 0, nullptr) == MG_ERR_WORKSPACE);
    // the size arithmetic over a sweep of layer shapes
    for (int H : {1, 7, 14, 56, 224})
        for (int C : {3, 64, 130})
            for (int st : {1, 2, 3})
                for (int R : {1, 3, 7}) {
                    mg_conv2d_shape_t t = shape(4, H, H, C, 96, R, R, st, st, R / 2, R / 2);
                    (void)mg_conv2d_bwd_workspace_bytes(&t, kStrict);
                    (void)mg_conv2d_bwd_data_workspace_bytes(&t, kStrict);
                    (void)mg_conv2d_bwd_filter_workspace_bytes(&t, kStrict);
                }
}

void runtime_checks() {
    for (int st = 0; st <= 5; ++st)
        EXPECT(std::strncmp(mg_status_string(static_cast<mg_status_t>(st)), "MG_", 3) == 0);
    EXPECT(std::strcmp(mg_status_string(static_cast<mg_status_t>(99)), "MG_ERR_UNKNOWN") == 0);
    double out = 0.0;
    EXPECT(mg_mfma_peak(3, 100, &out, nullptr) == MG_ERR_INVALID_ARGUMENT);
    EXPECT(mg_mfma_peak(0, 0, &out, nullptr) == MG_ERR_INVALID_ARGUMENT);
    EXPECT(mg_mfma_peak(1, 100, nullptr, nullptr) == MG_ERR_INVALID_ARGUMENT);
    EXPECT(mg_lds_probe(7, 256, 100, &out, nullptr) == MG_ERR_INVALID_ARGUMENT);
    EXPECT(mg_lds_probe(11, 64, 100, &out, nullptr) == MG_ERR_INVALID_ARGUMENT);
    EXPECT(mg_lds_probe(17, 64, 100, &out, nullptr) == MG_ERR_INVALID_ARGUMENT);
    EXPECT(mg_lds_probe(19, 256, 100, &out, nullptr) == MG_ERR_INVALID_ARGUMENT);
    EXPECT(mg_lds_probe(0, 264, 100, &out, nullptr) == MG_ERR_INVALID_ARGUMENT);
    EXPECT(mg_lds_probe(0, 256, 0, &out, nullptr) == MG_ERR_INVALID_ARGUMENT);
    EXPECT(mg_lds_probe(0, 256, 100, nullptr, nullptr) == MG_ERR_INVALID_ARGUMENT);
    // the profiler with nothing recorded
    EXPECT(mg_profile_enable(1) == MG_OK);
    const char *names[4];
    int64_t launches[4];
    double ms[4];
    EXPECT(mg_profile_collect(names, launches, ms, 4) == 0);
    EXPECT(mg_profile_enable(0) == MG_OK);
    mg_profile_reset();
    // the error detail belongs to the calling thread
    EXPECT(fwd(good5(), 0) == MG_ERR_INVALID_ARGUMENT);
    const std::string mine = mg_last_error_detail();
    std::string fresh, own;
    std::thread t1([&] { fresh = mg_last_error_detail(); });
    t1.join();
    std::thread t2([&] {
        EXPECT(fwd(good5(), 1, 1, 8, 48) == MG_ERR_UNSUPPORTED);
        own = mg_last_error_detail();
    });
    t2.join();
    EXPECT(fresh.empty());
    EXPECT(!own.empty() && own != mine);
    EXPECT(mine == mg_last_error_detail());
    // several threads failing at once
    std::vector<std::thread> ts;
    for (int i = 0; i < 8; ++i)
        ts.emplace_back([i] {
            for (int r = 0; r < 200; ++r) {
                EXPECT(fwd(good5(), 1, 1, 8, 40 + i) == MG_ERR_UNSUPPORTED);
                EXPECT(std::strstr(mg_last_error_detail(), std::to_string(40 + i).c_str()) !=
                       nullptr);
            }
        });
    for (auto &t : ts) t.join();
}

}  // namespace

int main() {
    attention_checks();
    conv_checks();
    runtime_checks();
    if (g_failures != 0) {
        std::fprintf(stderr, "%d check(s) failed\n", g_failures);
        return 1;
    }
    std::printf("abi host checks passed\n");
    return 0;
}
