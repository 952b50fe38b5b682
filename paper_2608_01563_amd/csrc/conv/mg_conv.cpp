// mg_conv.cpp -- C ABI of the convolution derivatives: argument validation,
// workspace sizing and launch on the caller's stream.  Validation runs on
// the host before anything is enqueued.
#include "mg_conv.h"

#include <cstdint>
#include <cstdio>

#include "conv_launch.h"
#include "host_runtime.h"

namespace {

using mg::host::fail;
using mg::host::ok;
using mg::host::run_kernel;

constexpr int64_t kMaxBytes = INT32_MAX;   // 32-bit byte offsets in the kernels

mg_status_t check_contract(mg_contract_t c) {
    if (c == MG_CONTRACT_FAST_BF16)
        return fail(MG_ERR_UNSUPPORTED, "the convolution derivatives have no bf16 contract");
    if (c != MG_CONTRACT_STRICT_F32 && c != MG_CONTRACT_ACCELERATED)
        return fail(MG_ERR_INVALID_ARGUMENT, "unknown contract %d", (int)c);
    return MG_OK;
}

// Shape checks and the derived output size; fills `p` on success.
mg_status_t check_shape(const mg_conv2d_shape_t *s, mg::ConvProblem *p) {
    if (s == nullptr) return fail(MG_ERR_INVALID_ARGUMENT, "shape is NULL");
    if (s->N < 1 || s->H < 1 || s->W < 1 || s->C < 1 || s->K < 1 || s->R < 1 || s->S < 1)
        return fail(MG_ERR_INVALID_ARGUMENT,
                    "sizes must be >= 1 (N=%d H=%d W=%d C=%d K=%d R=%d S=%d)", s->N, s->H, s->W,
                    s->C, s->K, s->R, s->S);
    if (s->stride_h < 1 || s->stride_w < 1 || s->pad_h < 0 || s->pad_w < 0)
        return fail(MG_ERR_INVALID_ARGUMENT, "strides must be >= 1 and padding >= 0");
    const int64_t span_h = (int64_t)s->H + 2 * (int64_t)s->pad_h - s->R;
    const int64_t span_w = (int64_t)s->W + 2 * (int64_t)s->pad_w - s->S;
    if (span_h < 0 || span_w < 0)
        return fail(MG_ERR_INVALID_ARGUMENT, "the filter does not fit the padded input");
    const int64_t P = span_h / s->stride_h + 1, Q = span_w / s->stride_w + 1;
    const int64_t x = (int64_t)s->N * s->H * s->W * s->C * 4;
    const int64_t y = (int64_t)s->N * P * Q * s->K * 4;
    const int64_t w = (int64_t)s->K * s->R * s->S * s->C * 4;
    if (x > kMaxBytes || y > kMaxBytes || w > kMaxBytes)
        return fail(MG_ERR_INVALID_ARGUMENT, "a tensor exceeds 2^31-1 bytes (X %lld, dY %lld, "
                    "W %lld)", (long long)x, (long long)y, (long long)w);
    *p = mg::ConvProblem{s->N, s->H, s->W, s->C, s->K, s->R, s->S, s->stride_h, s->stride_w,
                         s->pad_h, s->pad_w, (int)P, (int)Q};
    return MG_OK;
}

// Output elements of each derivative, and the workspace of its split sum.
size_t dgrad_elems(const mg::ConvProblem &p) { return (size_t)p.N * p.H * p.W * p.C; }
size_t wgrad_elems(const mg::ConvProblem &p) { return (size_t)p.K * p.R * p.S * p.C; }

size_t dgrad_workspace(const mg::ConvProblem &p) {
    const int ns = mg::conv_dgrad_splits(p);
    return ns > 1 ? (size_t)ns * dgrad_elems(p) * sizeof(float) : 0;
}

size_t wgrad_workspace(const mg::ConvProblem &p) {
    const int ns = mg::conv_wgrad_splits(p);
    return ns > 1 ? (size_t)ns * wgrad_elems(p) * sizeof(float) : 0;
}

// Both derivatives at once: the data gradient's partials, then (from a
// 256-byte boundary) the filter gradient's.
size_t both_workspace(const mg::ConvProblem &p) {
    const size_t w = wgrad_workspace(p);
    return w > 0 ? mg::host::round256(dgrad_workspace(p)) + w : dgrad_workspace(p);
}

mg_status_t check_workspace(const void *workspace, size_t bytes, size_t need) {
    if (need == 0) return MG_OK;
    if (workspace == nullptr || bytes < need)
        return fail(MG_ERR_WORKSPACE, "workspace of %zu bytes given, %zu needed",
                    workspace ? bytes : (size_t)0, need);
    return mg::host::check_device_ptrs({{workspace, "workspace"}}, 16);
}

// Query helper: the workspace size for valid arguments, 0 otherwise; the
// caller's last error detail is left as it was.
template <typename F>
size_t query_workspace(const mg_conv2d_shape_t *shape, mg_contract_t contract, F &&bytes) {
    const std::string saved = mg::host::saved_detail();
    mg::ConvProblem p;
    const bool good = check_contract(contract) == MG_OK && check_shape(shape, &p) == MG_OK;
    mg::host::restore_detail(saved);
    return good ? bytes(p) : 0;
}

}  // namespace

extern "C" {

size_t mg_conv2d_bwd_data_workspace_bytes(const mg_conv2d_shape_t *shape,
                                          mg_contract_t contract) {
    return query_workspace(shape, contract, dgrad_workspace);
}

mg_status_t mg_conv2d_bwd_data(const float *dY, const float *W, float *dX,
                               const mg_conv2d_shape_t *shape, mg_contract_t contract,
                               void *workspace, size_t workspace_bytes, hipStream_t stream) {
    mg::ConvProblem p;
    MG_TRY(check_contract(contract));
    MG_TRY(check_shape(shape, &p));
    const size_t need = dgrad_workspace(p);
    MG_TRY(check_workspace(workspace, workspace_bytes, need));
    MG_TRY(mg::host::check_device_ptrs({{dY, "dY"}, {W, "W"}, {dX, "dX"}}, 16));
    float *part = need > 0 ? (float *)workspace : nullptr;
    MG_TRY(run_kernel("conv_dgrad_f32", stream,
                      [&] { return mg::launch_conv_dgrad_f32(p, dY, W, dX, part, stream); }));
    if (part != nullptr)
        MG_TRY(run_kernel("conv_dgrad_reduce_f32", stream, [&] {
            return mg::launch_conv_split_reduce_f32(part, mg::conv_dgrad_splits(p),
                                                    (int)dgrad_elems(p), dX, stream);
        }));
    return ok();
}

size_t mg_conv2d_bwd_filter_workspace_bytes(const mg_conv2d_shape_t *shape,
                                            mg_contract_t contract) {
    return query_workspace(shape, contract, wgrad_workspace);
}

mg_status_t mg_conv2d_bwd_filter(const float *X, const float *dY, float *dW,
                                 const mg_conv2d_shape_t *shape, mg_contract_t contract,
                                 void *workspace, size_t workspace_bytes, hipStream_t stream) {
    mg::ConvProblem p;
    MG_TRY(check_contract(contract));
    MG_TRY(check_shape(shape, &p));
    const size_t need = wgrad_workspace(p);
    MG_TRY(check_workspace(workspace, workspace_bytes, need));
    MG_TRY(mg::host::check_device_ptrs({{X, "X"}, {dY, "dY"}, {dW, "dW"}}, 16));
    float *part = need > 0 ? (float *)workspace : nullptr;
    MG_TRY(run_kernel("conv_wgrad_f32", stream,
                      [&] { return mg::launch_conv_wgrad_f32(p, X, dY, dW, part, stream); }));
    if (part != nullptr)
        MG_TRY(run_kernel("conv_wgrad_reduce_f32", stream, [&] {
            return mg::launch_conv_split_reduce_f32(part, mg::conv_wgrad_splits(p),
                                                    (int)wgrad_elems(p), dW, stream);
        }));
    return ok();
}

size_t mg_conv2d_bwd_workspace_bytes(const mg_conv2d_shape_t *shape, mg_contract_t contract) {
    return query_workspace(shape, contract, [](const mg::ConvProblem &p) {
        return both_workspace(p);
    });
}

mg_status_t mg_conv2d_bwd(const float *X, const float *W, const float *dY, float *dX, float *dW,
                          const mg_conv2d_shape_t *shape, mg_contract_t contract,
                          void *workspace, size_t workspace_bytes, hipStream_t stream) {
    mg::ConvProblem p;
    MG_TRY(check_contract(contract));
    MG_TRY(check_shape(shape, &p));
    const size_t need = both_workspace(p);
    MG_TRY(check_workspace(workspace, workspace_bytes, need));
    MG_TRY(mg::host::check_device_ptrs({{X, "X"}, {W, "W"}, {dY, "dY"}, {dX, "dX"}, {dW, "dW"}},
                                       16));
    const size_t dbytes = dgrad_workspace(p);
    float *dpart = dbytes > 0 ? (float *)workspace : nullptr;
    float *wpart = wgrad_workspace(p) > 0
        ? (float *)((char *)workspace + mg::host::round256(dbytes)) : nullptr;
    MG_TRY(run_kernel("conv_bwd_f32", stream, [&] {
        return mg::launch_conv_bwd_f32(p, X, W, dY, dX, dW, dpart, wpart, stream);
    }));
    if (dpart != nullptr && wpart != nullptr)
        MG_TRY(run_kernel("conv_bwd_reduce_f32", stream, [&] {
            return mg::launch_conv_split_reduce2_f32(dpart, mg::conv_dgrad_splits(p),
                                                     (int)dgrad_elems(p), dX, wpart,
                                                     mg::conv_wgrad_splits(p),
                                                     (int)wgrad_elems(p), dW, stream);
        }));
    else if (dpart != nullptr || wpart != nullptr)
        MG_TRY(run_kernel("conv_bwd_reduce_f32", stream, [&] {
            return dpart != nullptr
                ? mg::launch_conv_split_reduce_f32(dpart, mg::conv_dgrad_splits(p),
                                                   (int)dgrad_elems(p), dX, stream)
                : mg::launch_conv_split_reduce_f32(wpart, mg::conv_wgrad_splits(p),
                                                   (int)wgrad_elems(p), dW, stream);
        }));
    return ok();
}

}  // extern "C"
