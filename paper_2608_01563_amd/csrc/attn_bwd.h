// attn_bwd.h -- the attention backward's validation and launch sequence,
// shared by the entry points that take a caller workspace and the one whose
// workspace is the library's static scratch array (internal).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "mg_attn.h"

namespace mg {

// Sizes, contract and scale (the checks that touch no pointer).
mg_status_t attn_bwd_check_shape(int B, int H, int Lq, int Lk, int d, float scale,
                                 mg_contract_t contract);

// Pointer checks: null and alignment of every pointer first, then that each
// is device memory.  `workspace` is checked only when non-null.
mg_status_t attn_bwd_check_args(const void *Q, const void *K, const void *V, const void *O,
                                const float *LSE, const void *dO, void *dQ, void *dK,
                                void *dV, const int32_t *key_len, const void *workspace);

// The dQ-partial size above which strict f32 uses the separate dQ pass
// (the limit of the caller-workspace entry points).
size_t attn_bwd_partial_limit();

// Workspace bytes of a backward that keeps dQ partials only when they fit
// in `partial_limit` bytes (0: never, so the workspace is D alone).
size_t attn_bwd_workspace(int B, int H, int Lq, int Lk, int d, int causal,
                          mg_contract_t contract, size_t partial_limit);

// Enqueue the backward's kernels on `stream` with `workspace`: 256-byte
// aligned device memory of at least attn_bwd_workspace(..., partial_limit)
// bytes.  Arguments must have passed the checks above.
mg_status_t attn_bwd_enqueue(const void *Q, const void *K, const void *V, const void *O,
                             const float *LSE, const void *dO, void *dQ, void *dK, void *dV,
                             const int32_t *key_len, int B, int H, int Lq, int Lk, int d,
                             int causal, float scale, mg_contract_t contract, void *workspace,
                             size_t partial_limit, hipStream_t stream);

}  // namespace mg
