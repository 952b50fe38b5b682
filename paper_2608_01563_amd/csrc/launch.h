// launch.h -- host-side launchers of the attention kernels (internal).
//
// Each launcher enqueues exactly one kernel on `stream` and returns the
// launch status; argument validation happens before, in mg_attn.cpp.  The
// launch geometry of every kernel is fixed together with its template
// instance inside its launcher, never chosen separately.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace mg {

// Q, O, dO, dQ are [B][H][Lq][d]; K, V, dK, dV are [B][H][Lk][d]; LSE and D
// are [B][H][Lq].  Under a causal mask query row i sees keys j <= i + Lk - Lq
// (bottom-right alignment; j <= i when Lq == Lk).
struct AttnProblem {
    int B, H, Lq, Lk, d;
    int causal;
    float scale;
    const int32_t *key_len;  // device [B] or nullptr
};

// Rank-order layer of a causal tile grid (the `layer` argument of
// serpentine_rank in device_common.h).  When all `grid` workgroups of
// `kernel` (`block` threads each, no dynamic LDS) are resident on the current
// device at once and its CU count is a multiple of the head count BH, the
// dispatcher places workgroup i on CU i mod CUs, so layers of CUs/BH ranks
// that alternate direction give every CU a mix of heavy and light causal
// tiles.  Otherwise 0: heavy tiles first, and the dispatcher hands the light
// ones to whichever CU frees up first.  Non-causal grids get 0.
int causal_rank_layer(const void *kernel, int block, long grid, int BH, int causal);

// Forward, strict f32: O, LSE from Q, K, V.
hipError_t launch_fwd_f32(const AttnProblem &p, const float *Q, const float *K,
                          const float *V, float *O, float *LSE, hipStream_t s);
// Forward, bf16 inputs/outputs, f32 accumulation.
hipError_t launch_fwd_bf16(const AttnProblem &p, const uint16_t *Q, const uint16_t *K,
                           const uint16_t *V, uint16_t *O, float *LSE, hipStream_t s);

// Forward under the accelerated contract: f32 Q, K, V, O, LSE; Q, K, V and
// P rounded to f16 as matrix-core inputs, f32 accumulation.
hipError_t launch_fwd_accel(const AttnProblem &p, const float *Q, const float *K,
                            const float *V, float *O, float *LSE, hipStream_t s);

// Backward step 1: D_i = sum_k dO_ik O_ik (f32 out, one per row).
hipError_t launch_bwd_rowdot_f32(const AttnProblem &p, const float *O, const float *dO,
                                 float *Dws, hipStream_t s);

// Backward step 2: dK, dV with the key tile stationary.
hipError_t launch_bwd_dkdv_f32(const AttnProblem &p, const float *Q, const float *K,
                               const float *V, const float *dO, const float *LSE,
                               const float *Dws, float *dK, float *dV, hipStream_t s);
hipError_t launch_bwd_dkdv_bf16(const AttnProblem &p, const uint16_t *Q,
                                const uint16_t *K, const uint16_t *V, const uint16_t *dO,
                                const float *LSE, const float *Dws, uint16_t *dK,
                                uint16_t *dV, hipStream_t s);

// Backward steps 2+3 fused (strict f32, d <= 64): dK, dV as above plus one
// f32 dQ partial per (key tile, query row) written to dQp, laid out
// [key tile][B*H][Lq][d]; then dQ = scale * sum of a row's partials.  The
// key-tile height (64 or 128) depends on the problem.  When the key tiles
// alone give too small a grid, each key tile's query tiles are split over
// fused_dq_query_splits(p) workgroups, which write dK/dV partials to dKVp
// ([dK, dV][split][B*H][Lk][d] f32; unused, may be null, with one split)
// for launch_bwd_reduce_f32 to add, together with the dQ partials, in one
// launch (launch_bwd_dq_reduce_f32 alone when there is one split).
// Small grids (fused_local_d) compute D inside the kernel from O and dO, so
// Dws is not read and needs no D launch before; with one key tile per head
// and no split (fused_direct_dq) dQp must be dQ itself: the kernel writes
// the scaled dQ there, zeros included, and no reduction follows.
int fused_dq_key_rows(const AttnProblem &p);
int fused_dq_query_splits(const AttnProblem &p);
bool fused_local_d(const AttnProblem &p);
bool fused_direct_dq(const AttnProblem &p);
hipError_t launch_bwd_dkdvq_f32(const AttnProblem &p, const float *Q, const float *K,
                                const float *V, const float *O, const float *dO,
                                const float *LSE, const float *Dws, float *dK, float *dV,
                                float *dQp, float *dKVp, hipStream_t s);
hipError_t launch_bwd_reduce_f32(const AttnProblem &p, const float *dKVp, float *dK,
                                 float *dV, const float *dQp, float *dQ, hipStream_t s);
hipError_t launch_bwd_dq_reduce_f32(const AttnProblem &p, const float *dQp, float *dQ,
                                    hipStream_t s);

// Backward step 3: dQ with the query tile stationary.
hipError_t launch_bwd_dq_f32(const AttnProblem &p, const float *Q, const float *K,
                             const float *V, const float *dO, const float *LSE,
                             const float *Dws, float *dQ, hipStream_t s);
// bf16: the dQ kernel also computes D_i = sum_k dO_ik O_ik for its rows
// and writes it to Dws; it runs first, and the dK/dV kernel reads D from
// Dws after it.
hipError_t launch_bwd_dq_bf16(const AttnProblem &p, const uint16_t *Q, const uint16_t *K,
                              const uint16_t *V, const uint16_t *O, const uint16_t *dO,
                              const float *LSE, float *Dws, uint16_t *dQ, hipStream_t s);

}  // namespace mg
