/*
 * mg_attn.h -- C ABI of the MI355X (gfx950) attention library.
 *
 * Multi-head scaled-dot-product attention, forward and backward, as the
 * paper's tiled attention forward kernel, fused dK+dV kernel and dQ kernel
 * (Sec. 3.3 "Kernel archetypes and specialization"; Sec. 7.3, where the
 * backward pair is the largest measured cost of the Whisper training step).
 * The operation is exact attention:
 *
 *   allowed(i,j) = (!causal || j <= i) && j < key_len[b]
 *   S = scale * Q K^T,  P = softmax over allowed j (masked P is exactly 0)
 *   O = P V,  LSE_i = ln sum_j exp(S_ij)      (natural log)
 *   D_i = sum_k dO_ik O_ik,  dP = dO V^T,  dS = P o (dP - D)
 *   dQ = scale * dS K,  dK = scale * dS^T Q,  dV = P^T dO
 *
 * Arithmetic contracts (Sec. 4.2 "Arithmetic contracts", Table of arithmetic
 * permissions):
 *   MG_CONTRACT_STRICT_F32  every tensor f32; products on f32 matrix cores
 *                           with f32 accumulation (the paper's --strict mode).
 *   MG_CONTRACT_FAST_BF16   Q,K,V,O,dO,dQ,dK,dV are bf16; products run on
 *                           bf16 matrix cores with f32 accumulation, P and dS
 *                           are rounded to bf16 (nearest even) as operands;
 *                           outputs are rounded to bf16 (nearest even).  The
 *                           paper's reduced-input mode uses f16 and keeps the
 *                           backward f32; this contract uses bf16 (f32
 *                           exponent range) for both passes.
 *   MG_CONTRACT_ACCELERATED the paper's practical default: every tensor f32;
 *                           the forward rounds Q, K, V (and P as the operand
 *                           of P V) to f16, nearest even, and multiplies on
 *                           f16 matrix cores with f32 accumulation; the
 *                           backward is exactly the strict_f32 backward.
 *   LSE and the workspace are always f32.
 *
 * Layout: Q, K, V, O, dO, dQ, dK, dV are contiguous [B][H][L][d] with d
 * fastest; LSE is [B][H][L].  key_len is an int32 device array [B] or NULL
 * (no padding); its values are clamped to [0, L] on the device.  A row with
 * no allowed key (key_len[b] == 0) yields O = 0, LSE = -inf and zero
 * gradients.  Causal masking: query row i sees keys j <= i (equal query and
 * key lengths; see mg_attn_fwd_cross for the general case).
 *
 * Ownership: the caller owns every buffer, including the backward workspace.
 * The library allocates no device memory, keeps no per-call state and is
 * reentrant.  All pointers except key_len must be device pointers, 16-byte
 * aligned.  Outputs must not alias inputs (not checked; undefined results).
 *
 * Asynchrony: every call enqueues kernels on `stream` and returns without
 * synchronizing.  Results are valid once the stream reaches that point.
 *
 * Errors: argument errors are detected on the host before anything is
 * enqueued; the call then returns a non-MG_OK status and enqueues nothing.
 * Launch failures return MG_ERR_HIP.  mg_last_error_detail() gives a
 * message for the last failing call on the calling thread.
 */
#ifndef MG_ATTN_H
#define MG_ATTN_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Both enums span the whole range of int (the two range markers are not
 * values any call accepts): a caller may pass any int, and the library
 * rejects an unknown contract with MG_ERR_INVALID_ARGUMENT instead of
 * receiving a value its own type cannot hold.
 */
typedef enum {
    MG_CONTRACT_STRICT_F32 = 0,
    MG_CONTRACT_FAST_BF16 = 1,
    MG_CONTRACT_ACCELERATED = 2,
    MG_CONTRACT_RANGE_MIN_ = (-0x7fffffff - 1),
    MG_CONTRACT_RANGE_MAX_ = 0x7fffffff
} mg_contract_t;

typedef enum {
    MG_OK = 0,
    MG_ERR_INVALID_ARGUMENT = 1, /* null pointer, size < 1, non-finite scale,
                                    bad contract, B*H*L*d > 2^31-1
                                    (cross: B*H*max(Lq,Lk)*d)               */
    MG_ERR_UNSUPPORTED = 2,      /* head dimension d not in {32, 64, 128}   */
    MG_ERR_MISALIGNED = 3,       /* a tensor pointer not 16-byte aligned    */
    MG_ERR_WORKSPACE = 4,        /* backward workspace missing or too small */
    MG_ERR_HIP = 5,              /* a HIP runtime call or launch failed     */
    MG_STATUS_RANGE_MIN_ = (-0x7fffffff - 1),
    MG_STATUS_RANGE_MAX_ = 0x7fffffff
} mg_status_t;

/*
 * Forward pass: O and LSE from Q, K, V (the paper's tiled attention forward,
 * Sec. 3.3).  Inputs Q, K, V [B][H][L][d]; outputs O [B][H][L][d] and LSE
 * [B][H][L] (f32, natural log, saved for the backward pass).  Element type of
 * Q, K, V, O follows `contract`.  `scale` multiplies Q K^T (typically
 * 1/sqrt(d)); it must be finite.
 */
mg_status_t mg_attn_fwd(const void *Q, const void *K, const void *V,
                        void *O, float *LSE,
                        const int32_t *key_len,
                        int B, int H, int L, int d, int causal, float scale,
                        mg_contract_t contract, hipStream_t stream);

/*
 * Bytes of device workspace that mg_attn_bwd needs for these arguments:
 * f32 D = rowsum(dO o O), one per query row, rounded up to 256 bytes, plus,
 * for strict_f32 and accelerated with d <= 64 when they fit in 1 GiB, one f32
 * dQ partial per (key tile, query row): ceil(L/T) * B*H*L*d floats with key
 * tiles of T = 128 keys when causal and ceil(L/128)*B*H >= 512, else T = 64.
 * The partials let the dK/dV kernel produce dQ without a second recompute.
 * When ceil(L/T)*B*H < 512 (too few key tiles to fill the GPU), the query
 * tiles of each key tile are split over S workgroups and 2*S*B*H*L*d more
 * f32 hold their dK and dV partials (S = min(ceil(1024 / (ceil(L/T)*B*H)),
 * floor(n / m)) with n = ceil(L/32) query tiles and m = 2 when n <= 8, else
 * m = 4; no partials when S <= 1), each region starting on a 256-byte
 * boundary.  Returns 0 when the arguments are invalid.
 */
size_t mg_attn_bwd_workspace_bytes(int B, int H, int L, int d, int causal,
                                   mg_contract_t contract);

/*
 * Backward pass: dQ, dK, dV from Q, K, V, the forward outputs O and LSE, and
 * the upstream gradient dO (the paper's attention derivative node, Sec. 3.1,
 * lowered to a fused dK+dV kernel and a separate dQ kernel, Sec. 3.3 and
 * Sec. 8; for strict_f32 with d <= 64 the dK+dV kernel also emits per-tile
 * dQ partials that a reduction kernel sums, or, with a single key tile and
 * no query split, writes dQ itself).  P is recomputed from Q, K and
 * the saved LSE; nothing of size L x L is stored.  `workspace` is
 * caller-owned device memory of at least mg_attn_bwd_workspace_bytes(...)
 * bytes; its contents on entry are ignored
 * and on return are unspecified.  dK and dV rows of masked (padded) keys are
 * written as exact zeros.  Deterministic: no atomics, bitwise identical
 * results for identical inputs.
 */
mg_status_t mg_attn_bwd(const void *Q, const void *K, const void *V,
                        const void *O, const float *LSE, const void *dO,
                        void *dQ, void *dK, void *dV,
                        const int32_t *key_len,
                        int B, int H, int L, int d, int causal, float scale,
                        mg_contract_t contract,
                        void *workspace, size_t workspace_bytes,
                        hipStream_t stream);

/*
 * Cross-attention: queries and keys of different lengths (Sec. 10 workloads:
 * the U-Net's 77-token text cross-attention, the action expert's action and
 * context tokens).  Q, O, dO, dQ are [B][H][Lq][d]; K, V, dK, dV are
 * [B][H][Lk][d]; LSE and the workspace's D are [B][H][Lq]; key_len values
 * are clamped to [0, Lk].  The causal mask is bottom-right aligned: query row
 * i sees keys j <= i + Lk - Lq, so the last query row sees every key and,
 * when Lk < Lq, the first Lq - Lk rows see none (O = 0, LSE = -inf, no
 * gradient).  With Lq == Lk these are exactly mg_attn_fwd / mg_attn_bwd,
 * which call them.  Arguments, contracts, ownership, asynchrony and errors
 * are otherwise as there; the workspace holds D and, for strict_f32 and
 * accelerated with d <= 64 when they fit in 1 GiB, ceil(Lk/T) * B*H*Lq*d
 * f32 dQ partials and 2*S*B*H*Lk*d f32 dK/dV partials (T and S as above,
 * with Lk for the key length and ceil(Lq/32) query tiles).
 */
mg_status_t mg_attn_fwd_cross(const void *Q, const void *K, const void *V,
                              void *O, float *LSE,
                              const int32_t *key_len,
                              int B, int H, int Lq, int Lk, int d, int causal, float scale,
                              mg_contract_t contract, hipStream_t stream);

size_t mg_attn_bwd_cross_workspace_bytes(int B, int H, int Lq, int Lk, int d, int causal,
                                         mg_contract_t contract);

mg_status_t mg_attn_bwd_cross(const void *Q, const void *K, const void *V,
                              const void *O, const float *LSE, const void *dO,
                              void *dQ, void *dK, void *dV,
                              const int32_t *key_len,
                              int B, int H, int Lq, int Lk, int d, int causal, float scale,
                              mg_contract_t contract,
                              void *workspace, size_t workspace_bytes,
                              hipStream_t stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * backward of mg_attn_bwd_cross with its workspace in a static device array
 * of the library, MG_ATTN_NOALLOC_SCRATCH_BYTES bytes on each device it
 * runs on, held until the process ends.  Same arguments, kernels, results
 * and errors as mg_attn_bwd_cross without the workspace pair.  The call
 * allocates nothing (no hipMalloc or hipFree, no allocating library call).
 * When the caller-workspace layout (mg_attn_bwd_cross_workspace_bytes) fits
 * in the array it is used as is, and results are bitwise those of
 * mg_attn_bwd_cross; otherwise the workspace is D alone (B*H*Lq f32,
 * rounded up to 256 bytes) and dQ comes from the separate query-stationary
 * pass, which agrees with the partial-sum path within the contract's
 * tolerance.  MG_ERR_WORKSPACE when even D does not fit
 * (B*H*Lq > MG_ATTN_NOALLOC_SCRATCH_BYTES / 4).  The array is not cleared
 * between calls and nothing in it needs to be: every call writes what it
 * reads.  Every call on one device shares that device's array, so calls
 * that overlap in time on one device (other streams, other threads) race
 * and must be serialized by the caller.
 */
#define MG_ATTN_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

mg_status_t mg_attn_bwd_noalloc(const void *Q, const void *K, const void *V,
                                const void *O, const float *LSE, const void *dO,
                                void *dQ, void *dK, void *dV,
                                const int32_t *key_len,
                                int B, int H, int Lq, int Lk, int d, int causal, float scale,
                                mg_contract_t contract, hipStream_t stream);

/* Static, human-readable name of a status code. */
const char *mg_status_string(mg_status_t status);

/* Message describing the last failing call on the calling thread ("" if the
 * last call succeeded).  Valid until the next call on that thread. */
const char *mg_last_error_detail(void);

/*
 * Kernel timing for measurement tools (not needed for computation).  While
 * enabled, every kernel the library launches is bracketed by a pair of HIP
 * events recorded on the launch stream.  mg_profile_collect waits for the
 * recorded events, adds each kernel's durations to per-kernel totals, and
 * copies up to `max_entries` totals (name, launches, total milliseconds)
 * into the caller's arrays; it returns the number of distinct kernels
 * (which may exceed max_entries) or -1 on a HIP error.  mg_profile_reset
 * clears the totals.  Enabling and collecting are process-wide and
 * serialized by a mutex; events are created lazily and reused.
 */
mg_status_t mg_profile_enable(int enable);
int mg_profile_collect(const char **names, int64_t *launches, double *total_ms,
                       int max_entries);
void mg_profile_reset(void);

/*
 * Sustained matrix-core throughput of the current device, for reading the
 * roofline fractions against what the chip delivers at its running clock
 * (the published dense peaks assume 2.4 GHz).  Runs a kernel of independent
 * MFMA accumulator chains (no memory traffic, eight waves per SIMD, on
 * every CU) for `iters` steps on `stream`, after a warm-up launch of
 * iters/8 steps, and WAITS for it (unlike every other call here); *tflops
 * receives the achieved dense TFLOP/s.  kind: 0 = f32
 * (v_mfma_f32_16x16x4_f32, eight chains per wave), 1 = bf16 and 2 = f16
 * (v_mfma_f32_32x32x16_{bf16,f16}, four chains per wave).  iters in
 * [1, 2^24].  Allocates nothing; events are created and destroyed inside.
 */
mg_status_t mg_mfma_peak(int kind, int iters, double *tflops, hipStream_t stream);

/*
 * LDS read cost of one access pattern, for choosing the row strides of the
 * kernels' LDS tiles (a measuring tool, like mg_mfma_peak; synchronous).
 * Every wave of two 4-wave workgroups per CU issues `iters` x 8 reads of the
 * pattern back to back; *clocks receives the shader clocks one read
 * instruction costs a CU (its waves share the LDS), from the waves' own
 * clock counters.  A 16-byte read of 64 lanes moves 1 KB, so 4 clocks is
 * 256 bytes per clock, the conflict-free rate.  `row_bytes` (a multiple of
 * 16 in [16, 480]) is the row stride of the tile the pattern reads; lane l:
 *   0: 16-byte read, row l%16, chunk l/16        (16x16x32 operand rows)
 *   1: 16-byte read, row l%16, byte 64*(l/16)    (16x16x4 f32 operand groups)
 *   2: 16-byte read, row l%32, chunk l/32        (32x32x16 operand rows)
 *   3: 8-byte transpose read, row 4*(l/16) + (l%16)/4, byte 8*(l%4)
 *      (16x16x32 products over the tile's rows)
 *   4: 8-byte transpose read, row 4*(l/32) + (l%16)/4,
 *      byte 32*((l/16)%2) + 8*(l%4)               (32x32x16 products)
 *   5: 16-byte read at byte 16*l                   (contiguous reference)
 *   6: 4-byte read, row 4*(l/16), word l%16      (f32 products over rows)
 * Patterns 7..11 read the bf16 kernels' tiles themselves: [64][128] bf16
 * stored as column blocks of 32 (64-byte rows) or 64 columns (128-byte
 * rows), whose 16-byte chunks are permuted per row (chunk j of row r at
 * j ^ swz(r)); `row_bytes` must be that block row (128 for 11 and 16, else
 * 64):
 *   7: 16-byte read, row l%16, columns 8*(l/16)..+7, swz = (r/2)%4
 *      (dK/dV Q and dO tiles)
 *   8: transpose read of the same tile, row 4*(l/16) + (l%16)/4, columns
 *      4*(l%4)..+3
 *   9: 16-byte read, row l%32, columns 8*(l/32)..+7, swz = (r/4)%4
 *      (forward K, dQ K and V)
 *  10: transpose read of that tile, row 4*(l/32) + (l%16)/4, columns
 *      16*((l/16)%2) + 4*(l%4)..+3                (dQ K^T)
 *  11: as 10 on 64-column blocks, swz = 4*((r/2)%2) (forward V^T)
 *  12..16: patterns 7..11 with no chunk permutation (swz = 0).
 * Patterns 17 and 18 read the strict f32 forward's d = 64 tiles: 256-byte
 * rows whose 16-byte chunk j of row r sits at j ^ (r % 16); `row_bytes` must
 * be 256:
 *  17: 16-byte read, row l%16, floats 16*(l/16)..+3  (K, 16x16x4 operands)
 *  18: 4-byte read, row 4*(l/16), float l%16        (V, products over rows)
 * Allocates nothing.
 */
mg_status_t mg_lds_probe(int pattern, int row_bytes, int iters, double *clocks,
                         hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* MG_ATTN_H */
