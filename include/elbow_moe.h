/*
 * elbow_moe.h - C ABI of the elbow-routed MoE layer for AMD MI355X (gfx950).
 *
 * The layer (Section 2 of "Elbow-based MoE Routing: A Training-Free Inference Time Plugin
 * for Expert Selection"): for each token, router logits l = W_r x, probabilities
 * p = softmax(l), the probabilities sorted in descending order, a Kneedle-style elbow
 * index e on that sorted curve (Appendix A.1, Algorithm 1), the expert count
 * k = min(e + 1, K) capped at the model's top-K (Section 2.1), and the output
 * y = sum_{j<k} w_j FFN_{id_j}(x) over the selected experts, FFN being a bias-free SwiGLU
 * MLP.  Fixed top-K routing (the paper's baseline) runs through the same path.
 *
 * Conventions for every entry point:
 *  - All tensor pointers are DEVICE pointers owned by the caller; row-major, densely packed.
 *    The library never allocates, frees or synchronises device memory; scratch space
 *    comes only from the caller's workspace, which must be 256-byte aligned (as hipMalloc
 *    and torch allocations are).  Nothing is retained between calls.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).  Kernels are
 *    enqueued on it and the call returns without waiting for them.
 *  - Arguments are validated on the host BEFORE anything is enqueued.  On any error
 *    nothing is launched and nothing is written.  T = 0 is valid and enqueues nothing.
 *  - Return value: ELB_OK (0) or one of the ELB_ERR_* codes below; elb_last_error()
 *    gives a message for the last failing call of the calling thread.
 *  - Calls on the same stream are ordered; concurrent calls on different streams must not
 *    share output or workspace buffers.
 *  - Inputs must be finite, except that -inf logits are allowed when each row has at
 *    least one finite logit.  NaN inputs give unspecified (but in-bounds) results.
 *
 * Data types: ELB_F32 tensors are float; ELB_BF16 tensors are bfloat16 (uint16 storage,
 * round-to-nearest-even).  Router logits, routing weights and all accumulation are fp32.
 */
#ifndef ELBOW_MOE_H
#define ELBOW_MOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ELB_ABI_VERSION 1

/* Largest supported expert count N and cap K (any cap up to N: K = N is the uncapped
   elbow routing). */
#define ELB_MAX_EXPERTS 64
#define ELB_MAX_K 64

typedef enum {
    ELB_OK = 0,
    ELB_ERR_INVALID_ARG = 1, /* null pointer, negative size, K outside [1, N], eps < 0, ... */
    ELB_ERR_UNSUPPORTED = 2, /* a size outside what the kernels implement (e.g. N > 64) */
    ELB_ERR_WORKSPACE = 3,   /* workspace missing, not 256-byte aligned or smaller than
                                elb_*_workspace_bytes */
    ELB_ERR_HIP = 4          /* a HIP launch error (hipGetLastError after the launch) */
} elb_status;

typedef enum { ELB_F32 = 0, ELB_BF16 = 1 } elb_dtype;

typedef enum {
    ELB_MODE_ELBOW = 0, /* k = min(e + 1, K), Algorithm 1 with the cap of Section 2.1 */
    ELB_MODE_TOPK = 1   /* k = K: the fixed top-K routing the method prunes */
} elb_mode;

typedef struct {
    int32_t K;           /* cap: the model's top-K (8 for OLMoE); 1 <= K <= min(N, ELB_MAX_K) */
    float eps;           /* the normaliser's epsilon of Algorithm 1 (default 1e-8); >= 0 */
    int32_t mode;        /* elb_mode */
    int32_t renormalize; /* 0: w_j = p_(j) (full-softmax probability); 1: w_j = p_(j) /
                            sum_{i<k} p_(i) */
} elb_route_params;

/* ABI version (ELB_ABI_VERSION of the built library). */
int elb_abi_version(void);

/* Static description of a status code. */
const char *elb_status_str(int status);

/* Message of the last failing call on the calling thread ("" if none). */
const char *elb_last_error(void);

/*
 * Router logits (Section 2: a learned router produces logits l(x) in R^N per token).
 *   x        [T, d]  dtype            token activations
 *   W_router [N, d]  dtype            router weight (nn.Linear layout, no bias)
 *   logits   [T, N]  float (output)   l = x W_router^T, fp32 accumulation
 * Requirements: 2 <= N <= ELB_MAX_EXPERTS, d >= 1 (d % 32 == 0 for ELB_BF16).
 */
int elb_router_logits(const void *x, const void *W_router, int64_t T, int32_t d, int32_t N,
                      int32_t dtype, float *logits, void *stream);

/*
 * Routing (Section 2 and 2.1; Appendix A.1 Algorithm 1).  Per token:
 *   p = softmax(l); sort p descending (equal logits: lower expert id first);
 *   p'_i = (p_(0) - p_(i)) / (p_(0) - p_(N-1) + eps),  x'_i = i / (N - 1),
 *   D_i = p'_i - x'_i,  e = smallest index maximising D,  k = min(e + 1, K)
 *   (ELB_MODE_TOPK: k = K).
 * The normalised curve runs from (0,0) to (1,1), the orientation of the paper's elbow
 * angle (Section 2.3); D_i is the depth of sorted point i below the chord.
 *   logits [T, N] float   input
 *   k      [T]    int32   output, 1 <= k <= K
 *   ids    [T, K] int32   output, expert ids in descending-probability order; -1 for j >= k
 *   w      [T, K] float   output, weights (see elb_route_params.renormalize); 0 for j >= k
 * Requirements: 2 <= N <= ELB_MAX_EXPERTS; params valid.
 */
int elb_route(const float *logits, int64_t T, int32_t N, const elb_route_params *params,
              int32_t *k, int32_t *ids, float *w, void *stream);

/*
 * Router and routing fused (elb_router_logits followed by elb_route, in one kernel): each
 * block computes the logits of 16 tokens on the matrix cores, keeps them in LDS and routes
 * them there with the routing kernel's own per-token code, so k, ids and w are bit-identical
 * to the two-step path and the logits need not be written to memory.
 *   x, W_router          as elb_router_logits (ELB_BF16 only, d % 32 == 0)
 *   params               as elb_route, with K <= 16
 *   logits_out [T, N]    float output, or NULL to skip writing the logits
 *   k, ids, w            as elb_route
 * Other dtypes or caps: ELB_ERR_UNSUPPORTED (use the two calls).
 */
int elb_router_route(const void *x, const void *W_router, int64_t T, int32_t d, int32_t N,
                     int32_t dtype, const elb_route_params *params, float *logits_out,
                     int32_t *k, int32_t *ids, float *w, void *stream);

/*
 * Tail randomisation (Section 2.2): the elbow's k = min(e + 1, K) experts, as elb_route
 * selects them, followed by K - k further experts drawn uniformly without replacement from
 * the N - k experts outside that selection, so every token uses exactly K experts.  The draw
 * is the caller's: `rand[t, c]` is a uniform sample for expert c of token t, and the tail is
 * the K - k unselected experts with the smallest draws, in increasing draw order (equal
 * draws: lower expert id first).  With i.i.d. uniform draws this is a uniform draw without
 * replacement; the caller owns the random stream, so results are reproducible.
 *   logits  [T, N] float   input
 *   rand    [T, N] float   input, the draws (any finite values; only their order matters)
 *   k_elbow [T]    int32   output, the elbow's k (1 <= k <= K)
 *   ids     [T, K] int32   output, the elbow's experts in descending-probability order,
 *                          then the tail in increasing draw order; never -1
 *   w       [T, K] float   output, each expert's own full-softmax probability, or with
 *                          params->renormalize the probability over the K selected experts
 * Requirements as elb_route; params->mode = ELB_MODE_TOPK gives k = K and no tail.
 */
int elb_route_tail_random(const float *logits, const float *rand, int64_t T, int32_t N,
                          const elb_route_params *params, int32_t *k_elbow, int32_t *ids,
                          float *w, void *stream);

/*
 * Elbow angle (Section 2.3): the angle at the elbow point P_e = (x'_e, p'_e) of the
 * normalised sorted curve between the vectors to its ends (0,0) and (1,1),
 *   theta = arccos(v1 . v2 / (|v1| |v2|)),  v1 = -P_e,  v2 = (1,1) - P_e,
 * in degrees; small angles mark sharp elbows (confident routing), angles near 180 a curve
 * close to the chord.  e is the uncapped elbow index of elb_route (before min(e + 1, K));
 * when no point has D_i > 0, e = 0 and theta is taken as 180 (a straight curve).
 * Every elbow point lies in the unit square, inside the circle whose diameter is the chord
 * from (0,0) to (1,1), so 90 <= theta <= 180.
 *   logits [T, N] float   input
 *   e      [T]    int32   output, 0 <= e <= N - 1 (may be NULL)
 *   theta  [T]    float   output, degrees (may be NULL)
 * Requirements: 2 <= N <= ELB_MAX_EXPERTS; eps >= 0 and finite.
 */
int elb_elbow_angle(const float *logits, int64_t T, int32_t N, float eps, int32_t *e,
                    float *theta, void *stream);

/*
 * Variable-k dispatch: expert-major token lists built from a routing (deterministic:
 * within an expert, rows are in increasing token order).
 *   k, ids            [T], [T, K]   a routing as written by elb_route
 *   counts    [N]     int32 output  assignments per expert, sum = sum_t k_t
 *   offsets   [N + 1] int32 output  exclusive prefix sum of counts (offsets[N] = sum k)
 *   row_token [T * K] int32 output  row r of the expert-major order holds token
 *                                   row_token[r]; rows >= offsets[N] are left untouched
 *   inv       [T, K]  int32 output  row of (t, j) for j < k_t, -1 otherwise
 *   workspace          device scratch of at least elb_dispatch_workspace_bytes(T, N) bytes
 */
size_t elb_dispatch_workspace_bytes(int64_t T, int32_t N);
int elb_dispatch(const int32_t *k, const int32_t *ids, int64_t T, int32_t N, int32_t K,
                 int32_t *counts, int32_t *offsets, int32_t *row_token, int32_t *inv,
                 void *workspace, size_t workspace_bytes, void *stream);

/*
 * Expert part of the layer for a given routing: dispatch, the grouped SwiGLU expert
 * GEMMs and the weighted combine, in rank order with fp32 accumulation:
 *   y_t = [residual_t +] sum_{j<k_t} w_tj FFN_{ids_tj}(x_t),
 *   FFN_e(x) = W_down[e] (silu(W_gate[e] x) * (W_up[e] x)),  silu(z) = z / (1 + e^-z).
 *   x         [T, d]      dtype
 *   W_gate_up [N, 2m, d]  dtype   rows [0, m) = W_gate[e], rows [m, 2m) = W_up[e]
 *   W_down    [N, d, m]   dtype
 *   k, ids, w             a routing ([T], [T, K], [T, K]) as written by elb_route
 *   residual  [T, d]      dtype   optional (NULL: none)
 *   y         [T, d]      dtype   output; may alias residual, must not alias x
 *   workspace             at least elb_moe_workspace_bytes(T, d, N, m, K, dtype) bytes
 * Requirements: 2 <= N <= ELB_MAX_EXPERTS; 1 <= K <= min(N, ELB_MAX_K);
 * ELB_BF16: d % 64 == 0 and m % 64 == 0; ELB_F32: d % 16 == 0 and m % 16 == 0.
 */
size_t elb_moe_workspace_bytes(int64_t T, int32_t d, int32_t N, int32_t m, int32_t K,
                               int32_t dtype);
int elb_moe_experts(const void *x, const void *W_gate_up, const void *W_down,
                    const int32_t *k, const int32_t *ids, const float *w, const void *residual,
                    int64_t T, int32_t d, int32_t N, int32_t m, int32_t K, int32_t dtype,
                    void *y, void *workspace, size_t workspace_bytes, void *stream);

/*
 * The whole layer: elb_router_logits and elb_route (fused as in elb_router_route for bf16 and
 * K <= 16; with N = 64 the router's contraction is split into four quarters, whose partial
 * logits are summed in a fixed order before the routing -- one launch up to 4096 tokens when
 * d % 256 == 0, two above or for other d; every form gives the same bits), then
 * elb_moe_experts, on one stream, with no host round trip.  Arguments as above; the optional debug outputs (NULL to
 * skip) receive the intermediate results of this call:
 *   logits_out [T, N] float, k_out [T], ids_out [T, K], w_out [T, K],
 *   counts_out [N] int32 (assignments per expert).
 * With T = 0 nothing is launched and no output (counts_out included) is written.
 */
int elb_moe_forward(const void *x, const void *W_router, const void *W_gate_up,
                    const void *W_down, const void *residual, int64_t T, int32_t d, int32_t N,
                    int32_t m, int32_t dtype, const elb_route_params *params, void *y,
                    void *workspace, size_t workspace_bytes, float *logits_out,
                    int32_t *k_out, int32_t *ids_out, float *w_out, int32_t *counts_out,
                    void *stream);

/*
 * The whole layer (elb_moe_forward) without a caller workspace and without any allocation,
 * for callers that cannot allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  Scratch comes from a static device array of
 * ELB_NOALLOC_SCRATCH_BYTES per GPU (256 MiB, held by every GPU the library runs on until the
 * process ends; its address is looked up once per device, on the first call there, with the
 * stream's device current).  The caller still passes inputs and outputs, as for
 * elb_moe_forward, whose kernels and results (bit for bit) this call shares.
 * Limits and behaviour:
 *  - a problem whose elb_moe_workspace_bytes(T, d, N, m, K, dtype) exceeds
 *    ELB_NOALLOC_SCRATCH_BYTES is rejected with ELB_ERR_UNSUPPORTED before anything is
 *    enqueued (the OLMoE-shaped layer, d = 2048, N = 64, m = 1024, K = 8, fits up to 5307
 *    tokens);
 *  - nothing in the scratch has to start at zero, and nothing is cleared;
 *  - every call on one GPU uses that GPU's one array, so calls that overlap in time on one
 *    GPU (different streams, or different host threads) race and must be serialised by the
 *    caller; calls in order on one stream are safe;
 *  - with elb_profile_enable(1) the library creates timing events; leave profiling off where
 *    no allocation of any kind is allowed.
 */
#define ELB_NOALLOC_SCRATCH_BYTES ((size_t)256 << 20)
int elb_moe_forward_noalloc(const void *x, const void *W_router, const void *W_gate_up,
                            const void *W_down, const void *residual, int64_t T, int32_t d,
                            int32_t N, int32_t m, int32_t dtype, const elb_route_params *params,
                            void *y, float *logits_out, int32_t *k_out, int32_t *ids_out,
                            float *w_out, int32_t *counts_out, void *stream);

/*
 * Packed expert weights for decode-sized batches.  When an expert gets at most 16 rows on
 * average (T K <= 16 N), the expert GEMMs are bound by reading the weights; the layer then
 * streams each expert's weights in 64-row tasks.  elb_pack_expert_weights writes a copy of
 * W_gate_up and W_down in exactly that streaming order (per task, stage and MFMA operand, the
 * 64 lanes' 16-byte pieces contiguous), so that every load reads 1 KB contiguous; it is done
 * once, outside the per-call path.  The packed copy has the size of the two weight tensors
 * together (elb_packed_expert_bytes), is bf16 only (d % 64 == 0, m % 64 == 0) and is valid
 * until the weights change.
 *   W_gate_up [N, 2m, d], W_down [N, d, m]   bf16 input (as for elb_moe_experts)
 *   packed                                   device output, elb_packed_expert_bytes bytes
 * elb_moe_experts_packed / elb_moe_forward_packed are elb_moe_experts / elb_moe_forward with
 * that copy as an extra argument: the decode-sized kernels read it, every other path reads
 * W_gate_up and W_down as usual (so both are still required).  Results are bit-identical to
 * the unpacked calls.
 */
size_t elb_packed_expert_bytes(int32_t N, int32_t d, int32_t m);
int elb_pack_expert_weights(const void *W_gate_up, const void *W_down, int32_t N, int32_t d,
                            int32_t m, int32_t dtype, void *packed, void *stream);
int elb_moe_experts_packed(const void *x, const void *W_gate_up, const void *W_down,
                           const void *packed, const int32_t *k, const int32_t *ids,
                           const float *w, const void *residual, int64_t T, int32_t d,
                           int32_t N, int32_t m, int32_t K, int32_t dtype, void *y,
                           void *workspace, size_t workspace_bytes, void *stream);
int elb_moe_forward_packed(const void *x, const void *W_router, const void *W_gate_up,
                           const void *W_down, const void *packed, const void *residual,
                           int64_t T, int32_t d, int32_t N, int32_t m, int32_t dtype,
                           const elb_route_params *params, void *y, void *workspace,
                           size_t workspace_bytes, float *logits_out, int32_t *k_out,
                           int32_t *ids_out, float *w_out, int32_t *counts_out, void *stream);

/*
 * Calibration of the matrix-core roofline (a measurement aid, not part of the layer): a
 * kernel of `blocks` blocks of 4 waves, each wave issuing iters x 8 back-to-back
 * v_mfma_f32_32x32x16_bf16 instructions (32 x 32 x 16 multiply-adds each) on register
 * operands, with no memory traffic.  Timing it gives the bf16 MFMA rate the chip sustains,
 * clock and power included.
 *   out [blocks * 4] float   device output (one sum per wave, so the work is kept)
 * Returns the number of MFMA instructions enqueued (> 0), or a negative elb_status.
 */
int64_t elb_calibrate_mfma_bf16(int32_t blocks, int32_t iters, float *out, void *stream);

/*
 * Calibration of the HBM read roofline (a measurement aid, not part of the layer): `blocks`
 * blocks of 4 waves read the whole of buf once, each block its own contiguous share, with
 * coalesced non-temporal 16-byte loads (sixteen in flight per lane), and fold the words into
 * one per wave.
 * Timing it over a buffer larger than the last-level cache gives the read rate the chip
 * sustains.
 *   buf   [bytes] device memory, 16-byte aligned; bytes a positive multiple of 16 (read only)
 *   out   [blocks * 4] uint32 device output (one word per wave, so the reads are kept)
 * Returns ELB_OK or an elb_status; nothing is allocated.
 */
int elb_calibrate_read_stream(const void *buf, int64_t bytes, int32_t blocks, uint32_t *out,
                              void *stream);

/*
 * Per-kernel timing (hipEvents attached to each launch the library makes).
 * elb_profile_enable(1) starts recording on the calling process for every launch,
 * elb_profile_enable(2) for the grouped expert GEMMs only, elb_profile_enable(0) stops; a
 * recorded launch carries a start/stop event pair in its own dispatch
 * (hipExtLaunchKernelGGL).  Timed launches run measurably slower than untimed back-to-back
 * ones (on MI355X the large expert GEMMs by about 10 %), so per-kernel figures from this
 * are upper bounds.  elb_profile_read() synchronises on the
 * recorded events, fills up to `cap` entries of names (static strings), total
 * milliseconds and launch counts per kernel, clears the records and returns the number
 * of kernels (or a negative elb_status).  Not for use under graph capture.
 */
int elb_profile_enable(int on);
int elb_profile_read(const char **names, double *total_ms, int64_t *launches, int cap);

#ifdef __cplusplus
}
#endif

#endif /* ELBOW_MOE_H */
