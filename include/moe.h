/*
 * moe.h -- C ABI of one routed Mixture-of-Experts layer on one MI355X (gfx950).
 *
 * The layer is the per-token data path of a routed MoE layer as the paper
 * trains it (Section 5.2: token dispatch, grouped-GEMM experts, fused
 * permutation): router logits -> top-K routing -> dispatch of hidden states
 * and routed probabilities into an expert-contiguous buffer -> per-expert
 * FFN -> probability-weighted combine back to token order, plus the
 * backward pass through the experts and the permutation.  On one GPU the
 * expert-parallel all-to-alls of the paper become the local dispatch and
 * combine copies; their payloads are exactly what Eq. 1 counts.
 *
 * Notation (Section 1, Eq. 1; Table 2):
 *   S  tokens in this call (sequence length x micro-batch, flattened)
 *   D  dispatch dimension (hidden width of what is dispatched)
 *   E  routed experts;  K  experts per token (top-K);  R = S*K routed rows
 *   F  per-expert FFN width (f_expert);  H  model hidden when a latent
 *      projection precedes dispatch (d_latent = D)
 *   b_x = 2 (bf16 hidden elements),  b_p = 4 (fp32 routed probabilities)
 *
 * Conventions for every entry point:
 *   - Tensor pointers are DEVICE pointers to row-major, contiguous arrays.
 *     bf16 arrays and the probability arrays must be 16-byte aligned;
 *     int32 arrays 4-byte aligned.
 *   - The caller allocates and frees every buffer, including the workspace
 *     sized by the matching *_workspace_bytes query.  The library never
 *     allocates, frees or synchronises; it keeps no state between calls.
 *   - Work is enqueued on `stream` (NULL = the null stream) and the call
 *     returns at once.  Arguments are validated synchronously before any
 *     launch; on a validation error nothing is enqueued.
 *   - Outputs must not alias inputs.  Results are deterministic: the same
 *     inputs give bit-identical outputs on every call.
 *   - S == 0 (or R == 0) is valid and enqueues nothing.
 *   - Every entry point enqueues kernels only (no allocation, copy, memset or
 *     host synchronisation), so a call made while `stream` is being captured
 *     records the whole call into the graph; replays read the buffers' contents
 *     at replay time.
 *   - Debugging only: with MOE_DEBUG_SYNC=1 in the environment (read once per
 *     process) every launch is followed by a synchronisation of `stream` and
 *     an error check, so a kernel fault is reported as MOE_ERR_HIP by the
 *     entry point that enqueued it; a stream under graph capture is not
 *     synchronised.  Off by default.
 *   - Limits: 1 <= E <= 1024, 1 <= K <= min(E, 32), D and F multiples of 8
 *     in [8, 65536], S*K < 2^31.  The grouped GEMM copies its
 *     operands through range-checked buffer descriptors of at most 2^31
 *     bytes, so one expert's weight (D*F*2 bytes; H*D*2 for the latent
 *     projections) and, for the weight gradients, S*K*max(D, F)*2 must stay
 *     below 2^31; larger requests return MOE_ERR_UNSUPPORTED.
 */
#ifndef MOE_H
#define MOE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MOE_ABI_VERSION 5

typedef uint16_t moe_bf16; /* bit pattern of a bfloat16 value (b_x = 2 bytes) */

typedef enum {
    MOE_OK = 0,
    MOE_ERR_NULL = -1,        /* a required pointer is NULL */
    MOE_ERR_SHAPE = -2,       /* a size is out of range or inconsistent */
    MOE_ERR_ALIGN = -3,       /* a pointer violates its alignment */
    MOE_ERR_WORKSPACE = -4,   /* workspace missing or smaller than required */
    MOE_ERR_HIP = -5,         /* a HIP launch failed (see hipGetLastError) */
    MOE_ERR_UNSUPPORTED = -6  /* valid request this build does not implement */
} moe_status;

/* ABI version of the loaded library (MOE_ABI_VERSION at build time). */
int moe_abi_version(void);

/* Static, human-readable text for a moe_status value. Never NULL. */
const char* moe_status_string(int status);

/* Forward dispatch payload in bytes, S*K*(D*b_x + b_p): every routed row
 * carries its bf16 hidden state and its fp32 routed probability (Eq. 1).
 * Returns 0 for negative sizes. Host-only, touches no device. */
uint64_t moe_payload_bytes(int64_t S, int32_t K, int32_t D);

/* ---------------------------------------------------------------------- */
/* Router logits (the router scores every token against every expert,     */
/* Section 5.2).                                                          */
/* ---------------------------------------------------------------------- */
/* Workspace bytes moe_router_logits needs (3 * E * D * 2 rounded up to
 * 256: the router weight split into three bf16 planes); 0 for invalid sizes. */
size_t moe_router_logits_workspace_bytes(int32_t D, int32_t E);

/* logits[t,e] = sum_d x_r[t,d] * Wr[d,e] + bias[e], accumulated in fp32.
 *   x_r    [S, D]  bf16   router input (the dispatch-width activations)
 *   Wr     [D, E]  fp32   router weight (4-byte aligned)
 *   bias   [E]     fp32   per-expert logit offset, or NULL for none
 *   logits [S, E]  fp32   output
 *   ws, ws_bytes          device scratch of at least
 *                         moe_router_logits_workspace_bytes(D, E) bytes,
 *                         16-byte aligned; overwritten by the call.
 * Each fp32 weight is used as the sum of three bf16 terms (its bf16
 * rounding and the bf16 roundings of the two successive remainders), which
 * equals it to within 2^-24 relative, so the logits carry fp32 accuracy.
 * Errors: MOE_ERR_SHAPE (S < 0, D not a multiple of 8 in [8, 65536], E not
 * in [1, 1024]), MOE_ERR_NULL / MOE_ERR_ALIGN for missing or misaligned
 * buffers, MOE_ERR_WORKSPACE for a missing or short ws. */
int moe_router_logits(const moe_bf16* x_r, const float* Wr, const float* bias,
                      int64_t S, int32_t D, int32_t E, float* logits,
                      void* ws, size_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------- */
/* Top-K routing and the expert permutation (dropless, unpadded top-K     */
/* routing, Section 1; fused permutation, Section 5.2).                   */
/* ---------------------------------------------------------------------- */
/* Workspace bytes moe_route_topk needs for these sizes. */
size_t moe_route_workspace_bytes(int64_t S, int32_t E, int32_t K);

/* Per token t, over the fp32 scores s = logits[t, :]:
 *   topk_idx[t, 0..K-1]  the K best experts, best first, under the order
 *                        (score descending, expert index ascending); -0 == +0
 *                        and NaN ranks below -inf;
 *   topk_prob[t, k]      softmax over all E, restricted to the K picked and
 *                        renormalised to sum to 1 (fp32).  Each token needs a
 *                        finite best score; otherwise its probabilities are
 *                        unspecified (indices stay well defined).
 * Over all tokens:
 *   counts[e]            routed rows per expert, sum = S*K
 *   offsets[e]           exclusive prefix sum of counts, offsets[E] = S*K
 *   perm[pos]            = t*K+k of the row stored at position pos of the
 *                        expert-contiguous order (experts ascending, tokens
 *                        ascending inside an expert)
 *   inv_perm[t*K+k]      = pos  (perm and inv_perm are inverse bijections)
 * Shapes: logits [S,E] fp32; topk_idx, perm, inv_perm int32; topk_prob fp32;
 * counts [E], offsets [E+1] int32.  ws: >= moe_route_workspace_bytes, 16-byte
 * aligned, contents need no initialisation. */
int moe_route_topk(const float* logits, int64_t S, int32_t E, int32_t K,
                   int32_t* topk_idx, float* topk_prob, int32_t* counts, int32_t* offsets,
                   int32_t* perm, int32_t* inv_perm, void* ws, size_t ws_bytes,
                   hipStream_t stream);

/* ---------------------------------------------------------------------- */
/* Dispatch: the forward dispatch payload of Eq. 1 (D*b_x + b_p per row).  */
/* ---------------------------------------------------------------------- */
/* x_disp[inv_perm[t*K+k], :] = x[t, :]   (bf16 copy, bit-exact)
 * p_disp[inv_perm[t*K+k]]    = topk_prob[t, k]   (fp32 copy)
 * topk_prob and p_disp may both be NULL to move hidden states only.
 *   x [S, D] bf16;  inv_perm [S*K] int32;  x_disp [S*K, D] bf16;  p_disp [S*K] fp32 */
int moe_dispatch(const moe_bf16* x, const float* topk_prob, const int32_t* inv_perm,
                 int64_t S, int32_t D, int32_t K, moe_bf16* x_disp, float* p_disp,
                 hipStream_t stream);

/* ---------------------------------------------------------------------- */
/* Grouped expert FFN (grouped GEMM over expert segments, Section 5.2).    */
/* ---------------------------------------------------------------------- */
/* Workspace bytes moe_grouped_ffn needs. */
size_t moe_grouped_ffn_workspace_bytes(int32_t E, int64_t R, int32_t D, int32_t F);

/* For every expert e and row r in [offsets[e], offsets[e+1]):
 *   u[r]      = x_disp[r, :] @ W1[e]          (fp32 accumulation)
 *   h[r]      = bf16(max(u[r], 0)^2)          squared-ReLU, ungated
 *   y_disp[r] = bf16(h[r] @ W2[e])            (fp32 accumulation)
 *   x_disp [R, D] bf16;  offsets [E+1] int32 on the device (as produced by
 *   moe_route_topk, offsets[E] == R);  W1 [E, D, F] bf16;  W2 [E, F, D] bf16;
 *   h [R, F] bf16 (output, also the down-projection input);
 *   u_save [R, F] bf16 pre-activation kept for the backward pass, or NULL;
 *   y_disp [R, D] bf16 output (unweighted expert outputs). */
int moe_grouped_ffn(const moe_bf16* x_disp, const int32_t* offsets, int32_t E, int64_t R,
                    int32_t D, int32_t F, const moe_bf16* W1, const moe_bf16* W2,
                    moe_bf16* h, moe_bf16* u_save, moe_bf16* y_disp,
                    void* ws, size_t ws_bytes, hipStream_t stream);

/* moe_grouped_ffn without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  The call allocates nothing: its only
 * scratch, the grouped GEMM's tile schedule, lives in a fixed device array of
 * MOE_STATIC_SCRATCH_BYTES that the library holds on each GPU it runs on until
 * the process ends.  Outputs and their meaning are those of moe_grouped_ffn
 * (the same kernels: the results are bit-identical).
 * Limit: R < 2^21 rows (with E <= 1024, the schedule then fits the array);
 * larger R returns MOE_ERR_WORKSPACE before anything is enqueued.
 * Every call on one GPU shares that GPU's array: calls that overlap on one
 * GPU (on different streams, or from different threads) race and must be
 * ordered by the caller.  The array needs no initialisation: each call
 * rewrites the schedule it reads. */
#define MOE_STATIC_SCRATCH_BYTES (448 * 1024)
#define MOE_STATIC_MAX_ROWS ((int64_t)1 << 21)
int moe_grouped_ffn_static(const moe_bf16* x_disp, const int32_t* offsets, int32_t E, int64_t R, int32_t D,
                           int32_t F, const moe_bf16* W1, const moe_bf16* W2, moe_bf16* h, moe_bf16* u_save,
                           moe_bf16* y_disp, hipStream_t stream);

/* The two products of moe_grouped_ffn as separate launches (for callers that
 * schedule or time them individually).
 *
 * moe_grouped_schedule builds, on the device, the tile schedule the grouped
 * GEMM reads for expert segments offsets[0..E] over R rows: per-expert counts
 * of 128-row tiles (sched starts with mtile_start[E+1] int32: mtile_start[0] =
 * 0, mtile_start[e+1] = mtile_start[e] + ceil(count[e] / 128)) followed by one
 * entry per tile.  Segments are clamped to [0, R).  sched: device buffer of at
 * least moe_grouped_schedule_bytes(E, R) bytes, 16-byte aligned. */
size_t moe_grouped_schedule_bytes(int32_t E, int64_t R);
int moe_grouped_schedule(const int32_t* offsets, int32_t E, int64_t R, void* sched, size_t sched_bytes,
                         hipStream_t stream);

/* One grouped GEMM over expert segments, one kernel launch:
 *   C[r, :] = epi( A[r, :] @ W[e] ),  r in expert e's segment
 *   A [R, Kd] bf16;  W [E, Kd, N] bf16;  C [R, N] bf16;  sched from
 *   moe_grouped_schedule for the same offsets, E and R.
 *   epilogue 0: C = bf16(acc)                        (down projection)
 *   epilogue 1: C = bf16(max(acc,0)^2), u_save = bf16(acc) if u_save != NULL
 *                                                    (up projection)  */
int moe_grouped_gemm(const moe_bf16* A, const void* sched, int32_t E, int64_t R, int32_t Kd, int32_t N,
                     const moe_bf16* W, int32_t epilogue, moe_bf16* C, moe_bf16* u_save,
                     hipStream_t stream);

/* moe_grouped_gemm with the dispatch fused into its A operand (the
 * permutation fused into the expert GEMM, Section 5.2): row r of expert e's
 * segment is x[perm[r] / K, :] instead of a materialised x_disp row, so
 *   C[r, :] = epi( x[perm[r] / K, :] @ W[e] ),
 * bit-identical to moe_dispatch followed by moe_grouped_gemm on x_disp.
 *   x [S, Kd] bf16 (S * Kd * 2 < 2^31);  perm [R] int32 from moe_route_topk
 *   (R = S * K);  sched, W, epilogue, C, u_save as in moe_grouped_gemm.
 * Errors: as moe_grouped_gemm, plus MOE_ERR_UNSUPPORTED if S * Kd * 2
 * reaches 2^31 and MOE_ERR_SHAPE if R != S * K. */
int moe_grouped_gemm_gather(const moe_bf16* x, const int32_t* perm, int64_t S, int32_t K, const void* sched,
                            int32_t E, int64_t R, int32_t Kd, int32_t N, const moe_bf16* W, int32_t epilogue,
                            moe_bf16* C, moe_bf16* u_save, hipStream_t stream);

/* ---------------------------------------------------------------------- */
/* Combine: probability-weighted sum back to token order (the hidden       */
/* combine of Section 4.1's footnote; D*b_x per routed row, Eq. 1).        */
/* ---------------------------------------------------------------------- */
/* y[t, :] = bf16( sum_{k<K} p_disp[pos] * y_disp[pos, :] ),  pos = inv_perm[t*K+k],
 * accumulated in fp32 in ascending k, no atomics.  p_disp NULL = unit weights.
 *   y_disp [S*K, D] bf16;  p_disp [S*K] fp32 or NULL;  y [S, D] bf16 */
int moe_combine(const moe_bf16* y_disp, const float* p_disp, const int32_t* inv_perm,
                int64_t S, int32_t D, int32_t K, moe_bf16* y, hipStream_t stream);

/* ---------------------------------------------------------------------- */
/* Dense projection for a LatentMoE-style dispatch dimension (Section 1,   */
/* dispatch-dimension lever; Table 2 d_latent).                            */
/* ---------------------------------------------------------------------- */
/* C = bf16(A @ W) with fp32 accumulation.
 *   A [M, Kd] bf16;  W [Kd, N] bf16;  C [M, N] bf16.  Kd, N multiples of 8. */
int moe_latent_proj(const moe_bf16* A, const moe_bf16* W, int64_t M, int32_t Kd, int32_t N,
                    moe_bf16* C, hipStream_t stream);

/* ---------------------------------------------------------------------- */
/* Whole layer forward on one stream, no host synchronisation.             */
/* ---------------------------------------------------------------------- */
typedef struct {
    uint32_t struct_size;      /* sizeof(moe_layer_fwd_args), or MOE_LAYER_FWD_ARGS_BASE_SIZE for a
                                  caller that fills only the fields up to ws_bytes (every later
                                  field then reads as zero / NULL) */
    int64_t S;
    int32_t H;                 /* 0: no latent projection (x is [S, D]) */
    int32_t D, E, K, F;
    const moe_bf16* x;         /* [S, H] if H > 0 else [S, D] */
    const float* Wr;           /* [D, E] fp32 router weight */
    const float* router_bias;  /* [E] fp32 or NULL */
    const moe_bf16* Wdown;     /* [H, D] when H > 0, else NULL */
    const moe_bf16* W1;        /* [E, D, F] */
    const moe_bf16* W2;        /* [E, F, D] */
    const moe_bf16* Wup;       /* [D, H] when H > 0, else NULL */
    moe_bf16* y;               /* [S, H] if H > 0 else [S, D] */
    /* Optional exported intermediates: NULL means "keep in workspace". */
    float* logits;             /* [S, E] */
    int32_t* topk_idx;         /* [S, K] */
    float* topk_prob;          /* [S, K] */
    int32_t* counts;           /* [E] */
    int32_t* offsets;          /* [E+1] */
    int32_t* perm;             /* [S*K] */
    int32_t* inv_perm;         /* [S*K] */
    moe_bf16* x_disp;          /* [S*K, D] */
    float* p_disp;             /* [S*K] */
    moe_bf16* h;               /* [S*K, F] */
    moe_bf16* u_save;          /* [S*K, F] pre-activation; NULL = not saved */
    moe_bf16* y_disp;          /* [S*K, D] */
    void* ws;                  /* workspace, >= moe_layer_fwd_workspace_bytes */
    size_t ws_bytes;
    /* ---- extensions after the base layout (read only when struct_size covers them) ---- */
    moe_bf16* x_lat;           /* [S, D] exported latent router/dispatch input (H > 0 only) */
    moe_bf16* y_lat;           /* [S, D] exported latent combine output (H > 0 only) */
    /* The paper's production variant (Section 5.2); all zero / NULL gives
     * the softmax layer above.  See the production-router section below. */
    int32_t score_fn;          /* MOE_SCORE_SOFTMAX or MOE_SCORE_SIGMOID */
    int32_t Fs;                /* shared-expert width (multiple of 8); 0 = none (H must be 0) */
    const float* sel_bias;     /* [E] selection-only bias (sigmoid scores only) or NULL */
    const moe_bf16* Ws1;       /* [D, Fs] when Fs > 0 */
    const moe_bf16* Ws2;       /* [Fs, D] when Fs > 0 */
    int64_t seq_len;           /* balance loss over sequences of seq_len tokens; 0 = none */
    float aux_coeff;           /* balance-loss coefficient (the paper trains with 1e-4) */
    float* aux_loss;           /* [1] fp32, required when seq_len > 0 */
    int32_t* seq_counts;       /* [S / seq_len, E] routed counts per sequence, or NULL */
    moe_bf16* h_s;             /* [S, Fs] shared-expert activation, or NULL */
    moe_bf16* u_s;             /* [S, Fs] its pre-activation (saved only if given) */
    float* y_s;                /* [S, D] fp32 shared-expert output, or NULL */
    /* Dispatch payload precision (Section 1's precision lever on b_x). */
    int32_t payload;           /* MOE_PAYLOAD_BF16 or MOE_PAYLOAD_MXFP8 (D a multiple of 32) */
    uint8_t* x_q;              /* [S*K, D] MX-FP8 codes, exported or NULL */
    uint8_t* x_scale;          /* [S*K, D/32] their E8M0 block scales, exported (in an allocation
                                  of moe_mx_scale_alloc_bytes(S*K, D) bytes) or NULL */
} moe_layer_fwd_args;

/* Size of the base layout: struct_size for callers that fill only the fields
 * from struct_size through ws_bytes (the plain softmax layer with a bf16
 * payload; a latent layer then keeps x_lat and y_lat in the workspace). */
#define MOE_LAYER_FWD_ARGS_BASE_SIZE offsetof(moe_layer_fwd_args, x_lat)

enum { MOE_PAYLOAD_BF16 = 0, MOE_PAYLOAD_MXFP8 = 1 };

enum { MOE_SCORE_SOFTMAX = 0, MOE_SCORE_SIGMOID = 1 };

/* Workspace bytes moe_layer_fwd needs for these arguments (intermediates the
 * caller does not export are carved from it).  0 if the sizes are invalid. */
size_t moe_layer_fwd_workspace_bytes(const moe_layer_fwd_args* a);

/* [x_lat = bf16(x @ Wdown)] -> logits -> route -> dispatch -> experts ->
 * combine -> [y = bf16(y_lat @ Wup)], all enqueued on `stream`.
 * With the bf16 payload and x_disp not exported, the dispatch is fused into
 * the up projection's operand copy (it gathers each routed row from the
 * router input through perm; the route also writes p_disp), so the
 * dispatched rows are never materialised; the results are bit-identical to
 * the materialised path, which runs when the caller exports x_disp.
 * With payload = MOE_PAYLOAD_MXFP8 the dispatch sends MX-FP8 rows
 * (moe_dispatch_mxfp8) and the up projection reads them as sent
 * (moe_grouped_gemm_mxfp8: the decoded bf16 values, decoded in its operand
 * path); x_disp, if exported, receives the decoded rows (moe_mxfp8_dequant)
 * and is not written otherwise.
 * With score_fn = MOE_SCORE_SIGMOID the route is moe_route_sigmoid (with
 * sel_bias); seq_len > 0 adds moe_seq_aux_loss; Fs > 0 runs the shared
 * expert and adds its fp32 output in the combine, before the one bf16
 * rounding of y (moe_combine_add).  A shared expert with a latent
 * projection (H > 0) returns MOE_ERR_UNSUPPORTED. */
int moe_layer_fwd(const moe_layer_fwd_args* a, hipStream_t stream);

/* ---------------------------------------------------------------------- */
/* Backward through combine, experts and dispatch (the inverse routes of   */
/* the backward pass, Section 4.1 footnote; Eq. 1's factor of 2).          */
/* ---------------------------------------------------------------------- */
/* dy_disp[pos] = bf16(p_disp[pos] * dy[t]),  dp[t,k] = <dy[t], y_disp[pos]> (fp32),
 * pos = inv_perm[t*K+k].  p_disp NULL = unit weights; dp may be NULL.
 *   dy [S, D] bf16;  y_disp [S*K, D] bf16;  dy_disp [S*K, D] bf16;  dp [S, K] fp32 */
int moe_combine_bwd(const moe_bf16* dy, const moe_bf16* y_disp, const float* p_disp,
                    const int32_t* inv_perm, int64_t S, int32_t D, int32_t K,
                    moe_bf16* dy_disp, float* dp, hipStream_t stream);

/* Workspace bytes moe_grouped_ffn_bwd needs (the [R, F] bf16 du, the tile
 * schedule and the experts' order by row count). */
size_t moe_grouped_ffn_bwd_workspace_bytes(int32_t E, int64_t R, int32_t D, int32_t F);

/* Per expert e over its rows (chain rule of moe_grouped_ffn):
 *   du      = bf16( (dy_disp @ W2[e]^T) * 2*max(u_save, 0) )
 *   dx_disp = bf16( du @ W1[e]^T )
 *   dW2[e]  = h^T @ dy_disp      (fp32)
 *   dW1[e]  = x_disp^T @ du      (fp32)
 * Experts with no rows get dW1[e] = dW2[e] = 0.
 *   x_disp, dy_disp, dx_disp [R, D] bf16;  u_save, h [R, F] bf16;
 *   dW1 [E, D, F] fp32;  dW2 [E, F, D] fp32 (fully overwritten). */
int moe_grouped_ffn_bwd(const moe_bf16* x_disp, const moe_bf16* u_save, const moe_bf16* h,
                        const moe_bf16* dy_disp, const int32_t* offsets, int32_t E, int64_t R,
                        int32_t D, int32_t F, const moe_bf16* W1, const moe_bf16* W2,
                        moe_bf16* dx_disp, float* dW1, float* dW2,
                        void* ws, size_t ws_bytes, hipStream_t stream);

/* dx[t] = bf16( sum_{k<K} dx_disp[inv_perm[t*K+k]] ), the transpose of
 * moe_dispatch (an unweighted combine): the K rows are summed in fp32 in
 * ascending k and the sum is rounded once.
 *   dx_disp [S*K, D] bf16;  inv_perm [S*K] int32;  dx [S, D] bf16 */
int moe_dispatch_bwd(const moe_bf16* dx_disp, const int32_t* inv_perm, int64_t S, int32_t D, int32_t K,
                     moe_bf16* dx, hipStream_t stream);

/* moe_dispatch_bwd with an fp32 addend: dx[t] = bf16( sum_k dx_disp[pos_k] +
 * dx_add[t] ), the addend (the router's contribution to the input gradient,
 * moe_router_bwd's dx_r, or the shared expert's) added after the K rows and
 * before the one rounding.  dx_add [S, D] fp32, 16-byte aligned. */
int moe_dispatch_bwd_add(const moe_bf16* dx_disp, const int32_t* inv_perm, const float* dx_add, int64_t S,
                         int32_t D, int32_t K, moe_bf16* dx, hipStream_t stream);

/* ---------------------------------------------------------------------- */
/* Router backward (the learned router of Section 5.2) with the expert     */
/* selection held fixed: top-K is piecewise constant in the scores, so no  */
/* gradient flows through which experts are picked.                        */
/* ---------------------------------------------------------------------- */
/* Workspace bytes moe_router_bwd needs; 0 for invalid sizes. */
size_t moe_router_bwd_workspace_bytes(int64_t S, int32_t D, int32_t E);

/* From the gradient dp[t,k] of the routed probabilities (moe_combine_bwd's
 * dp), with p = topk_prob (the softmax of the K selected scores):
 *   dlogits[t, T_k] = p_k (dp_k - sum_j p_j dp_j),  0 for unselected experts
 *   dWr   = x_r^T dlogits        [D, E] fp32 (fp32 accuracy: dlogits enters
 *                                the MFMA as three bf16 terms)
 *   dbias = sum_t dlogits[t]     [E] fp32, or NULL
 *   dx_r  = dlogits Wr^T         [S, D] fp32 (the K nonzero terms, fp32 FMA),
 *                                or NULL; pass it to moe_dispatch_bwd_add as dx_add
 * Every sum has a fixed order (deterministic).
 *   x_r [S, D] bf16;  Wr [D, E] fp32;  topk_idx, topk_prob, dp [S, K];
 *   dlogits [S, E] fp32 or NULL (then kept in the workspace).
 * Errors: as moe_route_topk's shapes, D a multiple of 8 in [8, 65536],
 * MOE_ERR_UNSUPPORTED if S*max(D, 3E)*2 >= 2^31, MOE_ERR_WORKSPACE. */
int moe_router_bwd(const moe_bf16* x_r, const float* Wr, const int32_t* topk_idx,
                   const float* topk_prob, const float* dp, int64_t S, int32_t D, int32_t E,
                   int32_t K, float* dlogits, float* dWr, float* dbias, float* dx_r,
                   void* ws, size_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------- */
/* Latent projection backward (LatentMoE-style dispatch dimension,         */
/* Section 1; Table 2 d_latent).                                           */
/* ---------------------------------------------------------------------- */
/* Workspace bytes moe_latent_proj_bwd needs for dW; 0 for invalid sizes. */
size_t moe_latent_proj_bwd_workspace_bytes(int64_t M, int32_t Kd, int32_t N);

/* For out = x_in @ W (moe_latent_proj) and its gradient dout:
 *   dx_in = bf16(dout @ W^T)   [M, Kd] bf16, or NULL
 *   dW    = x_in^T @ dout      [Kd, N] fp32 (fixed-order sum over row
 *                              chunks), or NULL
 * Covers both projections: (x_in, W, dout) = (x, Wdown, dx_lat) gives dx and
 * dWdown; (y_lat, Wup, dy) gives dy_lat and dWup.
 *   x_in [M, Kd] bf16 (needed for dW);  W [Kd, N] bf16 (needed for dx_in);
 *   dout [M, N] bf16.
 * Errors: M in [0, 2^31), Kd and N multiples of 8 in [8, 65536],
 * MOE_ERR_UNSUPPORTED if Kd*N*2 or (with dW) M*max(Kd, N)*2 reaches 2^31. */
int moe_latent_proj_bwd(const moe_bf16* x_in, const moe_bf16* W, const moe_bf16* dout,
                        int64_t M, int32_t Kd, int32_t N, moe_bf16* dx_in, float* dW,
                        void* ws, size_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------- */
/* Lower-precision dispatch payload (Section 1: the precision lever on b_x */
/* in Eq. 1).  Format: OCP microscaling (MX) with FP8 E4M3 elements -- per  */
/* block of 32 consecutive elements of a row one E8M0 scale byte s + 127,  */
/* s = floor(log2 max|x|) - 8 clamped to [-127, 127] (all-zero block:      */
/* -127), and per element the E4M3 code nearest to x * 2^-s (ties to even, */
/* saturated to +-448).  b_x becomes 1 + 1/32 bytes.                       */
/* ---------------------------------------------------------------------- */
/* Forward dispatch payload bytes with MX-FP8 hidden elements:
 * S*K*(D + D/32 + 4) (Eq. 1 with b_x = 1 + 1/32, b_p = 4). */
uint64_t moe_mx_payload_bytes(int64_t S, int32_t K, int32_t D);

/* moe_dispatch with the MX-FP8 payload: each token row of x is encoded once
 * (bit-exact to the format above) and its codes and scales are written to
 * the token's K routed rows; p_disp as in moe_dispatch.
 *   x [S, D] bf16 (finite);  x_q [S*K, D] uint8 (8-byte aligned);
 *   x_scale [S*K, D/32] uint8.
 * Errors: as moe_dispatch, plus D % 32 != 0 (MOE_ERR_SHAPE). */
int moe_dispatch_mxfp8(const moe_bf16* x, const float* topk_prob, const int32_t* inv_perm, int64_t S,
                       int32_t D, int32_t K, uint8_t* x_q, uint8_t* x_scale, float* p_disp,
                       hipStream_t stream);

/* Receive side: out = bf16 of the decoded payload (exact; values below
 * bf16's normal range rounded to nearest even).  out [R, D] bf16. */
int moe_mxfp8_dequant(const uint8_t* x_q, const uint8_t* x_scale, int64_t R, int32_t D, moe_bf16* out,
                      hipStream_t stream);

/* Bytes to allocate for R rows of E8M0 scales of D-element rows when the
 * grouped GEMM below reads them: R * D/32 rounded up to a multiple of 4 (it
 * reads whole 4-byte words; the pad bytes are never used).  0 if D is not a
 * positive multiple of 32. */
uint64_t moe_mx_scale_alloc_bytes(int64_t R, int32_t D);

/* moe_grouped_gemm with the MX-FP8 payload as its A operand, decoded inside
 * the operand path (the up projection reading the dispatch payload as sent,
 * with no separate decode pass):
 *   C[r, :] = epi( decode(x_q, x_scale)[r, :] @ W[e] ),  r in expert e's segment
 * where decode is exactly moe_mxfp8_dequant, so C (and u_save) are
 * bit-identical to moe_mxfp8_dequant followed by moe_grouped_gemm.
 *   x_q [R, Kd] uint8 codes (16-byte aligned), Kd a multiple of 32;
 *   x_scale [R, Kd/32] uint8 scales as written by moe_dispatch_mxfp8, in an
 *   allocation of at least moe_mx_scale_alloc_bytes(R, Kd) bytes;
 *   sched, W, epilogue, C, u_save as in moe_grouped_gemm.
 * The codes must be ones the encoder emits (no E4M3 NaN code; scale bytes
 * at most 246), as every payload of moe_dispatch_mxfp8 is.
 * Errors: as moe_grouped_gemm, plus Kd % 32 != 0 (MOE_ERR_SHAPE). */
int moe_grouped_gemm_mxfp8(const uint8_t* x_q, const uint8_t* x_scale, const void* sched, int32_t E, int64_t R,
                           int32_t Kd, int32_t N, const moe_bf16* W, int32_t epilogue, moe_bf16* C,
                           moe_bf16* u_save, hipStream_t stream);

/* ---------------------------------------------------------------------- */
/* The paper's production router and shared expert (Section 5.2): sigmoid  */
/* router scores with a selection-only expert bias, sequence-level         */
/* auxiliary load balancing, and an ungated shared expert whose output is  */
/* added to the combined routed output.  The paper names these parts; the  */
/* formulas are the published sigmoid gating with a selection-only bias    */
/* and its per-sequence balance loss:                                      */
/*   s = sigmoid(logit);  T_t = top-K of s + sel_bias;                     */
/*   g_k = s[T_k] / sum_j s[T_j]  (the routed weight, b_p);               */
/*   loss = coeff / B * sum_b sum_e f_be P_be,  f_be = E/(K T) n_be,       */
/*   P_be = mean over the sequence's tokens of s[t,e] / sum_e' s[t,e'].    */
/* ---------------------------------------------------------------------- */
/* Sigmoid routing: like moe_route_topk (same outputs, same ordering rules
 * on the selection score s + sel_bias computed in fp32, same workspace
 * moe_route_workspace_bytes), with topk_gate = the routed weights g.
 * sel_bias [E] fp32 or NULL (zero).  Rows whose selected scores are all 0
 * (every selected logit -inf) and NaN logits give unspecified weights. */
int moe_route_sigmoid(const float* logits, const float* sel_bias, int64_t S, int32_t E, int32_t K,
                      int32_t* topk_idx, float* topk_gate, int32_t* counts, int32_t* offsets,
                      int32_t* perm, int32_t* inv_perm, void* ws, size_t ws_bytes, hipStream_t stream);

/* Workspace bytes moe_seq_aux_loss needs; 0 for invalid sizes. */
size_t moe_seq_aux_loss_workspace_bytes(int64_t S, int32_t E, int64_t seq_len);

/* The sequence balance loss of the sigmoid scores of `logits` for the
 * routing topk_idx, over the S / seq_len sequences of seq_len tokens:
 *   loss [1] fp32 (fixed-order sums, fp64 across chunks);
 *   seq_counts [S / seq_len, E] int32 routed rows per sequence and expert,
 *   or NULL (moe_router_bwd_sigmoid needs them for the loss gradient).
 * Errors: route shapes, seq_len >= 1 dividing S (MOE_ERR_SHAPE),
 * MOE_ERR_WORKSPACE. */
int moe_seq_aux_loss(const float* logits, const int32_t* topk_idx, int64_t S, int32_t E, int32_t K,
                     int64_t seq_len, float coeff, float* loss, int32_t* seq_counts, void* ws,
                     size_t ws_bytes, hipStream_t stream);

/* Workspace bytes moe_router_bwd_sigmoid needs; 0 for invalid sizes. */
size_t moe_router_bwd_sigmoid_workspace_bytes(int64_t S, int32_t D, int32_t E);

/* Backward of the sigmoid router with the selection held fixed, for the
 * loss  <dg, g> + balance loss:
 *   dlogits = s (1 - s) * ( on the picked experts (dg_k - sum_j g_j dg_j) / Z,
 *                           Z = sum_j s[T_j];
 *                           plus, with seq_counts, the balance-loss gradient
 *                           (a_e - sum_e' a_e' s_e'/sum s) / sum s,
 *                           a_e = coeff E n_be / (K seq_len^2 B) )
 *   dWr, dbias, dx_r as for moe_router_bwd.  Without the balance loss dx_r
 *   is the K nonzero terms in fp32; with it, dlogits is dense and dx_r is
 *   one MFMA product of three-term bf16 splits of dlogits and Wr (error
 *   within a few 2^-24 of |dlogits| |Wr|^T).
 *   logits [S, E] fp32 (the router's output);  topk_idx, topk_gate, dg [S, K];
 *   seq_counts [S / seq_len, E] from moe_seq_aux_loss, or NULL (no loss);
 *   dlogits [S, E] fp32 or NULL (kept in the workspace);  dWr [D, E];
 *   dbias [E] or NULL;  dx_r [S, D] fp32 (16-byte aligned) or NULL.
 * Errors: as moe_router_bwd; seq_len must divide S when seq_counts is given. */
int moe_router_bwd_sigmoid(const moe_bf16* x_r, const float* Wr, const float* logits,
                           const int32_t* topk_idx, const float* topk_gate, const float* dg,
                           const int32_t* seq_counts, int64_t seq_len, float coeff, int64_t S,
                           int32_t D, int32_t E, int32_t K, float* dlogits, float* dWr, float* dbias,
                           float* dx_r, void* ws, size_t ws_bytes, hipStream_t stream);

/* Load-driven update of the selection-only bias (it is not trained by
 * gradient): sel_bias[e] += rate * sign(mean(counts) - counts[e]), the sign
 * taken exactly in integers.  counts [E] (moe_route_sigmoid's), sel_bias [E]
 * fp32 updated in place. */
int moe_expert_bias_update(const int32_t* counts, int32_t E, float rate, float* sel_bias,
                           hipStream_t stream);

/* y[t] = bf16( sum_{k<K} p_disp[pos] y_disp[pos] + y_add[t] ): moe_combine
 * with an fp32 addend (the shared expert's output) added after the K-term
 * sum and before the one rounding.  y_add [S, D] fp32, 16-byte aligned. */
int moe_combine_add(const moe_bf16* y_disp, const float* p_disp, const int32_t* inv_perm,
                    const float* y_add, int64_t S, int32_t D, int32_t K, moe_bf16* y,
                    hipStream_t stream);

/* Shared expert forward on every token (ungated, squared-ReLU):
 *   u_s = x @ Ws1 (bf16, saved if u_s != NULL);  h_s = bf16(max(u_s, 0)^2);
 *   y_s = h_s @ Ws2  (fp32, for moe_combine_add).
 *   x [S, D] bf16;  Ws1 [D, Fs];  Ws2 [Fs, D];  h_s [S, Fs];  y_s [S, D] fp32.
 * Errors: D, Fs multiples of 8 in [8, 65536]; MOE_ERR_UNSUPPORTED if D*Fs*2
 * reaches 2^31. */
int moe_shared_expert_fwd(const moe_bf16* x, const moe_bf16* Ws1, const moe_bf16* Ws2, int64_t S,
                          int32_t D, int32_t Fs, moe_bf16* h_s, moe_bf16* u_s, float* y_s,
                          hipStream_t stream);

/* Workspace bytes moe_shared_expert_bwd needs; 0 for invalid sizes. */
size_t moe_shared_expert_bwd_workspace_bytes(int64_t S, int32_t D, int32_t Fs);

/* Shared expert backward for the layer-output gradient dy:
 *   du   = bf16( (dy @ Ws2^T) * 2 max(u_s, 0) )      (workspace)
 *   dx   = du @ Ws1^T  fp32 [S, D]; with accumulate_dx, added to what dx
 *          holds (e.g. moe_router_bwd*'s dx_r, then pass it as dx_add to
 *          moe_dispatch_bwd_add); dx may be NULL
 *   dWs1 = x^T du  [D, Fs] fp32;   dWs2 = h_s^T dy  [Fs, D] fp32
 *   (fixed-order sums over row chunks).
 * Errors: as moe_shared_expert_fwd; MOE_ERR_UNSUPPORTED if S*max(D, Fs)*2
 * reaches 2^31; MOE_ERR_WORKSPACE. */
int moe_shared_expert_bwd(const moe_bf16* x, const moe_bf16* u_s, const moe_bf16* h_s,
                          const moe_bf16* dy, const moe_bf16* Ws1, const moe_bf16* Ws2, int64_t S,
                          int32_t D, int32_t Fs, float* dx, int32_t accumulate_dx, float* dWs1,
                          float* dWs2, void* ws, size_t ws_bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* MOE_H */
