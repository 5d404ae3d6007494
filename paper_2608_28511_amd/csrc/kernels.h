// Launchers of the gfx950 kernels (internal to the library; the public
// surface is include/moe.h).  Each returns the HIP error of its launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "moe.h"

namespace moe {

enum { EPI_BF16 = 0, EPI_RELU2 = 1, EPI_DRELU2 = 2, EPI_F32 = 3 };

// Compute units of the current device (read once per device).
int cu_count();

// Router workspace: the three bf16 planes [3][E][D] of the split router weight.
size_t router_ws_bytes(int D, int E);
hipError_t launch_router_logits(const moe_bf16* x, const float* Wr, const float* bias, int64_t S,
                                int D, int E, float* logits, void* ws, hipStream_t st);

// Router backward (selection held fixed): dlogits (optional; else internal),
// dWr [D,E], dbias [E] (optional), dx_r [S,D] fp32 (optional).
// dense: the sigmoid router with the balance loss (ds dense over E).
size_t router_bwd_ws_bytes(int64_t S, int D, int E, bool dense = false);
hipError_t launch_router_bwd(const moe_bf16* x_r, const float* Wr, const int32_t* topk_idx, const float* topk_prob,
                             const float* dp, int64_t S, int D, int E, int K, float* dlogits, float* dWr,
                             float* dbias, float* dx_r, void* ws, hipStream_t st);
// Sigmoid router backward: dg is the gradient of the routed weights; with
// seq_counts (per sequence of seq_len tokens and expert) the balance-loss
// gradient coef * count is added (coef = coeff * E / (K * T^2 * B)).
hipError_t launch_router_bwd_sigmoid(const moe_bf16* x_r, const float* Wr, const float* logits,
                                     const int32_t* topk_idx, const float* topk_gate, const float* dg,
                                     const int32_t* seq_counts, int64_t seq_len, float coef, int64_t S, int D,
                                     int E, int K, float* dlogits, float* dWr, float* dbias, float* dx_r,
                                     void* ws, hipStream_t st);
// Sequence balance loss forward: loss[0] (fp32) and seq_counts [B, E] (may be null).
size_t seq_aux_ws_bytes(int64_t S, int E, int64_t seq_len);
hipError_t launch_seq_aux_loss(const float* logits, const int32_t* topk_idx, int64_t S, int E, int K,
                               int64_t seq_len, double coef, float* loss, int32_t* seq_counts, void* ws,
                               hipStream_t st);
// sel_bias[e] += rate * sign(mean(counts) - counts[e])
hipError_t launch_expert_bias_update(const int32_t* counts, int E, float rate, float* sel_bias, hipStream_t st);
// out[m,n] = sum_c sum_{s=P-1..0} part[c][m][s*ldp+n] (fixed order; rows of part hold P*ldp)
hipError_t launch_sum_planes(const float* part, int nchunk, int M, int N, int P, int ldp, float* out,
                             hipStream_t st);
int wgrad_chunks(int64_t rows, int M, int N);

size_t route_ws_bytes(int64_t S, int E);
// sigmoid: the production router (sigmoid scores, selection by score +
// sel_bias (nullable), weights = picked sigmoids over their sum); otherwise
// the softmax router.  With p_disp, each routed row's probability is also
// written at its position (p_disp[inv_perm[t*K+k]] = topk_prob[t, k]); with
// sched, the launch also builds the grouped GEMM's tile tables.
hipError_t launch_route(const float* logits, int64_t S, int E, int K, int32_t* topk_idx,
                        float* topk_prob, int32_t* counts, int32_t* offsets, int32_t* perm,
                        int32_t* inv_perm, void* ws, hipStream_t st, bool sigmoid = false,
                        const float* sel_bias = nullptr, float* p_disp = nullptr, void* sched = nullptr);

// With sched (and the expert offsets sched_offsets [E+1] of the same
// routing), the launch also builds the grouped GEMM's tile tables in sched,
// as launch_tile_schedule would.
hipError_t launch_dispatch(const moe_bf16* x, const float* prob, const int32_t* inv_perm, int64_t S,
                           int D, int K, moe_bf16* x_disp, float* p_disp, hipStream_t st,
                           const int32_t* sched_offsets = nullptr, int E = 0, void* sched = nullptr);
// MX-FP8 payload (D a multiple of 32): codes [S*K, D] and E8M0 scales
// [S*K, D/32] of each token row at its K routed rows (with sched: the tile
// tables as in launch_dispatch); decode to bf16.
hipError_t launch_dispatch_mx(const moe_bf16* x, const float* prob, const int32_t* inv_perm, int64_t S, int D,
                              int K, uint8_t* x_q, uint8_t* x_scale, float* p_disp, hipStream_t st,
                              const int32_t* sched_offsets = nullptr, int E = 0, void* sched = nullptr);
hipError_t launch_dequant_mx(const uint8_t* x_q, const uint8_t* x_scale, int64_t R, int D, moe_bf16* out,
                             hipStream_t st);
// y[t] = bf16(sum_k w_k y_disp[pos_k] (+ add[t], fp32 [S,D], after the sum; NULL for none))
hipError_t launch_combine(const moe_bf16* y_disp, const float* p_disp, const int32_t* inv_perm,
                          int64_t S, int D, int K, const float* add, moe_bf16* y, hipStream_t st);
hipError_t launch_combine_bwd(const moe_bf16* dy, const moe_bf16* y_disp, const float* p_disp,
                              const int32_t* inv_perm, int64_t S, int D, int K, moe_bf16* dy_disp,
                              float* dp, hipStream_t st);

int gemm_tile_m();

// Bytes of the fixed device scratch of the entry point that allocates
// nothing (its tile schedule), and that array's address on the current device.
constexpr size_t kStaticScratchBytes = 448 * 1024;
hipError_t static_scratch(void** ptr);
// Schedule buffer of the grouped GEMM: mtile_start [E+1] then the per-tile table.
size_t gemm_schedule_bytes(int E, int64_t R);
hipError_t launch_tile_schedule(const int32_t* offsets, int E, int64_t R, void* sched, hipStream_t st);
// ROWS mode: C[r, :] = A[r, :] @ B_e per expert segment (sched from launch_tile_schedule
// for the same offsets, E and R), or dense over R rows when sched == nullptr.
// b_kmajor: B_e stored [N, Kd] (product with its transpose) instead of [Kd, N].
// EPI_F32 writes fp32 C (ldc in floats); with accumulate, C += product.
hipError_t launch_grouped_rows(const moe_bf16* A, int64_t lda, const moe_bf16* B, int64_t ldb,
                               int64_t b_stride, bool b_kmajor, void* C, int64_t ldc, int epi,
                               const moe_bf16* aux_in, moe_bf16* aux_out, const void* sched,
                               int E, int64_t R, int N, int Kd, hipStream_t st, bool accumulate = false);
// ROWS mode with the dispatch fused into the A copy: row r of expert
// segment e is X[perm[r] / div, :] (X [x_rows, Kd] bf16, ldx elements per
// row; perm as moe_route_topk writes it, div = K), B N-contiguous.  Equal to
// launch_grouped_rows on the dispatched rows, without materialising them.
hipError_t launch_grouped_rows_gather(const moe_bf16* X, int64_t ldx, int64_t x_rows, const int32_t* perm, int div,
                                      const moe_bf16* B, int64_t ldb, int64_t b_stride, void* C, int64_t ldc, int epi,
                                      moe_bf16* aux_out, const void* sched, int E, int64_t R, int N, int Kd,
                                      hipStream_t st);
// ROWS mode over an MX-FP8 A: codes Aq [R, Kd] uint8 (16-byte aligned, Kd a
// multiple of 32) and E8M0 scales A_scale [R, Kd / 32] (allocation rounded up
// to 4 bytes), decoded in the operand path; B N-contiguous; epi EPI_BF16 or
// EPI_RELU2.  Bit-identical to launch_grouped_rows on the decoded bf16 A.
hipError_t launch_grouped_rows_mx(const uint8_t* Aq, const uint8_t* A_scale, const moe_bf16* B, int64_t ldb,
                                  int64_t b_stride, void* C, int64_t ldc, int epi, moe_bf16* aux_out,
                                  const void* sched, int E, int64_t R, int N, int Kd, hipStream_t st);
// KGRP mode: C_e[m, n] = sum over expert e's rows r of A[r, m] * B[r, n]  (fp32 out).
// KGRP over a dense contraction cut into nchunk row ranges of kchunk rows:
// C + c*c_stride = A[rows of chunk c]^T @ B[rows of chunk c]  (fp32 partials).
hipError_t launch_chunked_wgrad(const moe_bf16* A, int64_t lda, const moe_bf16* B, int64_t ldb, float* C,
                                int64_t ldc, int64_t c_stride, int nchunk, int64_t kchunk, int M, int N,
                                int64_t R, hipStream_t st);
// Two KGRP products over the same expert segments in one launch (the expert
// FFN's dW2 and dW1): the experts' items in `order` (required, from
// launch_expert_order), the largest contractions first, dealt evenly to the
// XCDs in chunks of consecutive items.
hipError_t launch_grouped_wgrad2(const moe_bf16* A0, int64_t lda0, const moe_bf16* B0, int64_t ldb0, float* C0,
                                 int64_t ldc0, int64_t c_stride0, int M0, int N0, const moe_bf16* A1, int64_t lda1,
                                 const moe_bf16* B1, int64_t ldb1, float* C1, int64_t ldc1, int64_t c_stride1, int M1,
                                 int N1, const int32_t* offsets, const int32_t* order, int E, int64_t R,
                                 hipStream_t st);
// order[rank] = expert with the rank-th most rows of offsets[0..E] (ties to the lower index).
hipError_t launch_expert_order(const int32_t* offsets, int E, int64_t R, int32_t* order, hipStream_t st);

}  // namespace moe
