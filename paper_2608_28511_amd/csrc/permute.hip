// Dispatch and combine on gfx950: the local form of the expert-parallel
// hidden dispatch, probability dispatch and hidden combine (Section 4.1
// footnote), whose per-row payloads Eq. 1 counts.
//
// All four kernels are HBM-bound row copies.  One wavefront owns one token:
// it reads the token's row once with 16-byte loads (8 bf16 per lane) and
// writes it to (dispatch) or gathers it from (combine) the token's K rows of
// the expert-contiguous buffer, each a contiguous D*2-byte row.  The combine
// sums in fp32 in ascending slot order inside the wave, so it needs no
// atomics and is deterministic.
#include "common.h"
#include "kernels.h"

namespace moe {

constexpr int kRowThreads = 256;               // 4 tokens per block
constexpr int kRowTok = kRowThreads / kWave;
constexpr int kCPL = 4;                        // 16-byte chunks per lane per pass

__global__ __launch_bounds__(kRowThreads) void dispatch_kernel(const uint4* __restrict__ x,
                                                               const float* __restrict__ prob,
                                                               const int32_t* __restrict__ inv_perm,
                                                               int64_t S, int D8, int K,
                                                               uint4* __restrict__ x_disp,
                                                               float* __restrict__ p_disp) {
    const int lane = threadIdx.x & 63;
    const int64_t t = (int64_t)blockIdx.x * kRowTok + (threadIdx.x >> 6);
    if (t >= S) return;
    const int64_t R = S * K;
    int pos_l = lane < K ? inv_perm[t * K + lane] : 0;
    if ((uint32_t)pos_l >= (uint64_t)R) pos_l = -1;  // out-of-range entries are not written
    if (p_disp != nullptr && lane < K && pos_l >= 0) p_disp[pos_l] = prob[t * K + lane];
    const uint4* src = x + t * D8;
    for (int c0 = 0; c0 < D8; c0 += kWave * kCPL) {
        uint4 v[kCPL];
#pragma unroll
        for (int i = 0; i < kCPL; ++i) {
            const int c = c0 + lane + kWave * i;
            if (c < D8) v[i] = src[c];
        }
        for (int k = 0; k < K; ++k) {
            const int64_t pos = __shfl(pos_l, k);
            if (pos < 0) continue;
            uint4* dst = x_disp + pos * D8;
#pragma unroll
            for (int i = 0; i < kCPL; ++i) {
                const int c = c0 + lane + kWave * i;
                if (c < D8) dst[c] = v[i];
            }
        }
    }
}

__device__ __forceinline__ void fma8(float* acc, float w, const uint4& v) {
    acc[0] = fmaf(w, bf16_lo(v.x), acc[0]);
    acc[1] = fmaf(w, bf16_hi(v.x), acc[1]);
    acc[2] = fmaf(w, bf16_lo(v.y), acc[2]);
    acc[3] = fmaf(w, bf16_hi(v.y), acc[3]);
    acc[4] = fmaf(w, bf16_lo(v.z), acc[4]);
    acc[5] = fmaf(w, bf16_hi(v.z), acc[5]);
    acc[6] = fmaf(w, bf16_lo(v.w), acc[6]);
    acc[7] = fmaf(w, bf16_hi(v.w), acc[7]);
}

__device__ __forceinline__ uint4 pack8(const float* a) {
    uint4 o;
    o.x = pack_bf16x2(a[0], a[1]);
    o.y = pack_bf16x2(a[2], a[3]);
    o.z = pack_bf16x2(a[4], a[5]);
    o.w = pack_bf16x2(a[6], a[7]);
    return o;
}

// y[t] = bf16(sum_k w_k * y_disp[pos_k]); w_k = p_disp[pos_k] or 1.
__global__ __launch_bounds__(kRowThreads) void combine_kernel(const uint4* __restrict__ y_disp,
                                                              const float* __restrict__ p_disp,
                                                              const int32_t* __restrict__ inv_perm,
                                                              int64_t S, int D8, int K,
                                                              const float4* __restrict__ add,
                                                              uint4* __restrict__ y) {
    const int lane = threadIdx.x & 63;
    const int64_t t = (int64_t)blockIdx.x * kRowTok + (threadIdx.x >> 6);
    if (t >= S) return;
    const int64_t R = S * K;
    int pos_l = lane < K ? inv_perm[t * K + lane] : 0;
    if ((uint32_t)pos_l >= (uint64_t)R) pos_l = -1;  // out-of-range entries contribute nothing
    const float w_l = (lane < K && pos_l >= 0) ? (p_disp != nullptr ? p_disp[pos_l] : 1.f) : 0.f;
    for (int c0 = 0; c0 < D8; c0 += kWave * kCPL) {
        float acc[kCPL][8];
#pragma unroll
        for (int i = 0; i < kCPL; ++i)
#pragma unroll
            for (int q = 0; q < 8; ++q) acc[i][q] = 0.f;
        for (int k = 0; k < K; ++k) {
            const int64_t pos = __shfl(pos_l, k);
            const float w = __shfl(w_l, k);
            if (pos < 0) continue;
            const uint4* src = y_disp + pos * D8;
            uint4 v[kCPL];
#pragma unroll
            for (int i = 0; i < kCPL; ++i) {
                const int c = c0 + lane + kWave * i;
                if (c < D8) v[i] = src[c];
            }
#pragma unroll
            for (int i = 0; i < kCPL; ++i)
                if (c0 + lane + kWave * i < D8) fma8(acc[i], w, v[i]);
        }
#pragma unroll
        for (int i = 0; i < kCPL; ++i) {
            const int c = c0 + lane + kWave * i;
            if (c >= D8) continue;
            if (add != nullptr) {  // fp32 addend, summed after the K rows, before the rounding
                const float4 a0 = add[(t * D8 + c) * 2], a1 = add[(t * D8 + c) * 2 + 1];
                acc[i][0] += a0.x; acc[i][1] += a0.y; acc[i][2] += a0.z; acc[i][3] += a0.w;
                acc[i][4] += a1.x; acc[i][5] += a1.y; acc[i][6] += a1.z; acc[i][7] += a1.w;
            }
            y[t * D8 + c] = pack8(acc[i]);
        }
    }
}

// dy_disp[pos_k] = bf16(w_k * dy[t]);  dp[t,k] = <dy[t], y_disp[pos_k]>.
__global__ __launch_bounds__(kRowThreads) void combine_bwd_kernel(
    const uint4* __restrict__ dy, const uint4* __restrict__ y_disp, const float* __restrict__ p_disp,
    const int32_t* __restrict__ inv_perm, int64_t S, int D8, int K, uint4* __restrict__ dy_disp,
    float* __restrict__ dp) {
    const int lane = threadIdx.x & 63;
    const int64_t t = (int64_t)blockIdx.x * kRowTok + (threadIdx.x >> 6);
    if (t >= S) return;
    const int64_t R = S * K;
    int pos_l = lane < K ? inv_perm[t * K + lane] : 0;
    if ((uint32_t)pos_l >= (uint64_t)R) pos_l = -1;  // out-of-range entries are skipped
    const float w_l = (lane < K && pos_l >= 0) ? (p_disp != nullptr ? p_disp[pos_l] : 1.f) : 0.f;
    const uint4* g = dy + t * D8;
    for (int k = 0; k < K; ++k) {
        const int64_t pos = __shfl(pos_l, k);
        const float w = __shfl(w_l, k);
        if (pos < 0) continue;
        const uint4* yd = y_disp + pos * D8;
        uint4* out = dy_disp + pos * D8;
        float dot = 0.f;
        for (int c0 = 0; c0 < D8; c0 += kWave * kCPL) {
            uint4 gv[kCPL], yv[kCPL];
#pragma unroll
            for (int i = 0; i < kCPL; ++i) {
                const int c = c0 + lane + kWave * i;
                if (c < D8) {
                    gv[i] = g[c];
                    yv[i] = yd[c];
                }
            }
#pragma unroll
            for (int i = 0; i < kCPL; ++i) {
                const int c = c0 + lane + kWave * i;
                if (c < D8) {
                    float a[8], b[8];
                    a[0] = bf16_lo(gv[i].x); a[1] = bf16_hi(gv[i].x);
                    a[2] = bf16_lo(gv[i].y); a[3] = bf16_hi(gv[i].y);
                    a[4] = bf16_lo(gv[i].z); a[5] = bf16_hi(gv[i].z);
                    a[6] = bf16_lo(gv[i].w); a[7] = bf16_hi(gv[i].w);
                    b[0] = bf16_lo(yv[i].x); b[1] = bf16_hi(yv[i].x);
                    b[2] = bf16_lo(yv[i].y); b[3] = bf16_hi(yv[i].y);
                    b[4] = bf16_lo(yv[i].z); b[5] = bf16_hi(yv[i].z);
                    b[6] = bf16_lo(yv[i].w); b[7] = bf16_hi(yv[i].w);
#pragma unroll
                    for (int q = 0; q < 8; ++q) {
                        dot = fmaf(a[q], b[q], dot);
                        a[q] *= w;
                    }
                    out[c] = pack8(a);
                }
            }
        }
#pragma unroll
        for (int m = 32; m > 0; m >>= 1) dot += __shfl_xor(dot, m);
        if (dp != nullptr && lane == 0) dp[t * K + k] = dot;
    }
}

hipError_t launch_dispatch(const moe_bf16* x, const float* prob, const int32_t* inv_perm, int64_t S,
                           int D, int K, moe_bf16* x_disp, float* p_disp, hipStream_t st) {
    if (S == 0) return hipSuccess;
    hipLaunchKernelGGL(dispatch_kernel, dim3(grid_for(S, kRowTok)), dim3(kRowThreads), 0, st,
                       (const uint4*)x, prob, inv_perm, S, D / 8, K, (uint4*)x_disp, p_disp);
    return hipGetLastError();
}

hipError_t launch_combine(const moe_bf16* y_disp, const float* p_disp, const int32_t* inv_perm,
                          int64_t S, int D, int K, const float* add, moe_bf16* y, hipStream_t st) {
    if (S == 0) return hipSuccess;
    hipLaunchKernelGGL(combine_kernel, dim3(grid_for(S, kRowTok)), dim3(kRowThreads), 0, st,
                       (const uint4*)y_disp, p_disp, inv_perm, S, D / 8, K, (const float4*)add, (uint4*)y);
    return hipGetLastError();
}

hipError_t launch_combine_bwd(const moe_bf16* dy, const moe_bf16* y_disp, const float* p_disp,
                              const int32_t* inv_perm, int64_t S, int D, int K, moe_bf16* dy_disp,
                              float* dp, hipStream_t st) {
    if (S == 0) return hipSuccess;
    hipLaunchKernelGGL(combine_bwd_kernel, dim3(grid_for(S, kRowTok)), dim3(kRowThreads), 0, st,
                       (const uint4*)dy, (const uint4*)y_disp, p_disp, inv_perm, S, D / 8, K,
                       (uint4*)dy_disp, dp);
    return hipGetLastError();
}

}  // namespace moe
