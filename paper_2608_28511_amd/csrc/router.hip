// Router logits on gfx950: logits[t, e] = sum_d x[t, d] * Wr[d, e] + bias[e]
// in fp32 (the router scores every token against every expert, Section 5.2).
//
// A plain fp32 SIMT tile: 32 tokens x 64 experts per 256-thread block, each
// thread 2 tokens x 4 experts, the reduction dimension staged through LDS in
// 32-wide slabs (x converted from bf16 on the way in).  Every output is one
// fp32 FMA chain in ascending d, so results are deterministic.
#include "common.h"
#include "kernels.h"

namespace moe {

constexpr int kRT = 32;   // tokens per block
constexpr int kRE = 64;   // experts per block
constexpr int kRD = 32;   // reduction slab

__global__ __launch_bounds__(256) void router_logits_kernel(const uint16_t* __restrict__ x,
                                                            const float* __restrict__ Wr,
                                                            const float* __restrict__ bias,
                                                            int64_t S, int D, int E,
                                                            float* __restrict__ logits) {
    __shared__ float xs[kRD][kRT + 4];
    __shared__ float ws[kRD][kRE + 4];
    const int tid = threadIdx.x;
    const int tx = tid & 15;          // expert quad
    const int ty = tid >> 4;          // token pair
    const int64_t t0 = (int64_t)blockIdx.x * kRT;
    const int e0 = blockIdx.y * kRE;
    float acc[2][4] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
    for (int d0 = 0; d0 < D; d0 += kRD) {
        if (tid < kRT * kRD / 8) {    // 128 threads: one 8-wide bf16 chunk each
            const int tt = tid >> 2, dc = (tid & 3) * 8;
            const int64_t t = t0 + tt;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (t < S && d0 + dc < D) v = *(const uint4*)(x + t * D + d0 + dc);
            xs[dc + 0][tt] = bf16_lo(v.x); xs[dc + 1][tt] = bf16_hi(v.x);
            xs[dc + 2][tt] = bf16_lo(v.y); xs[dc + 3][tt] = bf16_hi(v.y);
            xs[dc + 4][tt] = bf16_lo(v.z); xs[dc + 5][tt] = bf16_hi(v.z);
            xs[dc + 6][tt] = bf16_lo(v.w); xs[dc + 7][tt] = bf16_hi(v.w);
        }
#pragma unroll
        for (int q = 0; q < kRD * kRE / 256; ++q) {
            const int idx = tid + 256 * q;
            const int dd = idx / kRE, ee = idx % kRE;
            const int d = d0 + dd, e = e0 + ee;
            ws[dd][ee] = (d < D && e < E) ? Wr[(int64_t)d * E + e] : 0.f;
        }
        __syncthreads();
#pragma unroll 8
        for (int dd = 0; dd < kRD; ++dd) {
            const float a0 = xs[dd][ty * 2], a1 = xs[dd][ty * 2 + 1];
            const float4 b = *(const float4*)&ws[dd][tx * 4];
            acc[0][0] = fmaf(a0, b.x, acc[0][0]); acc[0][1] = fmaf(a0, b.y, acc[0][1]);
            acc[0][2] = fmaf(a0, b.z, acc[0][2]); acc[0][3] = fmaf(a0, b.w, acc[0][3]);
            acc[1][0] = fmaf(a1, b.x, acc[1][0]); acc[1][1] = fmaf(a1, b.y, acc[1][1]);
            acc[1][2] = fmaf(a1, b.z, acc[1][2]); acc[1][3] = fmaf(a1, b.w, acc[1][3]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int64_t t = t0 + ty * 2 + i;
        if (t >= S) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int e = e0 + tx * 4 + j;
            if (e < E) logits[t * E + e] = acc[i][j] + (bias != nullptr ? bias[e] : 0.f);
        }
    }
}

hipError_t launch_router_logits(const moe_bf16* x, const float* Wr, const float* bias, int64_t S,
                                int D, int E, float* logits, hipStream_t st) {
    if (S == 0) return hipSuccess;
    dim3 grid(grid_for(S, kRT), (unsigned)((E + kRE - 1) / kRE));
    hipLaunchKernelGGL(router_logits_kernel, grid, dim3(256), 0, st, (const uint16_t*)x, Wr, bias, S,
                       D, E, logits);
    return hipGetLastError();
}

}  // namespace moe
