// Router logits on gfx950: logits[t, e] = sum_d x[t, d] * Wr[d, e] + bias[e]
// (the router scores every token against every expert, Section 5.2).
//
// The router weight is fp32 while x is bf16.  Each fp32 weight w is split
// into three bf16 terms, hi = bf16(w), mid = bf16(w - hi), lo = bf16(w - hi -
// mid), whose sum equals w to within 2^-27 |w|.  Products of bf16 values are
// exact in fp32, so three bf16 MFMAs (x*lo + x*mid + x*hi, accumulated in
// fp32) reproduce the fp32 product to fp32 accuracy while running on the
// matrix cores (bf16 splitting as in Henry, Tang and Heinecke, "Leveraging
// the bfloat16 artificial intelligence datatype for higher-precision
// computations", ARITH 2019).
//
// Tiles: 64 tokens x 64 experts x 64 d per 256-thread block, 4 wavefronts of
// 32 x 32 outputs; the split happens while the fp32 weight tile is written
// to LDS (transposed to expert rows of d-contiguous chunks, the MFMA operand
// layout), double buffered.  Every output is one fixed-order fp32 MFMA chain,
// so results are deterministic.
#include "common.h"
#include "kernels.h"

namespace moe {

constexpr int kRT = 64;       // tokens per block
constexpr int kRE = 64;       // experts per block
constexpr int kRK = 64;       // d per stage
constexpr int kRChunks = kRK / 8;
constexpr int kRTile = kRT * kRK * 2;   // bytes of one bf16 64x64 tile

// chunk c of row r stored at c ^ (r & 7): conflict-free 16-row ds_read_b128 on gfx950
__device__ __forceinline__ int rswz(int row) { return row & (kRChunks - 1); }
__device__ __forceinline__ int roff(int r, int c) { return (r * kRChunks + (c ^ rswz(r))) * 16; }

__device__ __forceinline__ float bf16_round_f32(float f, uint32_t* bits) {
    const uint32_t b = f32_to_bf16(f);
    *bits = b;
    return __uint_as_float(b << 16);
}

__global__ __launch_bounds__(256, 2) void router_logits_kernel(const uint16_t* __restrict__ x,
                                                               const float* __restrict__ Wr,
                                                               const float* __restrict__ bias,
                                                               int64_t S, int D, int E,
                                                               float* __restrict__ logits,
                                                               bool vec_w, bool vec_out) {
    // per stage: A [64 tok][64 d], B_hi, B_mid, B_lo [64 exp][64 d]
    __shared__ __attribute__((aligned(16))) char smem[2 * 4 * kRTile];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t t0 = (int64_t)blockIdx.x * kRT;
    const int e0 = blockIdx.y * kRE;

    uint4 av[2];
    float bw[4][4];  // [k row][expert] of this thread's 4x4 weight block
    const int eg = tid & 15, kg = tid >> 4;

    auto load = [&](int d0) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int q = tid + 256 * i;
            const int r = q >> 3, c = q & 7;
            const int64_t t = t0 + r;
            const int d = d0 + c * 8;
            av[i] = (t < S && d < D) ? *(const uint4*)(x + t * D + d) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int d = d0 + kg * 4 + q;
            const int e = e0 + eg * 4;
            if (d < D && vec_w && e + 3 < E) {
                const float4 v = *(const float4*)(Wr + (int64_t)d * E + e);
                bw[q][0] = v.x; bw[q][1] = v.y; bw[q][2] = v.z; bw[q][3] = v.w;
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    bw[q][j] = (d < D && e + j < E) ? Wr[(int64_t)d * E + e + j] : 0.f;
            }
        }
    };
    auto store = [&](char* st) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int q = tid + 256 * i;
            *(uint4*)(st + roff(q >> 3, q & 7)) = av[i];
        }
        char* bh = st + kRTile;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            uint32_t hb[4], mb[4], lb[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float w = bw[q][j];
                const float h = bf16_round_f32(w, &hb[q]);
                const float r1 = w - h;
                const float m = bf16_round_f32(r1, &mb[q]);
                lb[q] = f32_to_bf16(r1 - m);
            }
            const int r = eg * 4 + j;
            const int off = roff(r, kg >> 1) + (kg & 1) * 8;
            *(uint2*)(bh + off) = make_uint2(hb[0] | (hb[1] << 16), hb[2] | (hb[3] << 16));
            *(uint2*)(bh + kRTile + off) = make_uint2(mb[0] | (mb[1] << 16), mb[2] | (mb[3] << 16));
            *(uint2*)(bh + 2 * kRTile + off) = make_uint2(lb[0] | (lb[1] << 16), lb[2] | (lb[3] << 16));
        }
    };

    f32x4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int nk = (D + kRK - 1) / kRK;
    load(0);
    store(smem);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int cur = kt & 1;
        if (kt + 1 < nk) load((kt + 1) * kRK);
        const char* st = smem + cur * 4 * kRTile;
#pragma unroll
        for (int kk = 0; kk < kRK / 32; ++kk) {
            const int c = kk * 4 + (lane >> 4);
            bf16x8 af[2], bf[3][2];
#pragma unroll
            for (int i = 0; i < 2; ++i)
                af[i] = *(const bf16x8*)(st + roff(wm * 32 + i * 16 + (lane & 15), c));
#pragma unroll
            for (int s = 0; s < 3; ++s)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    bf[s][j] = *(const bf16x8*)(st + (1 + s) * kRTile +
                                                roff(wn * 32 + j * 16 + (lane & 15), c));
#pragma unroll
            for (int s = 2; s >= 0; --s)   // lo, mid, hi: smaller terms first
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bf[s][j], af[i], acc[i][j], 0, 0, 0);
        }
        if (kt + 1 < nk) store(smem + (cur ^ 1) * 4 * kRTile);
        __syncthreads();
    }

    // lane holds logits[t][e .. e+3]
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int64_t t = t0 + wm * 32 + i * 16 + (lane & 15);
        if (t >= S) continue;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int e = e0 + wn * 32 + j * 16 + 4 * (lane >> 4);
            float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
            if (bias != nullptr) {
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    if (e + q < E) v[q] += bias[e + q];
            }
            float* dst = logits + t * E + e;
            if (vec_out && e + 3 < E) {
                *(float4*)dst = make_float4(v[0], v[1], v[2], v[3]);
            } else {
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    if (e + q < E) dst[q] = v[q];
            }
        }
    }
}

hipError_t launch_router_logits(const moe_bf16* x, const float* Wr, const float* bias, int64_t S,
                                int D, int E, float* logits, hipStream_t st) {
    if (S == 0) return hipSuccess;
    dim3 grid(grid_for(S, kRT), (unsigned)((E + kRE - 1) / kRE));
    // 16-byte vector access only where every row start is 16-byte aligned
    const bool vec_w = (E % 4) == 0 && ((uintptr_t)Wr % 16) == 0;
    const bool vec_out = (E % 4) == 0 && ((uintptr_t)logits % 16) == 0;
    hipLaunchKernelGGL(router_logits_kernel, grid, dim3(256), 0, st, (const uint16_t*)x, Wr, bias, S,
                       D, E, logits, vec_w, vec_out);
    return hipGetLastError();
}

}  // namespace moe
