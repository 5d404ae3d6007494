// Router backward on gfx950 (the learned router of Section 5.2), with the
// expert selection held fixed: top-K is piecewise constant in the scores.
//
// The routed probability p_k is the softmax of the K selected scores, so per
// token, from the probability gradient dp (the combine's transpose),
//     ds[T_k] = p_k (dp_k - sum_j p_j dp_j),      ds = 0 elsewhere,
// and through logits = x_r Wr + bias:
//     dWr = x_r^T ds,   dbias = sum_t ds[t],   dx_r = ds Wr^T.
//
// Launches:
//   router_ds_kernel      one wavefront per token: ds (dense fp32 rows) and
//                         ds split into three bf16 planes hi / mid / lo
//                         (sum within 2^-24 relative of ds, as for the forward
//                         weight split) for the MFMA product below;
//   dWr                   the grouped GEMM's k-grouped mode, x_r^T [hi|mid|lo]
//                         over row chunks of S into fp32 partials, then
//                         sum_planes_kernel adds planes (lo, mid, hi) and
//                         chunks in a fixed order;
//   router_dbias_kernel   one wavefront per expert, fixed-order column sum;
//   router_dx_kernel      one wavefront per token: the K nonzero terms of
//                         ds Wr^T in fp32 from a transposed copy of Wr.
// Every reduction has a fixed order, so results are deterministic.
#include "common.h"
#include "kernels.h"

namespace moe {

constexpr int kRbTok = 4;  // tokens (wavefronts) per 256-thread block

template <int EPL>
__global__ __launch_bounds__(256) void router_ds_kernel(const int32_t* __restrict__ topk_idx,
                                                        const float* __restrict__ topk_prob,
                                                        const float* __restrict__ dp, int64_t S, int E,
                                                        int Ep, int K, float* __restrict__ ds,
                                                        uint16_t* __restrict__ ds3) {
    const int lane = threadIdx.x & 63;
    const int64_t t = (int64_t)blockIdx.x * kRbTok + (threadIdx.x >> 6);
    if (t >= S) return;
    int e_l = -1;
    float p_l = 0.f, g_l = 0.f;
    if (lane < K) {
        e_l = topk_idx[t * K + lane];
        p_l = topk_prob[t * K + lane];
        g_l = dp[t * K + lane];
    }
    float m = p_l * g_l;
#pragma unroll
    for (int msk = 32; msk > 0; msk >>= 1) m += __shfl_xor(m, msk);
    const float d_l = p_l * (g_l - m);
    float v[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) v[i] = 0.f;
    for (int k = 0; k < K; ++k) {
        const int ek = __shfl(e_l, k);
        const float dk = __shfl(d_l, k);
        if (ek < 0 || ek >= E) continue;  // malformed index: no contribution
#pragma unroll
        for (int i = 0; i < EPL; ++i)
            if (lane + 64 * i == ek) v[i] = dk;
    }
    // planes of Ep >= E columns (a multiple of 8, so every plane row starts
    // 16-byte aligned for the DMA); columns E .. Ep-1 are zero
    const int64_t E3 = 3 * (int64_t)Ep;
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
        const int e = lane + 64 * i;
        if (e >= Ep) break;
        const float w = e < E ? v[i] : 0.f;
        if (e < E) ds[t * E + e] = w;
        const uint32_t hi = f32_to_bf16(w);
        const float r1 = w - __uint_as_float(hi << 16);
        const uint32_t mid = f32_to_bf16(r1);
        const uint32_t lo = f32_to_bf16(r1 - __uint_as_float(mid << 16));
        ds3[t * E3 + e] = (uint16_t)hi;
        ds3[t * E3 + Ep + e] = (uint16_t)mid;
        ds3[t * E3 + 2 * Ep + e] = (uint16_t)lo;
    }
}

// dbias[e] = sum_t ds[t, e]: one wavefront per expert, lane l adds rows
// l, l + 64, ... in order, then a fixed butterfly.
__global__ __launch_bounds__(256) void router_dbias_kernel(const float* __restrict__ ds, int64_t S, int E,
                                                           float* __restrict__ dbias) {
    const int lane = threadIdx.x & 63;
    const int e = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (e >= E) return;
    float s = 0.f;
    for (int64_t t = lane; t < S; t += 64) s += ds[t * E + e];
#pragma unroll
    for (int msk = 32; msk > 0; msk >>= 1) s += __shfl_xor(s, msk);
    if (lane == 0) dbias[e] = s;
}

// WrT[e, d] = Wr[d, e] through a 32 x 33 LDS tile.
__global__ __launch_bounds__(256) void transpose_f32_kernel(const float* __restrict__ src, int rows, int cols,
                                                            float* __restrict__ dst) {
    __shared__ float tile[32][33];
    const int c0 = blockIdx.x * 32, r0 = blockIdx.y * 32;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 32 x 8
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int r = r0 + ty + 8 * q, c = c0 + tx;
        tile[ty + 8 * q][tx] = (r < rows && c < cols) ? src[(int64_t)r * cols + c] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int c = c0 + ty + 8 * q, r = r0 + tx;
        if (c < cols && r < rows) dst[(int64_t)c * rows + r] = tile[tx][ty + 8 * q];
    }
}

// dx_r[t, :] = sum_{k ascending} ds[t, T_k] * WrT[T_k, :], fp32.
__global__ __launch_bounds__(256) void router_dx_kernel(const float* __restrict__ ds,
                                                        const int32_t* __restrict__ topk_idx,
                                                        const float4* __restrict__ WrT, int64_t S, int D4,
                                                        int E, int K, float4* __restrict__ dx) {
    const int lane = threadIdx.x & 63;
    const int64_t t = (int64_t)blockIdx.x * kRbTok + (threadIdx.x >> 6);
    if (t >= S) return;
    int e_l = lane < K ? topk_idx[t * K + lane] : -1;
    if (e_l >= E) e_l = -1;
    const float w_l = e_l >= 0 ? ds[t * E + e_l] : 0.f;
    for (int c = lane; c < D4; c += 64) {
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int k = 0; k < K; ++k) {
            const int ek = __shfl(e_l, k);
            const float w = __shfl(w_l, k);
            if (ek < 0) continue;
            const float4 r = WrT[(int64_t)ek * D4 + c];
            acc.x += w * r.x; acc.y += w * r.y; acc.z += w * r.z; acc.w += w * r.w;
        }
        dx[t * D4 + c] = acc;
    }
}

// out[m, n] = sum over chunks c (ascending) of sum over planes s = P-1 .. 0 of
// part[c][m][s*ldp + n]; rows of part hold P*ldp values.
__global__ __launch_bounds__(256) void sum_planes_kernel(const float* __restrict__ part, int nchunk, int M, int N,
                                                         int P, int ldp, float* __restrict__ out) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)M * N) return;
    const int64_t m = i / N, n = i - m * N;
    const int64_t row = (int64_t)P * ldp, chunk = (int64_t)M * row;
    float s = 0.f;
    for (int c = 0; c < nchunk; ++c) {
        float c_sum = 0.f;
        for (int p = P - 1; p >= 0; --p) c_sum += part[c * chunk + m * row + (int64_t)p * ldp + n];
        s += c_sum;
    }
    out[i] = s;
}

hipError_t launch_sum_planes(const float* part, int nchunk, int M, int N, int P, int ldp, float* out,
                             hipStream_t st) {
    const int64_t n = (int64_t)M * N;
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(sum_planes_kernel, dim3(grid_for(n, 256)), dim3(256), 0, st, part, nchunk, M, N, P, ldp,
                       out);
    return hipGetLastError();
}

int wgrad_chunks(int64_t rows, int M, int N) {
    // enough row chunks that the k-grouped GEMM has ~512 workgroups
    const int64_t per = (int64_t)((M + 127) / 128) * ((N + 255) / 256);
    int64_t n = (512 + per - 1) / per;
    const int64_t max_n = (rows + 255) / 256;
    if (n > max_n) n = max_n;
    if (n < 1) n = 1;
    if (n > 64) n = 64;
    return (int)n;
}

struct RouterBwdWs {
    float* ds; uint16_t* ds3; float* WrT; float* part; size_t bytes; int nchunk;
};

static int pad8(int e) { return (e + 7) / 8 * 8; }

static RouterBwdWs router_bwd_layout(char* base, int64_t S, int D, int E) {
    RouterBwdWs w{};
    size_t off = 0;
    auto take = [&](size_t bytes) { void* p = base ? base + off : nullptr; off += (bytes + 255) / 256 * 256; return p; };
    const int Ep = pad8(E);
    w.nchunk = wgrad_chunks(S, D, 3 * Ep);
    w.ds = (float*)take((size_t)S * E * 4);
    w.ds3 = (uint16_t*)take((size_t)S * 3 * Ep * 2);
    w.WrT = (float*)take((size_t)E * D * 4);
    w.part = (float*)take((size_t)w.nchunk * D * 3 * Ep * 4);
    w.bytes = off;
    return w;
}

size_t router_bwd_ws_bytes(int64_t S, int D, int E) { return router_bwd_layout(nullptr, S, D, E).bytes; }

hipError_t launch_router_bwd(const moe_bf16* x_r, const float* Wr, const int32_t* topk_idx, const float* topk_prob,
                             const float* dp, int64_t S, int D, int E, int K, float* dlogits, float* dWr,
                             float* dbias, float* dx_r, void* ws, hipStream_t st) {
    RouterBwdWs w = router_bwd_layout((char*)ws, S, D, E);
    float* ds = dlogits != nullptr ? dlogits : w.ds;
    const int Ep = pad8(E);
    hipError_t err;
    if (S > 0) {
        const int epl = (Ep + 63) / 64;
#define MOE_DS_CASE(N)                                                                                      \
    hipLaunchKernelGGL(router_ds_kernel<N>, dim3(grid_for(S, kRbTok)), dim3(256), 0, st, topk_idx, topk_prob, \
                       dp, S, E, Ep, K, ds, w.ds3)
        if (epl <= 1) MOE_DS_CASE(1);
        else if (epl <= 2) MOE_DS_CASE(2);
        else if (epl <= 4) MOE_DS_CASE(4);
        else if (epl <= 8) MOE_DS_CASE(8);
        else MOE_DS_CASE(16);
#undef MOE_DS_CASE
        if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    // dWr [D, E] = x_r^T [hi | mid | lo](ds), fp32 partials per row chunk
    const int64_t kchunk = S > 0 ? (S + w.nchunk - 1) / w.nchunk : 1;
    if ((err = launch_chunked_wgrad(x_r, D, (const moe_bf16*)w.ds3, 3 * (int64_t)Ep, w.part, 3 * (int64_t)Ep,
                                    (int64_t)D * 3 * Ep, w.nchunk, kchunk, D, 3 * Ep, S, st)) != hipSuccess)
        return err;
    // (an empty row range contributes zero partials: the k-grouped kernel writes its zero accumulators)
    if ((err = launch_sum_planes(w.part, w.nchunk, D, E, 3, Ep, dWr, st)) != hipSuccess) return err;
    if (dbias != nullptr) {
        hipLaunchKernelGGL(router_dbias_kernel, dim3((unsigned)((E + 3) / 4)), dim3(256), 0, st, ds, S, E, dbias);
        if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    if (dx_r != nullptr && S > 0) {
        hipLaunchKernelGGL(transpose_f32_kernel, dim3((unsigned)((E + 31) / 32), (unsigned)((D + 31) / 32)),
                           dim3(256), 0, st, Wr, D, E, w.WrT);
        hipLaunchKernelGGL(router_dx_kernel, dim3(grid_for(S, kRbTok)), dim3(256), 0, st, ds, topk_idx,
                           (const float4*)w.WrT, S, D / 4, E, K, (float4*)dx_r);
        if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    return hipSuccess;
}

}  // namespace moe
