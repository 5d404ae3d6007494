// Load balancing of the production router (Section 5.2) on gfx950: the
// sequence-level balance loss and the load-driven update of the
// selection-only expert bias.
//
// Loss (per sequence b of T tokens, sigmoid scores s, routed counts n):
//     loss = coeff / B * sum_b sum_e f_be P_be,
//     f_be = E / (K T) * n_be,   P_be = (1/T) sum_{t in b} s[t, e] / sum_e' s[t, e']
//          = coef * sum_b sum_e n_be * (sum_{t in b} s[t, e] / sum_e' s[t, e']),
//     coef = coeff * E / (K T^2 B).
//
//   seq_aux_partial_kernel  one workgroup per 64-token chunk of a sequence
//                           (chunks never straddle sequences), one wavefront
//                           per 16 tokens in order: each token's normalised
//                           scores are added to per-lane running sums, the
//                           four waves' sums are added in wave order, and the
//                           chunk's routed counts are an LDS histogram
//                           (integer, so the order of its atomics is moot);
//   seq_aux_expert_kernel   one workgroup per expert: per sequence the chunk
//                           partials in a fixed tree (fp64) and the routed
//                           count, summed n_be * P_be over sequences;
//   seq_aux_final_kernel    one workgroup: a fixed tree over experts.
// Every sum has a fixed order, so the loss is deterministic.
#include "common.h"
#include "kernels.h"

namespace moe {

constexpr int kAuxTok = 64;                 // tokens per chunk
constexpr int kAuxTokPerWave = kAuxTok / 4;  // 16

__device__ __forceinline__ float aux_sigmoid(float l) { return 1.f / (1.f + expf(-l)); }

template <int EPL>
__global__ __launch_bounds__(256) void seq_aux_partial_kernel(const float* __restrict__ logits,
                                                              const int32_t* __restrict__ topk_idx, int E, int K,
                                                              int64_t T, int nck, float* __restrict__ partP,
                                                              int32_t* __restrict__ partC) {
    __shared__ float red[4][1024];
    __shared__ int32_t cnt[1024];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t b = blockIdx.x / nck, c = blockIdx.x % nck;
    const int64_t t0 = b * T + c * kAuxTok;
    const int64_t t_end = (t0 + kAuxTok) < (b + 1) * T ? (t0 + kAuxTok) : (b + 1) * T;
    for (int e = tid; e < E; e += 256) cnt[e] = 0;
    __syncthreads();

    float acc[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) acc[i] = 0.f;
    for (int j = 0; j < kAuxTokPerWave; ++j) {
        const int64_t t = t0 + wave * kAuxTokPerWave + j;
        if (t >= t_end) break;
        float sg[EPL], part = 0.f;
#pragma unroll
        for (int i = 0; i < EPL; ++i) {
            const int e = lane + 64 * i;
            sg[i] = e < E ? aux_sigmoid(logits[t * E + e]) : 0.f;
            part += sg[i];
        }
#pragma unroll
        for (int msk = 32; msk > 0; msk >>= 1) part += __shfl_xor(part, msk);
#pragma unroll
        for (int i = 0; i < EPL; ++i) acc[i] += sg[i] / part;
        if (lane < K) {
            const int e = topk_idx[t * K + lane];
            if (e >= 0 && e < E) atomicAdd(&cnt[e], 1);
        }
    }
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
        const int e = lane + 64 * i;
        if (e < E) red[wave][e] = acc[i];
    }
    __syncthreads();
    for (int e = tid; e < E; e += 256) {
        partP[(int64_t)blockIdx.x * E + e] = ((red[0][e] + red[1][e]) + red[2][e]) + red[3][e];
        partC[(int64_t)blockIdx.x * E + e] = cnt[e];
    }
}

// Per expert (one workgroup each): for every sequence, the chunk partials in
// a fixed tree (fp64), the routed count, and term[e] = sum_b n_be P_be.
__global__ __launch_bounds__(256) void seq_aux_expert_kernel(const float* __restrict__ partP,
                                                             const int32_t* __restrict__ partC, int64_t B,
                                                             int nck, int E, double* __restrict__ term,
                                                             int32_t* __restrict__ seq_counts) {
    __shared__ double rp[256];
    __shared__ long long rc[256];
    const int tid = threadIdx.x, e = blockIdx.x;
    double t_e = 0.0;
    for (int64_t b = 0; b < B; ++b) {
        double P = 0.0;
        long long n = 0;
        for (int c = tid; c < nck; c += 256) {
            const int64_t ix = (b * nck + c) * E + e;
            P += (double)partP[ix];
            n += partC[ix];
        }
        rp[tid] = P;
        rc[tid] = n;
        __syncthreads();
        for (int w = 128; w > 0; w >>= 1) {
            if (tid < w) {
                rp[tid] += rp[tid + w];
                rc[tid] += rc[tid + w];
            }
            __syncthreads();
        }
        if (tid == 0) {
            if (seq_counts != nullptr) seq_counts[b * E + e] = (int32_t)rc[0];
            t_e += (double)rc[0] * rp[0];
        }
        __syncthreads();
    }
    if (tid == 0) term[e] = t_e;
}

// loss = coef * sum_e term[e], a fixed tree over the experts.
__global__ __launch_bounds__(1024) void seq_aux_final_kernel(const double* __restrict__ term, int E, double coef,
                                                             float* __restrict__ loss) {
    __shared__ double red[1024];
    const int tid = threadIdx.x;
    red[tid] = tid < E ? term[tid] : 0.0;
    __syncthreads();
    for (int w = 512; w > 0; w >>= 1) {
        if (tid < w) red[tid] += red[tid + w];
        __syncthreads();
    }
    if (tid == 0) loss[0] = (float)(coef * red[0]);
}

struct AuxWs {
    float* partP; int32_t* partC; double* term; size_t bytes; int nck;
};

static AuxWs aux_layout(char* base, int64_t S, int E, int64_t T) {
    AuxWs w{};
    size_t off = 0;
    auto take = [&](size_t bytes) { void* p = base ? base + off : nullptr; off += (bytes + 255) / 256 * 256; return p; };
    const int64_t B = T > 0 ? S / T : 0;
    w.nck = (int)((T + kAuxTok - 1) / kAuxTok);
    w.partP = (float*)take((size_t)(B * w.nck * E * 4));
    w.partC = (int32_t*)take((size_t)(B * w.nck * E * 4));
    w.term = (double*)take((size_t)E * 8);
    w.bytes = off;
    return w;
}

size_t seq_aux_ws_bytes(int64_t S, int E, int64_t seq_len) { return aux_layout(nullptr, S, E, seq_len).bytes; }

hipError_t launch_seq_aux_loss(const float* logits, const int32_t* topk_idx, int64_t S, int E, int K,
                               int64_t seq_len, double coef, float* loss, int32_t* seq_counts, void* ws,
                               hipStream_t st) {
    AuxWs w = aux_layout((char*)ws, S, E, seq_len);
    const int64_t B = S / seq_len;
    const int64_t nblk = B * w.nck;
    if (nblk > 0) {
        const int epl = (E + 63) / 64;
#define MOE_AUX_CASE(N)                                                                                  \
    hipLaunchKernelGGL(seq_aux_partial_kernel<N>, dim3((unsigned)nblk), dim3(256), 0, st, logits, topk_idx, \
                       E, K, seq_len, w.nck, w.partP, w.partC)
        if (epl <= 1) MOE_AUX_CASE(1);
        else if (epl <= 2) MOE_AUX_CASE(2);
        else if (epl <= 4) MOE_AUX_CASE(4);
        else if (epl <= 8) MOE_AUX_CASE(8);
        else MOE_AUX_CASE(16);
#undef MOE_AUX_CASE
        hipError_t err = launch_check(st);
        if (err != hipSuccess) return err;
    }
    hipLaunchKernelGGL(seq_aux_expert_kernel, dim3((unsigned)E), dim3(256), 0, st, w.partP, w.partC, B, w.nck, E,
                       w.term, seq_counts);
    const hipError_t err = launch_check(st);
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(seq_aux_final_kernel, dim3(1), dim3(1024), 0, st, w.term, E, coef, loss);
    return launch_check(st);
}

// sel_bias[e] += rate * sign(mean(counts) - counts[e]); the sign is taken
// exactly in integers as sign(sum(counts) - E * counts[e]).
__global__ __launch_bounds__(1024) void expert_bias_update_kernel(const int32_t* __restrict__ counts, int E,
                                                                  float rate, float* __restrict__ sel_bias) {
    __shared__ long long red[1024];
    const int tid = threadIdx.x;
    red[tid] = tid < E ? (long long)counts[tid] : 0;
    __syncthreads();
    for (int w = 512; w > 0; w >>= 1) {
        if (tid < w) red[tid] += red[tid + w];
        __syncthreads();
    }
    if (tid < E) {
        const long long d = red[0] - (long long)E * counts[tid];
        sel_bias[tid] += d > 0 ? rate : (d < 0 ? -rate : 0.f);
    }
}

hipError_t launch_expert_bias_update(const int32_t* counts, int E, float rate, float* sel_bias, hipStream_t st) {
    hipLaunchKernelGGL(expert_bias_update_kernel, dim3(1), dim3(1024), 0, st, counts, E, rate, sel_bias);
    return launch_check(st);
}

}  // namespace moe
