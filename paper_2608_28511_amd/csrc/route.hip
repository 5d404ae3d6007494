// Top-K routing and the expert permutation on gfx950.
//
// Dropless top-K routing (Section 1) sends every token to exactly K distinct
// experts; the grouped-GEMM experts then need the S*K routed rows in
// expert-contiguous order (fused permutation, Section 5.2).  Three launches:
//
//   route_topk     one wavefront per token: K rounds of a wave-wide max over
//                  64-bit keys (orderable fp32 score | inverted expert id), so
//                  ties resolve to the lower expert id with no data-dependent
//                  order; renormalised softmax over the K winners; a per-block
//                  LDS bitmask per expert gives each (token, slot) its rank
//                  among the block's rows of that expert and the block's
//                  per-expert count.
//   route_scan     one workgroup: exclusive scan of the block counts along
//                  blocks (per expert) and of the totals along experts.
//   route_scatter  one thread per routed row: pos = offsets[e] + block base
//                  + rank; writes perm and inv_perm.
//
// No step depends on the order in which atomics land (the LDS OR is
// commutative and ranks come from popcounts), so the permutation is
// bit-for-bit deterministic.
#include "common.h"
#include "kernels.h"

namespace moe {

constexpr int kRouteTok = 32;  // tokens per block (one bit each in the masks)
constexpr int kRouteThreads = 256;
constexpr int kScanThreads = 1024;

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
    uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
    lo = __shfl_xor(lo, m);
    hi = __shfl_xor(hi, m);
    return ((uint64_t)hi << 32) | lo;
}

// Monotone map of an fp32 score to uint32 (larger score -> larger code).
// -0 is folded onto +0 and NaN maps to 0, below the code of -inf.
__device__ __forceinline__ uint32_t score_code(float f) {
    if (f != f) return 0u;
    uint32_t u = __float_as_uint(f);
    if (u == 0x80000000u) u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float code_score(uint32_t c) {
    uint32_t u = (c & 0x80000000u) ? (c & 0x7fffffffu) : ~c;
    return __uint_as_float(u);
}

template <int EPL>
__global__ __launch_bounds__(kRouteThreads) void route_topk_kernel(
    const float* __restrict__ logits, int64_t S, int E, int K, int32_t* __restrict__ topk_idx,
    float* __restrict__ topk_prob, int32_t* __restrict__ blkcnt, int32_t* __restrict__ rank_out) {
    __shared__ uint32_t mask[1024];
    __shared__ int16_t sel[kRouteTok][32];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t t_base = (int64_t)blockIdx.x * kRouteTok;
    for (int e = tid; e < E; e += kRouteThreads) mask[e] = 0u;
    __syncthreads();

    for (int j = wave; j < kRouteTok; j += kRouteThreads / kWave) {
        const int64_t t = t_base + j;
        if (t >= S) break;
        const float* row = logits + t * E;
        uint64_t key[EPL];
#pragma unroll
        for (int i = 0; i < EPL; ++i) {
            const int e = lane + kWave * i;
            key[i] = (e < E) ? (((uint64_t)score_code(row[e]) << 32) | (uint32_t)(0xffffu - e)) : 0ull;
        }
        int my_e = 0;
        float my_s = 0.f;
        for (int k = 0; k < K; ++k) {
            uint64_t best = key[0];
#pragma unroll
            for (int i = 1; i < EPL; ++i) best = key[i] > best ? key[i] : best;
#pragma unroll
            for (int m = 32; m > 0; m >>= 1) {
                const uint64_t o = shfl_xor_u64(best, m);
                best = o > best ? o : best;
            }
            const int e = 0xffff - (int)(uint32_t)(best & 0xffffffffu);
#pragma unroll
            for (int i = 0; i < EPL; ++i)
                if (lane + kWave * i == e) key[i] = 0ull;
            if (lane == k) {
                my_e = e;
                my_s = code_score((uint32_t)(best >> 32));
            }
        }
        const float s0 = __shfl(my_s, 0);
        float z = (lane < K) ? expf(my_s - s0) : 0.f;
        float sum = z;
#pragma unroll
        for (int m = 32; m > 0; m >>= 1) sum += __shfl_xor(sum, m);
        if (lane < K) {
            topk_idx[t * K + lane] = my_e;
            topk_prob[t * K + lane] = z / sum;
            sel[j][lane] = (int16_t)my_e;
            atomicOr(&mask[my_e], 1u << j);
        }
    }
    __syncthreads();

    const int n_tok = (int)((S - t_base) < kRouteTok ? (S - t_base) : kRouteTok);
    for (int q = tid; q < n_tok * K; q += kRouteThreads) {
        const int j = q / K, k = q - j * K;
        const int e = sel[j][k];
        rank_out[(t_base + j) * K + k] = __popc(mask[e] & ((1u << j) - 1u));
    }
    for (int e = tid; e < E; e += kRouteThreads)
        blkcnt[(int64_t)blockIdx.x * E + e] = __popc(mask[e]);
}

// One workgroup. blkcnt[b*E+e] (per-block counts) is replaced in place by the
// number of rows of expert e in blocks before b.  counts[e] = total rows of
// e; offsets = exclusive scan of counts with offsets[E] = total.
__global__ __launch_bounds__(kScanThreads) void route_scan_kernel(int32_t* __restrict__ blkcnt, int nblk,
                                                                  int E, int32_t* __restrict__ counts,
                                                                  int32_t* __restrict__ offsets) {
    __shared__ int32_t part[kScanThreads];
    __shared__ int32_t tot[kScanThreads];
    const int tid = threadIdx.x;
    int P = kScanThreads / E;
    if (P > 32) P = 32;
    if (P < 1) P = 1;
    const int chunk = (nblk + P - 1) / P;
    for (int e0 = 0; e0 < E; e0 += kScanThreads) {
        // lanes: e = e0 + tid % Ew, part index tid / Ew (Ew experts handled per pass)
        const int Ew = (E - e0) < kScanThreads / P ? (E - e0) : kScanThreads / P;
        const int e = e0 + tid % Ew;
        const int pi = tid / Ew;
        const bool active = pi < P && (tid < Ew * P);
        const int b0 = pi * chunk;
        const int b1 = (b0 + chunk) < nblk ? (b0 + chunk) : nblk;
        int s = 0;
        if (active)
            for (int b = b0; b < b1; ++b) s += blkcnt[(int64_t)b * E + e];
        part[tid] = s;
        __syncthreads();
        int before = 0, total = 0;
        if (active) {
            for (int q = 0; q < P; ++q) {
                const int v = part[q * Ew + (tid % Ew)];
                if (q < pi) before += v;
                total += v;
            }
            int run = before;
            for (int b = b0; b < b1; ++b) {
                const int64_t ix = (int64_t)b * E + e;
                const int c = blkcnt[ix];
                blkcnt[ix] = run;
                run += c;
            }
            if (pi == 0) tot[e] = total;
        }
        __syncthreads();
    }
    // exclusive scan of tot[0..E) (Hillis-Steele over 1024 slots)
    int v = tid < E ? tot[tid] : 0;
    if (tid < E) counts[tid] = v;
    part[tid] = v;
    __syncthreads();
    for (int d = 1; d < kScanThreads; d <<= 1) {
        const int add = tid >= d ? part[tid - d] : 0;
        __syncthreads();
        part[tid] += add;
        __syncthreads();
    }
    if (tid < E) offsets[tid + 1] = part[tid];
    if (tid == 0) offsets[0] = 0;
}

__global__ __launch_bounds__(256) void route_scatter_kernel(const int32_t* __restrict__ topk_idx,
                                                            const int32_t* __restrict__ blkbase,
                                                            const int32_t* __restrict__ offsets,
                                                            int32_t* __restrict__ inv_perm,
                                                            int32_t* __restrict__ perm, int64_t R,
                                                            int K, int E) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= R) return;
    const int64_t t = i / K;
    const int e = topk_idx[i];
    const int64_t b = t / kRouteTok;
    const int pos = offsets[e] + blkbase[b * E + e] + inv_perm[i];
    if ((uint32_t)pos >= (uint64_t)R) return;  // unreachable for consistent counts
    perm[pos] = (int32_t)i;
    inv_perm[i] = pos;
}

size_t route_ws_bytes(int64_t S, int E) {
    const int64_t nblk = (S + kRouteTok - 1) / kRouteTok;
    return (size_t)(((nblk * E * 4) + 255) / 256 * 256);
}

hipError_t launch_route(const float* logits, int64_t S, int E, int K, int32_t* topk_idx,
                        float* topk_prob, int32_t* counts, int32_t* offsets, int32_t* perm,
                        int32_t* inv_perm, void* ws, hipStream_t st) {
    const int nblk = (int)((S + kRouteTok - 1) / kRouteTok);
    int32_t* blkcnt = (int32_t*)ws;
    if (S > 0) {
        const int epl = (E + kWave - 1) / kWave;
#define MOE_ROUTE_CASE(N)                                                                      \
    hipLaunchKernelGGL(route_topk_kernel<N>, dim3(nblk), dim3(kRouteThreads), 0, st, logits, S, \
                       E, K, topk_idx, topk_prob, blkcnt, inv_perm)
        if (epl <= 1) MOE_ROUTE_CASE(1);
        else if (epl <= 2) MOE_ROUTE_CASE(2);
        else if (epl <= 4) MOE_ROUTE_CASE(4);
        else if (epl <= 8) MOE_ROUTE_CASE(8);
        else MOE_ROUTE_CASE(16);
#undef MOE_ROUTE_CASE
    }
    hipLaunchKernelGGL(route_scan_kernel, dim3(1), dim3(kScanThreads), 0, st, blkcnt, nblk, E,
                       counts, offsets);
    if (S > 0) {
        const int64_t R = S * K;
        hipLaunchKernelGGL(route_scatter_kernel, dim3(grid_for(R, 256)), dim3(256), 0, st, topk_idx,
                           blkcnt, offsets, inv_perm, perm, R, K, E);
    }
    return hipGetLastError();
}

}  // namespace moe
