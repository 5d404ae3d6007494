// Top-K routing and the expert permutation on gfx950.
//
// Dropless top-K routing (Section 1) sends every token to exactly K distinct
// experts; the grouped-GEMM experts then need the S*K routed rows in
// expert-contiguous order (fused permutation, Section 5.2).  Three launches:
//
//   route_topk     32 tokens per workgroup, 2 per wavefront (16 waves, so
//                  each SIMD has several waves whose dependent max and
//                  ballot chains overlap), all loaded up front.  K rounds,
//                  each over the wave's two tokens together (two independent
//                  chains), of: wave-wide max of the orderable 32-bit score
//                  codes of the experts not yet picked (DPP within rows of 16
//                  lanes, then the 4 row maxima), a ballot for the lowest
//                  expert id holding that code (ties go to the lower id, NaN
//                  ranks below -inf), and clearing the winner's code.  Then the
//                  softmax renormalised over the K winners (or, for sigmoid
//                  scores, the winners' sigmoids over their sum), and a per-block
//                  LDS bitmask per expert that gives each (token, slot) its
//                  rank among the block's rows of that expert and the block's
//                  per-expert count.
//   route_colscan  per expert (parallel over experts): exclusive scan of the
//                  block counts along blocks, in place; the total is
//                  counts[e].
//   route_scatter  one thread per routed row; every workgroup first rebuilds
//                  offsets = exclusive scan of counts in LDS (the first one
//                  also stores it), then pos = offsets[e] + block base + rank
//                  gives perm and inv_perm.  In the fused layer it also
//                  writes each routed row's probability p_disp[pos] (the
//                  probability half of the dispatch payload), and one extra
//                  workgroup builds the grouped GEMM's tile tables from the
//                  offsets it holds, so the layer needs no dispatch launch.
//
// No step depends on the order in which atomics land (the LDS OR is
// commutative and ranks come from popcounts), so the permutation is
// bit-for-bit deterministic.
#include "common.h"
#include "kernels.h"
#include "schedule.h"

namespace moe {

constexpr int kRouteTok = 32;  // tokens per block (one bit each in the masks)
constexpr int kRouteThreads = 1024;
constexpr int kTokPerWave = kRouteTok / (kRouteThreads / kWave);  // 2
constexpr int kScanCols = 4;    // experts per route_colscan workgroup
constexpr int kScanThreads = 256;

// Monotone map of an fp32 score to uint32 (larger score -> larger code).
// -0 is folded onto +0 and NaN maps to 1, below the code of -inf (0x007fffff,
// the smallest code of a number); 0 is left for experts already picked or
// past E, so that removing a pick is clearing its code.
__device__ __forceinline__ uint32_t score_code(float f) {
    if (f != f) return 1u;
    uint32_t u = __float_as_uint(f);
    if (u == 0x80000000u) u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float code_score(uint32_t c) {
    uint32_t u = (c & 0x80000000u) ? (c & 0x7fffffffu) : ~c;
    return __uint_as_float(u);
}

// Router score of the production variant (Section 5.2): the logistic
// sigmoid in fp32 (-inf -> 0, +inf -> 1).
__device__ __forceinline__ float sigmoid_f32(float l) { return 1.f / (1.f + expf(-l)); }

// Maximum of v over the 64 lanes (all active), returned wave-uniform.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
    // pairs, quads, half rows, rows of 16 lanes: full permutations within a row
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xf, 0xf, false));   // quad_perm 1,0,3,2
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xf, 0xf, false));   // quad_perm 2,3,0,1
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xf, 0xf, false));  // row_half_mirror
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xf, 0xf, false));  // row_mirror
    const uint32_t a = __builtin_amdgcn_readlane(v, 0), b = __builtin_amdgcn_readlane(v, 16);
    const uint32_t c = __builtin_amdgcn_readlane(v, 32), d = __builtin_amdgcn_readlane(v, 48);
    return max(max(a, b), max(c, d));
}

// SIG false: selection by the logits, weights = softmax over the K picked.
// SIG true: selection by sigmoid(logit) + sel_bias (bias may be null), weights
// = the picked sigmoids over their sum; the bias only steers selection.
template <int EPL, bool SIG>
__global__ __launch_bounds__(kRouteThreads) void route_topk_kernel(
    const float* __restrict__ logits, const float* __restrict__ sel_bias, int64_t S, int E, int K,
    int32_t* __restrict__ topk_idx, float* __restrict__ topk_prob, int32_t* __restrict__ blkcnt,
    int32_t* __restrict__ rank_out) {
    __shared__ uint32_t mask[1024];
    __shared__ int16_t sel[kRouteTok][32];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t t_base = (int64_t)blockIdx.x * kRouteTok;
    for (int e = tid; e < E; e += kRouteThreads) mask[e] = 0u;

    // this wave's tokens t_base + wave*8 + j: every score code loaded up front
    uint32_t code[kTokPerWave][EPL];
    float bias[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
        const int e = lane + kWave * i;
        bias[i] = (SIG && sel_bias != nullptr && e < E) ? sel_bias[e] : 0.f;
    }
#pragma unroll
    for (int j = 0; j < kTokPerWave; ++j) {
        const int64_t t = t_base + wave * kTokPerWave + j;
#pragma unroll
        for (int i = 0; i < EPL; ++i) {
            const int e = lane + kWave * i;
            if (t < S && e < E) {
                const float l = logits[t * E + e];
                code[j][i] = score_code(SIG ? sigmoid_f32(l) + bias[i] : l);
            } else {
                code[j][i] = 0u;
            }
        }
    }
    __syncthreads();

    // K rounds for the wave's tokens together (independent chains the
    // scheduler interleaves).  Every code of an expert not yet picked is >= 1
    // and K <= E, so a round's maximum is never a cleared code (a token past
    // S has only cleared codes; its picks are never stored).  Lane k keeps
    // the k-th pick of each token and its code.
    int my_e[kTokPerWave] = {};
    uint32_t my_c[kTokPerWave] = {};
    for (int k = 0; k < K; ++k) {
#pragma unroll
        for (int j = 0; j < kTokPerWave; ++j) {
            uint32_t m = code[j][0];
#pragma unroll
            for (int i = 1; i < EPL; ++i) m = max(m, code[j][i]);
            m = wave_max_u32(m);
            // the lowest expert id holding m: the lowest slot i with a
            // match, then its lowest lane
            int e_sel = 0;
#pragma unroll
            for (int i = EPL - 1; i >= 0; --i) {
                const uint64_t b = __ballot(code[j][i] == m);
                if (b != 0) e_sel = kWave * i + (__ffsll((unsigned long long)b) - 1);
            }
            const bool own = lane == (e_sel & (kWave - 1));
#pragma unroll
            for (int i = 0; i < EPL; ++i)
                if (own && i == (e_sel >> 6)) code[j][i] = 0u;
            if (lane == k) {
                my_e[j] = e_sel;
                my_c[j] = m;
            }
        }
    }

#pragma unroll
    for (int j = 0; j < kTokPerWave; ++j) {
        const int jt = wave * kTokPerWave + j;
        const int64_t t = t_base + jt;
        if (t >= S) break;
        const float my_s = code_score(my_c[j]);
        float z;
        if constexpr (SIG) {
            z = (lane < K) ? sigmoid_f32(logits[t * E + my_e[j]]) : 0.f;
        } else {
            const float s0 = __shfl(my_s, 0);
            z = (lane < K) ? expf(my_s - s0) : 0.f;
        }
        float sum = z;
#pragma unroll
        for (int msk = 32; msk > 0; msk >>= 1) sum += __shfl_xor(sum, msk);
        if (lane < K) {
            topk_idx[t * K + lane] = my_e[j];
            topk_prob[t * K + lane] = z / sum;
            sel[jt][lane] = (int16_t)my_e[j];
            atomicOr(&mask[my_e[j]], 1u << jt);
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

// blkcnt[b*E+e] (rows of expert e in token block b) is replaced in place by
// the rows of e in blocks before b; counts[e] = all rows of e.  A workgroup
// takes kScanCols experts; its 256 threads split the blocks into 64 chunks.
__global__ __launch_bounds__(kScanThreads) void route_colscan_kernel(int32_t* __restrict__ blkcnt, int nblk,
                                                                     int E, int32_t* __restrict__ counts) {
    constexpr int kChunks = kScanThreads / kScanCols;  // 64
    __shared__ int32_t part[kChunks][kScanCols];
    const int tid = threadIdx.x;
    const int c = tid % kScanCols, q = tid / kScanCols;
    const int e = blockIdx.x * kScanCols + c;
    const int chunk = (nblk + kChunks - 1) / kChunks;
    const int b0 = q * chunk;
    const int b1 = (b0 + chunk) < nblk ? (b0 + chunk) : nblk;
    int s = 0;
    if (e < E)
        for (int b = b0; b < b1; ++b) s += blkcnt[(int64_t)b * E + e];
    part[q][c] = s;
    __syncthreads();
    if (e >= E) return;
    int before = 0, total = 0;
    for (int r = 0; r < kChunks; ++r) {
        const int v = part[r][c];
        before += r < q ? v : 0;
        total += v;
    }
    int run = before;
    for (int b = b0; b < b1; ++b) {
        const int64_t ix = (int64_t)b * E + e;
        const int v = blkcnt[ix];
        blkcnt[ix] = run;
        run += v;
    }
    if (q == 0) counts[e] = total;
}

__global__ __launch_bounds__(256) void route_scatter_kernel(const int32_t* __restrict__ topk_idx,
                                                            const int32_t* __restrict__ blkbase,
                                                            const int32_t* __restrict__ counts,
                                                            int32_t* __restrict__ offsets,
                                                            int32_t* __restrict__ inv_perm,
                                                            int32_t* __restrict__ perm, int64_t R,
                                                            int K, int E, const float* __restrict__ prob,
                                                            float* __restrict__ p_disp, int sched_wg,
                                                            SchedPart sched_small, SchedPart sched_large) {
    __shared__ int32_t off[1024], seg_hi[1024];
    __shared__ int32_t wsum[4];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // exclusive scan of counts[0..E): each thread owns 4 consecutive experts
    int v[4], run = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int e = tid * 4 + u;
        v[u] = e < E ? counts[e] : 0;
        run += v[u];
    }
    int incl = run;  // inclusive scan of the per-thread sums within the wave
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        const int o = __shfl_up(incl, d);
        if (lane >= d) incl += o;
    }
    if (lane == kWave - 1) wsum[wave] = incl;
    __syncthreads();
    int base = incl - run;
    for (int w = 0; w < wave; ++w) base += wsum[w];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int e = tid * 4 + u;
        if (e < E) off[e] = base;
        base += v[u];
    }
    __syncthreads();
    if ((int)blockIdx.x == sched_wg) {
        // the tile tables from the segments [off[e], off[e+1]) held here,
        // clamped to [0, R) as the standalone builder clamps them
        const int total = wsum[0] + wsum[1] + wsum[2] + wsum[3];
        for (int e = tid; e < E; e += 256) seg_hi[e] = e + 1 < E ? off[e + 1] : total;
        __syncthreads();
        for (int e = tid; e < E; e += 256) {
            const int lo = off[e] < (int)R ? off[e] : (int)R;
            const int hi = seg_hi[e];
            off[e] = lo;
            seg_hi[e] = hi < lo ? lo : (hi > (int)R ? (int)R : hi);
        }
        __syncthreads();
        build_tile_schedule_lds(off, seg_hi, E, sched_small, sched_large);
        return;
    }
    if (blockIdx.x == 0) {
        for (int e = tid; e < E; e += 256) offsets[e] = off[e];
        if (tid == 0) offsets[E] = wsum[0] + wsum[1] + wsum[2] + wsum[3];
    }

    const int64_t i = (int64_t)blockIdx.x * blockDim.x + tid;
    if (i >= R) return;
    const int64_t t = i / K;
    const int e = topk_idx[i];
    const int64_t b = t / kRouteTok;
    const int pos = off[e] + blkbase[b * E + e] + inv_perm[i];
    if ((uint32_t)pos >= (uint64_t)R) return;  // unreachable for consistent counts
    perm[pos] = (int32_t)i;
    inv_perm[i] = pos;
    if (p_disp != nullptr) p_disp[pos] = prob[i];
}

size_t route_ws_bytes(int64_t S, int E) {
    const int64_t nblk = (S + kRouteTok - 1) / kRouteTok;
    return (size_t)(((nblk * E * 4) + 255) / 256 * 256);
}

template <bool SIG>
static void launch_topk(const float* logits, const float* sel_bias, int64_t S, int E, int K, int32_t* topk_idx,
                        float* topk_prob, int32_t* blkcnt, int32_t* rank, int nblk, hipStream_t st) {
    const int epl = (E + kWave - 1) / kWave;
#define MOE_ROUTE_CASE(N)                                                                          \
    hipLaunchKernelGGL((route_topk_kernel<N, SIG>), dim3(nblk), dim3(kRouteThreads), 0, st, logits, \
                       sel_bias, S, E, K, topk_idx, topk_prob, blkcnt, rank)
    if (epl <= 1) MOE_ROUTE_CASE(1);
    else if (epl <= 2) MOE_ROUTE_CASE(2);
    else if (epl <= 4) MOE_ROUTE_CASE(4);
    else if (epl <= 8) MOE_ROUTE_CASE(8);
    else MOE_ROUTE_CASE(16);
#undef MOE_ROUTE_CASE
}

hipError_t launch_route(const float* logits, int64_t S, int E, int K, int32_t* topk_idx,
                        float* topk_prob, int32_t* counts, int32_t* offsets, int32_t* perm,
                        int32_t* inv_perm, void* ws, hipStream_t st, bool sigmoid, const float* sel_bias,
                        float* p_disp, void* sched) {
    const int nblk = (int)((S + kRouteTok - 1) / kRouteTok);
    int32_t* blkcnt = (int32_t*)ws;
    if (S > 0) {
        if (sigmoid)
            launch_topk<true>(logits, sel_bias, S, E, K, topk_idx, topk_prob, blkcnt, inv_perm, nblk, st);
        else
            launch_topk<false>(logits, nullptr, S, E, K, topk_idx, topk_prob, blkcnt, inv_perm, nblk, st);
        const hipError_t e1 = launch_check(st);
        if (e1 != hipSuccess) return e1;
    }
    hipLaunchKernelGGL(route_colscan_kernel, dim3((unsigned)((E + kScanCols - 1) / kScanCols)),
                       dim3(kScanThreads), 0, st, blkcnt, nblk, E, counts);
    const hipError_t e2 = launch_check(st);
    if (e2 != hipSuccess) return e2;
    const int64_t R = S * K;
    // at least one workgroup, so that offsets are written even for S == 0;
    // with sched, one more (the last) builds the tile tables
    const unsigned grid = R > 0 ? grid_for(R, 256) : 1u;
    const SchedPart ss = sched ? sched_part(sched, E, R, false) : SchedPart{};
    const SchedPart sl = sched ? sched_part(sched, E, R, true) : SchedPart{};
    hipLaunchKernelGGL(route_scatter_kernel, dim3(grid + (sched ? 1u : 0u)), dim3(256), 0, st, topk_idx, blkcnt,
                       counts, offsets, inv_perm, perm, R, K, E, topk_prob, p_disp, sched ? (int)grid : -1, ss, sl);
    return launch_check(st);
}

}  // namespace moe
