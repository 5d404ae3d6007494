// Top-K routing and the expert permutation on gfx950.
//
// Dropless top-K routing (Section 1) sends every token to exactly K distinct
// experts; the grouped-GEMM experts then need the S*K routed rows in
// expert-contiguous order (fused permutation, Section 5.2).  Two launches:
//
//   route_topk     32 tokens per workgroup, one per row of 16 lanes (four per
//                  wavefront), all scores loaded up front; lane r of a row
//                  holds experts r + 16 i.  K rounds of: the row maximum of
//                  the orderable 32-bit score codes of the experts not yet
//                  picked (DPP within the row), the lowest expert id holding
//                  it (ties go to the lower id, NaN ranks below -inf; a
//                  lane's lowest matching slot, then the row minimum), and
//                  clearing the winner's code.  Then the softmax renormalised
//                  over the K winners (or, for sigmoid scores, the winners'
//                  sigmoids over their sum), and a per-block LDS bitmask per
//                  expert that gives each (token, slot) its rank among the
//                  block's rows of that expert and the block's per-expert
//                  count, stored as one byte (at most 32) in an expert-major
//                  count matrix [E][blocks].
//   route_scatter  each workgroup first sums, for every expert, its row of
//                  the count matrix in full (counts, then offsets by an
//                  exclusive scan in LDS; the first workgroup stores both)
//                  and up to its own first token block (the expert's rows in
//                  earlier blocks), four bytes per dot-product instruction;
//                  then pos = offsets[e] + rows in earlier blocks + rank
//                  gives perm and inv_perm for the rows of its blocks (all
//                  of them in one pass when their per-block prefixes fit in
//                  LDS).  In the fused layer it also writes each routed
//                  row's probability p_disp[pos] (the probability half of
//                  the dispatch payload), and eight extra workgroups each
//                  write a slice of the grouped GEMM's tile tables from the
//                  offsets they hold, so the layer needs no dispatch launch.
//                  Every workgroup reads the whole count matrix, so the
//                  blocks are dealt to at most 256 workgroups.
//
// No step depends on the order in which atomics land (the LDS OR is
// commutative and ranks come from popcounts), so the permutation is
// bit-for-bit deterministic.
#include "common.h"
#include "kernels.h"
#include "schedule.h"

namespace moe {

constexpr int kRouteTok = 32;  // tokens per block (one bit each in the masks)
constexpr int kScatThreads = 256;
constexpr int kScatMaxWg = 256;   // scatter workgroups (each reads the whole count matrix)
constexpr int kPfxInts = 8192;    // LDS per-block prefixes of a scatter workgroup (blocks x experts)

// Row length in bytes of the expert-major count matrix: the token blocks
// rounded up to whole 16-byte chunks (the padding bytes are zero).
inline __host__ __device__ int64_t cnt_row_bytes(int64_t nblk) { return (nblk + 15) / 16 * 16; }

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

// v plus its DPP-permuted copy (lanes of rows outside the row mask add 0).
template <int CTRL, int ROWS>
__device__ __forceinline__ float dpp_add(float x) {
    return x + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, ROWS, 0xf, false));
}

// Sum of the 16 count bytes of a chunk, and of its bytes before position lim.
__device__ __forceinline__ uint32_t bytes_sum(const uint4& c) {
    uint32_t s = __builtin_amdgcn_udot4(c.x, 0x01010101u, 0u, false);
    s = __builtin_amdgcn_udot4(c.y, 0x01010101u, s, false);
    s = __builtin_amdgcn_udot4(c.z, 0x01010101u, s, false);
    return __builtin_amdgcn_udot4(c.w, 0x01010101u, s, false);
}
__device__ __forceinline__ uint32_t bytes_sum_below(const uint4& c, int lim) {
    const uint32_t w[4] = {c.x, c.y, c.z, c.w};
    uint32_t s = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int n = lim - 4 * q;   // bytes of word q below lim
        const uint32_t m = n >= 4 ? 0xffffffffu : (n <= 0 ? 0u : (1u << (8 * n)) - 1u);
        s = __builtin_amdgcn_udot4(w[q] & m, 0x01010101u, s, false);
    }
    return s;
}

// Chunks c = c0, c0 + step, ... < nchunk of one count row: tot += all their
// bytes, pre += the bytes of blocks before chunk cb0's byte lim0.  Eight
// chunks are loaded before any is summed, so the loads overlap.
__device__ __forceinline__ void row_sums(const uint8_t* row8, int64_t c0, int step, int64_t nchunk, int64_t cb0,
                                         int lim0, uint32_t& tot, uint32_t& pre) {
    constexpr int kU = 8;
    const uint4* row = (const uint4*)row8;
    for (int64_t cb = c0; cb < nchunk; cb += (int64_t)kU * step) {
        uint4 v[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int64_t c = cb + (int64_t)u * step;
            v[u] = c < nchunk ? row[c] : make_uint4(0u, 0u, 0u, 0u);
        }
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int64_t c = cb + (int64_t)u * step;
            const uint32_t s = bytes_sum(v[u]);
            tot += s;
            pre += c < cb0 ? s : (c == cb0 ? bytes_sum_below(v[u], lim0) : 0u);
        }
    }
}

// Row form: one token per row of 16 lanes, so a wave holds four tokens and
// one instruction stream serves all four.  Lane r of a row holds experts
// r + 16 i (slot i < EPR); the row maximum and the lowest expert id holding
// it are both DPP reductions within the row (no readlane, no scalar chain),
// and lane r keeps picks r and r + 16 (K <= 32).
constexpr int kRowThreads = kRouteTok * 16;   // 512: 8 waves of 4 tokens

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xf, 0xf, false);
}
__device__ __forceinline__ uint32_t row_max_u32(uint32_t v) {
    v = max(v, dpp_u32<0xB1>(v));    // quad_perm 1,0,3,2
    v = max(v, dpp_u32<0x4E>(v));    // quad_perm 2,3,0,1
    v = max(v, dpp_u32<0x141>(v));   // row_half_mirror
    return max(v, dpp_u32<0x140>(v));   // row_mirror
}
__device__ __forceinline__ uint32_t row_min_u32(uint32_t v) {
    v = min(v, dpp_u32<0xB1>(v));
    v = min(v, dpp_u32<0x4E>(v));
    v = min(v, dpp_u32<0x141>(v));
    return min(v, dpp_u32<0x140>(v));
}
__device__ __forceinline__ float row_sum_f32(float v) {
    v = dpp_add<0xB1, 0xf>(v);
    v = dpp_add<0x4E, 0xf>(v);
    v = dpp_add<0x141, 0xf>(v);
    return dpp_add<0x140, 0xf>(v);
}

template <int EPR, bool SIG>
__global__ __launch_bounds__(kRowThreads) void route_topk_rows_kernel(
    const float* __restrict__ logits, const float* __restrict__ sel_bias, int64_t S, int E, int K,
    int32_t* __restrict__ topk_idx, float* __restrict__ topk_prob, uint8_t* __restrict__ blkcnt,
    int64_t nbp, int32_t* __restrict__ rank_out) {
    __shared__ uint32_t mask[1024];
    __shared__ int16_t sel[kRouteTok][32];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int r = lane & 15, jt = wave * 4 + (lane >> 4);
    const int64_t t_base = (int64_t)blockIdx.x * kRouteTok;
    const int64_t t = t_base + jt;
    for (int e = tid; e < E; e += kRowThreads) mask[e] = 0u;

    // every score loaded before any is used (entries past S or E read
    // element 0, which exists, and are masked afterwards)
    uint32_t code[EPR];
    {
        float l[EPR], bias[EPR];
#pragma unroll
        for (int i = 0; i < EPR; ++i) {
            const int e = r + 16 * i;
            bias[i] = 0.f;
            if constexpr (SIG) bias[i] = sel_bias != nullptr ? sel_bias[e < E ? e : 0] : 0.f;
            l[i] = logits[(t < S && e < E) ? t * E + e : 0];
        }
#pragma unroll
        for (int i = 0; i < EPR; ++i) {
            const int e = r + 16 * i;
            const uint32_t c = score_code(SIG ? sigmoid_f32(l[i]) + bias[i] : l[i]);
            code[i] = (t < S && e < E) ? c : 0u;
        }
    }
    __syncthreads();

    // K rounds: the row's maximum code (never a cleared one: K <= E), the
    // lowest expert id holding it (a lane's lowest matching slot, then the
    // row minimum), and clearing it.  Lane k % 16 of the row keeps the k-th
    // pick, in its slot k / 16.
    int my_e[2] = {0, 0};
    uint32_t my_c[2] = {0u, 0u};
    for (int k = 0; k < K; ++k) {
        uint32_t m = code[0];
#pragma unroll
        for (int i = 1; i < EPR; ++i) m = max(m, code[i]);
        m = row_max_u32(m);
        uint32_t cand = 0xffffu;
#pragma unroll
        for (int i = EPR - 1; i >= 0; --i) cand = code[i] == m ? (uint32_t)(r + 16 * i) : cand;
        const int e_sel = (int)row_min_u32(cand);
        const bool own = r == (e_sel & 15);
#pragma unroll
        for (int i = 0; i < EPR; ++i)
            if (own && i == (e_sel >> 4)) code[i] = 0u;
        if (r == (k & 15)) {
            if (k < 16) {
                my_e[0] = e_sel;
                my_c[0] = m;
            } else {
                my_e[1] = e_sel;
                my_c[1] = m;
            }
        }
    }

    const bool has0 = r < K, has1 = r + 16 < K;
    float z0, z1;
    if constexpr (SIG) {
        z0 = (has0 && t < S) ? sigmoid_f32(logits[t * E + my_e[0]]) : 0.f;
        z1 = (has1 && t < S) ? sigmoid_f32(logits[t * E + my_e[1]]) : 0.f;
    } else {
        const float s0 = code_score((uint32_t)__shfl((int)my_c[0], lane & 48));
        z0 = has0 ? expf(code_score(my_c[0]) - s0) : 0.f;
        z1 = has1 ? expf(code_score(my_c[1]) - s0) : 0.f;
    }
    const float sum = row_sum_f32(z0 + z1);
    if (t < S) {
        if (has0) {
            topk_idx[t * K + r] = my_e[0];
            topk_prob[t * K + r] = z0 / sum;
            sel[jt][r] = (int16_t)my_e[0];
            atomicOr(&mask[my_e[0]], 1u << jt);
        }
        if (has1) {
            topk_idx[t * K + r + 16] = my_e[1];
            topk_prob[t * K + r + 16] = z1 / sum;
            sel[jt][r + 16] = (int16_t)my_e[1];
            atomicOr(&mask[my_e[1]], 1u << jt);
        }
    }
    __syncthreads();

    const int n_tok = (int)((S - t_base) < kRouteTok ? (S - t_base) : kRouteTok);
    for (int q = tid; q < n_tok * K; q += kRowThreads) {
        const int j = q / K, k = q - j * K;
        const int e = sel[j][k];
        rank_out[(t_base + j) * K + k] = __popc(mask[e] & ((1u << j) - 1u));
    }
    for (int e = tid; e < E; e += kRowThreads)
        blkcnt[(int64_t)e * nbp + blockIdx.x] = (uint8_t)__popc(mask[e]);
    // the last block also zeroes every row's padding bytes
    const int64_t nblk = gridDim.x;
    if ((int64_t)blockIdx.x == nblk - 1) {
        const int pad = (int)(nbp - nblk);
        for (int q = tid; q < E * pad; q += kRowThreads)
            blkcnt[(int64_t)(q / pad) * nbp + nblk + q % pad] = 0;
    }
}

// Inclusive prefix sums out[e] = v(0) + ... + v(e) over e < E <= 1024, by a
// workgroup of kScatThreads threads (4 consecutive entries each); returns the
// total.  wsum is LDS scratch of 4 entries; out may be read after the call.
template <class V>
__device__ __forceinline__ int wg_incl_scan(V v, int E, int32_t* out, int32_t* wsum) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int x[4], acc = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int e = tid * 4 + u;
        x[u] = e < E ? v(e) : 0;
        acc += x[u];
    }
    int incl = acc;  // inclusive scan of the per-thread sums within the wave
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        const int o = __shfl_up(incl, d);
        if (lane >= d) incl += o;
    }
    __syncthreads();   // earlier readers of wsum are done
    if (lane == kWave - 1) wsum[wave] = incl;
    __syncthreads();
    int base = incl - acc;
    for (int w = 0; w < wave; ++w) base += wsum[w];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int e = tid * 4 + u;
        base += x[u];
        if (e < E) out[e] = base;
    }
    const int total = wsum[0] + wsum[1] + wsum[2] + wsum[3];
    __syncthreads();
    return total;
}

// Workgroup w < nrow takes token blocks [w * bpw, min((w + 1) * bpw, nblk)).
// With the tile tables requested (sched_small.tiles != null), the workgroups
// nrow .. gridDim.x - 1 each write one slice of both tables instead, while
// the others place rows.
__global__ __launch_bounds__(kScatThreads) void route_scatter_kernel(
    const int32_t* __restrict__ topk_idx, const uint8_t* __restrict__ blkcnt, int64_t nblk, int64_t nbp, int bpw,
    int nrow, int32_t* __restrict__ counts, int32_t* __restrict__ offsets, int32_t* __restrict__ inv_perm,
    int32_t* __restrict__ perm, int64_t S, int K, int E, const float* __restrict__ prob,
    float* __restrict__ p_disp, SchedPart sched_small, SchedPart sched_large) {
    __shared__ int32_t cnt[1024], off[1024], run[1024], seg_lo[1024], seg_hi[1024];
    __shared__ int32_t pfx[kPfxInts];
    __shared__ int32_t wsum[4];
    const int tid = threadIdx.x;
    const bool tab = (int)blockIdx.x >= nrow;
    const int64_t b0 = tab ? 0 : (int64_t)blockIdx.x * bpw;
    const int64_t b1 = tab ? 0 : (b0 + bpw < nblk ? b0 + bpw : nblk);

    // 1. per expert: rows in all blocks (cnt) and in blocks before b0 (run).
    // tpe adjacent lanes share an expert's row (E <= 128) and combine their
    // sums with xor shuffles; above 128 experts each lane takes whole rows.
    const int64_t nchunk = nbp / 16;
    const int64_t cb0 = b0 / 16;
    const int lim0 = (int)(b0 % 16);
    if (E <= 128) {
        int tpe = 64;
        while (tpe * E > kScatThreads) tpe >>= 1;
        const int e = tid / tpe, part = tid % tpe;
        uint32_t tot = 0, pre = 0;
        if (e < E) row_sums(blkcnt + (int64_t)e * nbp, part, tpe, nchunk, cb0, lim0, tot, pre);
        for (int m = 1; m < tpe; m <<= 1) {
            tot += __shfl_xor(tot, m);
            pre += __shfl_xor(pre, m);
        }
        if (e < E && part == 0) {
            cnt[e] = (int32_t)tot;
            run[e] = (int32_t)pre;
        }
    } else {
        for (int e = tid; e < E; e += kScatThreads) {
            uint32_t tot = 0, pre = 0;
            row_sums(blkcnt + (int64_t)e * nbp, 0, 1, nchunk, cb0, lim0, tot, pre);
            cnt[e] = (int32_t)tot;
            run[e] = (int32_t)pre;
        }
    }
    __syncthreads();

    // 2. offsets = exclusive scan of the counts (seg_hi holds the inclusive one)
    const int total = wg_incl_scan([&](int e) { return cnt[e]; }, E, seg_hi, wsum);
    for (int e = tid; e < E; e += kScatThreads) off[e] = seg_hi[e] - cnt[e];
    const int64_t R = S * K;
    if (blockIdx.x == 0) {
        for (int e = tid; e < E; e += kScatThreads) {
            offsets[e] = seg_hi[e] - cnt[e];
            counts[e] = cnt[e];
        }
        if (tid == 0) offsets[E] = total;
    }
    __syncthreads();

    // the tile tables: segments clamped to [0, R) as the standalone builder
    // clamps them; each height's tile counts scanned into cnt, then this
    // workgroup's slice of the table
    if (tab) {
        for (int e = tid; e < E; e += kScatThreads) {
            const int lo = off[e] < (int)R ? off[e] : (int)R;
            const int hi = seg_hi[e];
            seg_lo[e] = lo;
            seg_hi[e] = hi < lo ? lo : (hi > (int)R ? (int)R : hi);
        }
        __syncthreads();
        const int ntab = (int)gridDim.x - nrow, slice = (int)blockIdx.x - nrow;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const SchedPart& sp = h ? sched_large : sched_small;
            const int bm = kSchedBM[h];
            wg_incl_scan([&](int e) { return (seg_hi[e] - seg_lo[e] + bm - 1) / bm; }, E, cnt, wsum);
            const int per = (sp.max_tiles + ntab - 1) / ntab;
            const int mt0 = slice * per;
            sched_fill_slice(seg_lo, seg_hi, cnt, E, bm, sp, mt0, mt0 + per, slice == 0);
            __syncthreads();   // cnt is rescanned for the next height
        }
        return;
    }

    // 3. the rows of blocks b0 .. b1 - 1.  When their per-block prefixes fit
    // in LDS (pfx[(b - b0) * E + e] = rows of e in blocks before b), all rows
    // are placed in one pass; else one block at a time, run[e] holding the
    // rows of e in the blocks before the current one.
    const int nb = (int)(b1 - b0);
    if (nb > 1 && nb * E <= kPfxInts) {
        for (int e = tid; e < E; e += kScatThreads) {
            int acc = run[e];
            for (int q = 0; q < nb; ++q) {
                pfx[q * E + e] = acc;
                acc += blkcnt[(int64_t)e * nbp + b0 + q];
            }
        }
        __syncthreads();
        const int64_t t1 = b1 * kRouteTok < S ? b1 * kRouteTok : S;
        for (int64_t i = b0 * kRouteTok * K + tid; i < t1 * K; i += kScatThreads) {
            const int e = topk_idx[i];
            if ((unsigned)e >= (unsigned)E) continue;   // unreachable: top-K writes ids below E
            const int q = (int)(i / K / kRouteTok - b0);
            const int pos = off[e] + pfx[q * E + e] + inv_perm[i];
            if ((uint64_t)(uint32_t)pos >= (uint64_t)R) continue;  // unreachable for consistent counts
            perm[pos] = (int32_t)i;
            inv_perm[i] = pos;
            if (p_disp != nullptr) p_disp[pos] = prob[i];
        }
        return;
    }
    for (int64_t b = b0; b < b1; ++b) {
        const int64_t r0 = b * kRouteTok * K;
        const int64_t t1 = (b + 1) * kRouteTok < S ? (b + 1) * kRouteTok : S;
        for (int64_t i = r0 + tid; i < t1 * K; i += kScatThreads) {
            const int e = topk_idx[i];
            if ((unsigned)e >= (unsigned)E) continue;   // unreachable: top-K writes ids below E
            const int pos = off[e] + run[e] + inv_perm[i];
            if ((uint64_t)(uint32_t)pos >= (uint64_t)R) continue;  // unreachable for consistent counts
            perm[pos] = (int32_t)i;
            inv_perm[i] = pos;
            if (p_disp != nullptr) p_disp[pos] = prob[i];
        }
        if (b + 1 < b1) {
            __syncthreads();
            for (int e = tid; e < E; e += kScatThreads) run[e] += blkcnt[(int64_t)e * nbp + b];
            __syncthreads();
        }
    }
}

size_t route_ws_bytes(int64_t S, int E) {
    const int64_t nblk = (S + kRouteTok - 1) / kRouteTok;
    return (size_t)((cnt_row_bytes(nblk) * E + 255) / 256 * 256);
}

template <bool SIG>
static void launch_topk(const float* logits, const float* sel_bias, int64_t S, int E, int K, int32_t* topk_idx,
                        float* topk_prob, uint8_t* blkcnt, int64_t nbp, int32_t* rank, int nblk, hipStream_t st) {
    const int epr = (E + 15) / 16;   // E <= 1024: at most 64 slots per lane
#define MOE_ROUTE_ROWS(N)                                                                           \
    hipLaunchKernelGGL((route_topk_rows_kernel<N, SIG>), dim3(nblk), dim3(kRowThreads), 0, st, logits, \
                       sel_bias, S, E, K, topk_idx, topk_prob, blkcnt, nbp, rank)
    if (epr <= 1) MOE_ROUTE_ROWS(1);
    else if (epr <= 2) MOE_ROUTE_ROWS(2);
    else if (epr <= 4) MOE_ROUTE_ROWS(4);
    else if (epr <= 8) MOE_ROUTE_ROWS(8);
    else if (epr <= 16) MOE_ROUTE_ROWS(16);
    else if (epr <= 24) MOE_ROUTE_ROWS(24);
    else if (epr <= 32) MOE_ROUTE_ROWS(32);
    else if (epr <= 40) MOE_ROUTE_ROWS(40);
    else if (epr <= 48) MOE_ROUTE_ROWS(48);
    else MOE_ROUTE_ROWS(64);
#undef MOE_ROUTE_ROWS
}

hipError_t launch_route(const float* logits, int64_t S, int E, int K, int32_t* topk_idx,
                        float* topk_prob, int32_t* counts, int32_t* offsets, int32_t* perm,
                        int32_t* inv_perm, void* ws, hipStream_t st, bool sigmoid, const float* sel_bias,
                        float* p_disp, void* sched) {
    const int64_t nblk = (S + kRouteTok - 1) / kRouteTok;
    const int64_t nbp = cnt_row_bytes(nblk);
    uint8_t* blkcnt = (uint8_t*)ws;
    if (S > 0) {
        if (sigmoid)
            launch_topk<true>(logits, sel_bias, S, E, K, topk_idx, topk_prob, blkcnt, nbp, inv_perm, (int)nblk, st);
        else
            launch_topk<false>(logits, nullptr, S, E, K, topk_idx, topk_prob, blkcnt, nbp, inv_perm, (int)nblk, st);
        const hipError_t e1 = launch_check(st);
        if (e1 != hipSuccess) return e1;
    }
    // at least one workgroup, so that counts and offsets are written even
    // for S == 0
    const int bpw = (int)((nblk + kScatMaxWg - 1) / kScatMaxWg > 1 ? (nblk + kScatMaxWg - 1) / kScatMaxWg : 1);
    const int64_t nwg = nblk > 0 ? (nblk + bpw - 1) / bpw : 1;
    const int64_t R = S * K;
    const SchedPart ss = sched ? sched_part(sched, E, R, false) : SchedPart{};
    const SchedPart sl = sched ? sched_part(sched, E, R, true) : SchedPart{};
    // with the tile tables, kSchedWg more workgroups each write a slice of them
    constexpr int kSchedWg = 8;
    const int64_t grid = nwg + (sched ? kSchedWg : 0);
    hipLaunchKernelGGL(route_scatter_kernel, dim3((unsigned)grid), dim3(kScatThreads), 0, st, topk_idx, blkcnt, nblk,
                       nbp, bpw, (int)nwg, counts, offsets, inv_perm, perm, S, K, E, topk_prob, p_disp, ss, sl);
    return launch_check(st);
}

}  // namespace moe
