// Dispatch and combine on gfx950: the local form of the expert-parallel
// hidden dispatch, probability dispatch and hidden combine (Section 4.1
// footnote), whose per-row payloads Eq. 1 counts.
//
// All kernels are HBM-bound row copies.  Dispatch, its MX-FP8 form, the
// combine and its transpose take one workgroup per token, one lane per
// 16-byte chunk of the row (8 bf16).  A
// token's row is read once and written to (dispatch) or gathered from
// (combine) its K rows of the expert-contiguous buffer, each a contiguous
// row.  The combine sums each chunk in fp32 in ascending slot order, so it
// needs no atomics and is deterministic.  Every row that is read once is
// loaded with the non-temporal hint and every store is a plain one: with a
// cold last-level cache (a 512 MB write before each launch) that is the
// fastest or tied-fastest choice on the 64-, 128- and 256-expert layers
// (256-expert dispatch 65.9 -> 60.8 us, combine 105.6 -> 61.1 us).
#include "common.h"
#include "kernels.h"
#include "schedule.h"

namespace moe {

// One workgroup per token, one lane per 16-byte chunk of its row (blocks of
// 64..1024 lanes, looping for rows beyond 16 KB): each chunk is read once and
// written to the token's K routed rows.
// With sched_offsets, one more workgroup (the last) builds the grouped
// GEMM's tile tables from the expert offsets, so the layer needs no launch
// of its own for them.
__global__ __launch_bounds__(1024) void dispatch_kernel(const uint4* __restrict__ x,
                                                        const float* __restrict__ prob,
                                                        const int32_t* __restrict__ inv_perm,
                                                        int64_t S, int D8, int K,
                                                        uint4* __restrict__ x_disp,
                                                        float* __restrict__ p_disp,
                                                        const int32_t* __restrict__ sched_offsets, int E,
                                                        SchedPart sched_small, SchedPart sched_large) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int64_t t = blockIdx.x;
    const int64_t R = S * K;
    if (t >= S) {
        build_tile_schedule(sched_offsets, E, (int)R, sched_small, sched_large);
        return;
    }
    int pos_l = lane < K ? inv_perm[t * K + lane] : 0;
    if ((uint32_t)pos_l >= (uint64_t)R) pos_l = -1;  // out-of-range entries are not written
    if (tid < K && p_disp != nullptr && pos_l >= 0) p_disp[pos_l] = prob[t * K + lane];
    const uint4* src = x + t * D8;
    // the loop bound is wave-uniform, so every lane takes part in the
    // shuffles; only the chunk accesses are masked
    for (int cw = tid - lane; cw < D8; cw += blockDim.x) {
        const int c = cw + lane;
        const bool on = c < D8;
        uint4 v = {};
        if (on) v = ld_nt(src + c);
        for (int k = 0; k < K; ++k) {
            const int64_t pos = __shfl(pos_l, k);
            if (pos < 0 || !on) continue;
            x_disp[pos * D8 + c] = v;
        }
    }
}

// ---- MX-FP8 dispatch payload (the precision lever on b_x, Eq. 1) ----------
// OCP microscaling with FP8 E4M3 elements: per block of 32 elements of a row
// one E8M0 scale byte s + 127, s = floor(log2 max|x|) - 8 clamped to
// [-127, 127] (an all-zero block takes -127), and per element the E4M3 code
// nearest to x * 2^-s (ties to even), saturated to +-448.  A lane's 16-byte
// chunk is 8 elements, so one block is 4 adjacent lanes.

// E4M3 code of a finite fp32 value (round to nearest even, saturating).
__device__ __forceinline__ uint32_t e4m3_rne_sat(float v) {
    const uint32_t u = __float_as_uint(v);
    const uint32_t sign = (u >> 24) & 0x80u;
    const uint32_t a = u & 0x7fffffffu;
    if (a >= 0x43e00000u) return sign | 0x7eu;          // |v| >= 448
    if (a < 0x3c800000u) {                              // |v| < 2^-6: multiples of 2^-9
        const float q = rintf(__uint_as_float(a) * 512.f);  // exact scaling, ties to even
        return sign | (uint32_t)q;                      // 8 -> 0x08, the smallest normal
    }
    // normal: keep 3 mantissa bits of the fp32 value, ties to even
    const uint32_t r = (a + 0x7ffffu + ((a >> 20) & 1u)) & 0xfff00000u;
    const uint32_t e = (r >> 23) - 120u;                // fp32 exponent 121..135 -> E4M3 field 1..15
    return sign | (e << 3) | ((r >> 20) & 7u);
}

// bf16 bits of q * 2^t for an integer q in [0, 15] (exact, or rounded to
// nearest even below bf16's smallest normal), with the given sign bit.
__device__ __forceinline__ uint32_t bf16_of_scaled(uint32_t q, int t, uint32_t sign16) {
    if (q == 0) return sign16;
    const int L = 31 - __builtin_clz(q);                // q in [2^L, 2^(L+1))
    const int E = t + L;                                // exponent of the value
    if (E >= -126) return sign16 | ((uint32_t)(E + 127) << 7) | ((q << (7 - L)) & 0x7fu);
    const int sh = t + 133;                             // value = q * 2^sh * 2^-133
    uint32_t m;
    if (sh >= 0) {
        m = q << sh;
    } else {
        const int n = -sh;
        m = q >> n;
        const uint32_t rem = q & ((1u << n) - 1u), half = 1u << (n - 1);
        if (rem > half || (rem == half && (m & 1u))) ++m;
    }
    return sign16 | m;                                  // m == 128 encodes 2^-126 itself
}

// bf16 bits of one E4M3 code times 2^s.
__device__ __forceinline__ uint32_t e4m3_scaled_to_bf16(uint32_t c, int s) {
    const uint32_t sign16 = (c & 0x80u) << 8;
    const uint32_t e = (c >> 3) & 15u, m = c & 7u;
    return e == 0 ? bf16_of_scaled(m, s - 9, sign16) : bf16_of_scaled(8u | m, (int)e - 10 + s, sign16);
}

__device__ __forceinline__ uint32_t bf16_mag_max8(const uint4& v) {
    uint32_t m = max(max(v.x & 0x7fffu, v.x >> 16 & 0x7fffu), max(v.y & 0x7fffu, v.y >> 16 & 0x7fffu));
    return max(m, max(max(v.z & 0x7fffu, v.z >> 16 & 0x7fffu), max(v.w & 0x7fffu, v.w >> 16 & 0x7fffu)));
}

// One workgroup per token, one lane per 16-byte chunk (8 elements) of its
// row; a 32-element block is 4 adjacent lanes of one wavefront.  The row is
// encoded once and its codes and block scales are written to the token's K
// routed rows.  With sched_offsets, the last workgroup builds the grouped
// GEMM's tile tables (as in dispatch_kernel).
__global__ __launch_bounds__(1024) void dispatch_mx_kernel(const uint4* __restrict__ x,
                                                           const float* __restrict__ prob,
                                                           const int32_t* __restrict__ inv_perm,
                                                           int64_t S, int D8, int K,
                                                           uint2* __restrict__ x_q,
                                                           uint8_t* __restrict__ x_scale,
                                                           float* __restrict__ p_disp,
                                                           const int32_t* __restrict__ sched_offsets, int E,
                                                           SchedPart sched_small, SchedPart sched_large) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int64_t t = blockIdx.x;
    const int64_t R = S * K;
    if (t >= S) {
        build_tile_schedule(sched_offsets, E, (int)R, sched_small, sched_large);
        return;
    }
    const int D32 = D8 / 4;
    int pos_l = lane < K ? inv_perm[t * K + lane] : 0;
    if ((uint32_t)pos_l >= (uint64_t)R) pos_l = -1;  // out-of-range entries are not written
    if (tid < K && p_disp != nullptr && pos_l >= 0) p_disp[pos_l] = prob[t * K + lane];
    const uint4* src = x + t * D8;
    // the loop bound is wave-uniform, so every lane takes part in the
    // shuffles; only the chunk accesses are masked (D8 is a multiple of 4:
    // whole blocks per lane group)
    for (int cw = tid - lane; cw < D8; cw += blockDim.x) {
        const int c = cw + lane;
        const bool on = c < D8;
        const uint4 v = on ? ld_nt(src + c) : make_uint4(0, 0, 0, 0);
        uint32_t am = bf16_mag_max8(v);
        am = max(am, (uint32_t)__shfl_xor((int)am, 1));
        am = max(am, (uint32_t)__shfl_xor((int)am, 2));
        const int ef = (int)(am >> 7);            // bf16 exponent field of the block maximum
        const int sh = ef == 0 ? -127 : max(ef - 127 - 8, -127);
        const uint32_t sc = (uint32_t)(sh + 127);
        const float inv = __uint_as_float((uint32_t)(127 - sh) << 23);  // 2^-s, a normal fp32
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
        uint32_t b[2] = {0u, 0u};
#pragma unroll
        for (int h = 0; h < 4; ++h) {
            const uint32_t lo = e4m3_rne_sat(bf16_lo(w[h]) * inv);
            const uint32_t hi = e4m3_rne_sat(bf16_hi(w[h]) * inv);
            b[h >> 1] |= (lo | (hi << 8)) << (16 * (h & 1));
        }
        const uint2 q = make_uint2(b[0], b[1]);
        for (int k = 0; k < K; ++k) {
            const int64_t pos = __shfl(pos_l, k);
            if (pos < 0 || !on) continue;
            x_q[pos * D8 + c] = q;
            if ((lane & 3) == 0) x_scale[pos * D32 + c / 4] = (uint8_t)sc;
        }
    }
}

// out[r, :] = bf16 of the decoded MX-FP8 row (exact: 4 significant bits
// times a power of two), one thread per 8 elements.
__global__ __launch_bounds__(256) void dequant_mx_kernel(const uint2* __restrict__ x_q,
                                                         const uint8_t* __restrict__ x_scale, int64_t n8,
                                                         uint4* __restrict__ out) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n8) return;
    const uint2 q = x_q[i];
    const int s = (int)x_scale[i / 4] - 127;
    const uint32_t b[2] = {q.x, q.y};
    uint32_t o[4];
#pragma unroll
    for (int h = 0; h < 4; ++h) {
        const uint32_t w = b[h >> 1] >> (16 * (h & 1));
        o[h] = e4m3_scaled_to_bf16(w & 0xffu, s) | (e4m3_scaled_to_bf16((w >> 8) & 0xffu, s) << 16);
    }
    out[i] = make_uint4(o[0], o[1], o[2], o[3]);
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

// y[t] = bf16(sum_k w_k * y_disp[pos_k]); w_k = p_disp[pos_k] or 1.  One
// workgroup per token, one lane per 16-byte chunk; the loads of four slots
// are issued before their products, which are added in slot order.
__global__ __launch_bounds__(1024) void combine_kernel(const uint4* __restrict__ y_disp,
                                                       const float* __restrict__ p_disp,
                                                       const int32_t* __restrict__ inv_perm,
                                                       int64_t S, int D8, int K,
                                                       const float4* __restrict__ add,
                                                       uint4* __restrict__ y) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int64_t t = blockIdx.x;
    const int64_t R = S * K;
    int pos_l = lane < K ? inv_perm[t * K + lane] : 0;
    if ((uint32_t)pos_l >= (uint64_t)R) pos_l = -1;  // out-of-range entries contribute nothing
    const float w_l = (lane < K && pos_l >= 0) ? (p_disp != nullptr ? p_disp[pos_l] : 1.f) : 0.f;
    // the loop bound is wave-uniform, so every lane takes part in the
    // shuffles; only the chunk accesses are masked
    for (int cw = tid - lane; cw < D8; cw += blockDim.x) {
        const int c = cw + lane;
        const bool on = c < D8;
        float acc[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) acc[q] = 0.f;
        for (int k0 = 0; k0 < K; k0 += 8) {   // up to 8 rows' loads in flight before their products
            uint4 v[8];
            float w[8];
            bool ok[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int k = k0 + u;
                const int64_t pos = __shfl(pos_l, k < K ? k : 0);
                w[u] = __shfl(w_l, k < K ? k : 0);
                ok[u] = k < K && pos >= 0 && on;
                if (ok[u]) v[u] = ld_nt(y_disp + pos * D8 + c);
            }
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (ok[u]) fma8(acc, w[u], v[u]);
        }
        if (!on) continue;
        if (add != nullptr) {  // fp32 addend, summed after the K rows, before the rounding
            const float4 a0 = add[(t * D8 + c) * 2], a1 = add[(t * D8 + c) * 2 + 1];
            acc[0] += a0.x; acc[1] += a0.y; acc[2] += a0.z; acc[3] += a0.w;
            acc[4] += a1.x; acc[5] += a1.y; acc[6] += a1.z; acc[7] += a1.w;
        }
        y[t * D8 + c] = pack8(acc);
    }
}

// dy_disp[pos_k] = bf16(w_k * dy[t]);  dp[t,k] = <dy[t], y_disp[pos_k]>.
// One workgroup per token, one lane per 16-byte chunk; each dot is summed in
// a fixed order: a lane's chunks in order, a wave butterfly, then the waves'
// partials in wave order.
constexpr int kCbMaxWaves = 16;
__global__ __launch_bounds__(1024) void combine_bwd_kernel(
    const uint4* __restrict__ dy, const uint4* __restrict__ y_disp, const float* __restrict__ p_disp,
    const int32_t* __restrict__ inv_perm, int64_t S, int D8, int K, uint4* __restrict__ dy_disp,
    float* __restrict__ dp) {
    __shared__ float part[32][kCbMaxWaves];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t t = blockIdx.x;
    const int64_t R = S * K;
    int pos_l = lane < K ? inv_perm[t * K + lane] : 0;
    if ((uint32_t)pos_l >= (uint64_t)R) pos_l = -1;  // out-of-range entries are skipped
    const float w_l = (lane < K && pos_l >= 0) ? (p_disp != nullptr ? p_disp[pos_l] : 1.f) : 0.f;
    const uint4* g = dy + t * D8;
    float dot[32];
#pragma unroll
    for (int k = 0; k < 32; ++k) dot[k] = 0.f;
    // the loop bound is wave-uniform, so every lane takes part in the
    // shuffles; only the chunk accesses are masked
    for (int cw = tid - lane; cw < D8; cw += blockDim.x) {
        const int c = cw + lane;
        const bool on = c < D8;
        float a[8];
        {
            const uint4 gv = on ? ld_nt(g + c) : make_uint4(0, 0, 0, 0);
            a[0] = bf16_lo(gv.x); a[1] = bf16_hi(gv.x);
            a[2] = bf16_lo(gv.y); a[3] = bf16_hi(gv.y);
            a[4] = bf16_lo(gv.z); a[5] = bf16_hi(gv.z);
            a[6] = bf16_lo(gv.w); a[7] = bf16_hi(gv.w);
        }
#pragma unroll
        for (int k = 0; k < 32; ++k) {
            if (k >= K) break;
            const int64_t pos = __shfl(pos_l, k);
            const float w = __shfl(w_l, k);
            if (pos < 0 || !on) continue;
            const uint4 yv = ld_nt(y_disp + pos * D8 + c);
            float b[8];
            b[0] = bf16_lo(yv.x); b[1] = bf16_hi(yv.x);
            b[2] = bf16_lo(yv.y); b[3] = bf16_hi(yv.y);
            b[4] = bf16_lo(yv.z); b[5] = bf16_hi(yv.z);
            b[6] = bf16_lo(yv.w); b[7] = bf16_hi(yv.w);
            float o[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                dot[k] = fmaf(a[q], b[q], dot[k]);
                o[q] = a[q] * w;
            }
            dy_disp[pos * D8 + c] = pack8(o);
        }
    }
    if (dp == nullptr) return;
#pragma unroll
    for (int k = 0; k < 32; ++k) {
        if (k >= K) break;
        float v = dot[k];
#pragma unroll
        for (int m = 32; m > 0; m >>= 1) v += __shfl_xor(v, m);
        if (lane == 0) part[k][wave] = v;
    }
    __syncthreads();
    const int nw = blockDim.x >> 6;
    if (tid < K) {
        float v = 0.f;
        for (int q = 0; q < nw; ++q) v += part[tid][q];
        dp[t * K + tid] = v;
    }
}

hipError_t launch_dispatch(const moe_bf16* x, const float* prob, const int32_t* inv_perm, int64_t S,
                           int D, int K, moe_bf16* x_disp, float* p_disp, hipStream_t st,
                           const int32_t* sched_offsets, int E, void* sched) {
    if (S == 0) return hipSuccess;
    const int d8 = D / 8;
    const int nthr = d8 >= 1024 ? 1024 : (d8 + 63) / 64 * 64;
    const int64_t R = S * K;
    const SchedPart ss = sched ? sched_part(sched, E, R, false) : SchedPart{};
    const SchedPart sl = sched ? sched_part(sched, E, R, true) : SchedPart{};
    const unsigned grid = (unsigned)S + (sched ? 1u : 0u);
    hipLaunchKernelGGL(dispatch_kernel, dim3(grid), dim3(nthr), 0, st, (const uint4*)x, prob, inv_perm, S, d8, K,
                       (uint4*)x_disp, p_disp, sched_offsets, E, ss, sl);
    return launch_check(st);
}

hipError_t launch_combine(const moe_bf16* y_disp, const float* p_disp, const int32_t* inv_perm,
                          int64_t S, int D, int K, const float* add, moe_bf16* y, hipStream_t st) {
    if (S == 0) return hipSuccess;
    const int d8 = D / 8;
    hipLaunchKernelGGL(combine_kernel, dim3((unsigned)S), dim3(d8 >= 1024 ? 1024 : (d8 + 63) / 64 * 64), 0, st,
                       (const uint4*)y_disp, p_disp, inv_perm, S, d8, K, (const float4*)add, (uint4*)y);
    return launch_check(st);
}

hipError_t launch_combine_bwd(const moe_bf16* dy, const moe_bf16* y_disp, const float* p_disp,
                              const int32_t* inv_perm, int64_t S, int D, int K, moe_bf16* dy_disp,
                              float* dp, hipStream_t st) {
    if (S == 0) return hipSuccess;
    const int d8 = D / 8;
    hipLaunchKernelGGL(combine_bwd_kernel, dim3((unsigned)S), dim3(d8 >= 1024 ? 1024 : (d8 + 63) / 64 * 64), 0, st,
                       (const uint4*)dy, (const uint4*)y_disp, p_disp, inv_perm, S, D / 8, K,
                       (uint4*)dy_disp, dp);
    return launch_check(st);
}

}  // namespace moe

namespace moe {

hipError_t launch_dispatch_mx(const moe_bf16* x, const float* prob, const int32_t* inv_perm, int64_t S, int D,
                              int K, uint8_t* x_q, uint8_t* x_scale, float* p_disp, hipStream_t st,
                              const int32_t* sched_offsets, int E, void* sched) {
    if (S == 0) return hipSuccess;
    const int d8 = D / 8;
    const int64_t R = S * K;
    const SchedPart ss = sched ? sched_part(sched, E, R, false) : SchedPart{};
    const SchedPart sl = sched ? sched_part(sched, E, R, true) : SchedPart{};
    const unsigned grid = (unsigned)S + (sched ? 1u : 0u);
    hipLaunchKernelGGL(dispatch_mx_kernel, dim3(grid), dim3(d8 >= 1024 ? 1024 : (d8 + 63) / 64 * 64), 0, st,
                       (const uint4*)x, prob, inv_perm, S, d8, K, (uint2*)x_q, x_scale, p_disp, sched_offsets, E,
                       ss, sl);
    return launch_check(st);
}

hipError_t launch_dequant_mx(const uint8_t* x_q, const uint8_t* x_scale, int64_t R, int D, moe_bf16* out,
                             hipStream_t st) {
    const int64_t n8 = R * (D / 8);
    if (n8 == 0) return hipSuccess;
    hipLaunchKernelGGL(dequant_mx_kernel, dim3(grid_for(n8, 256)), dim3(256), 0, st, (const uint2*)x_q, x_scale, n8,
                       (uint4*)out);
    return launch_check(st);
}

}  // namespace moe
