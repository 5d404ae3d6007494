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
//   colsum kernels        dbias: fixed-order column sums in two passes;
//   router_dx_kernel      one wavefront per token: the K nonzero terms of
//                         ds Wr^T in fp32 from a transposed copy of Wr.
// Every reduction has a fixed order, so results are deterministic.
//
// The production router (sigmoid scores s = sigmoid(logit), weights
// g_k = s[T_k] / sum_j s[T_j], Section 5.2) differs only in the first step:
//   router_ds_sigmoid_kernel   d logit = s (1 - s) (d s), with, on the picked
//                              experts, d s[T_k] = (dg_k - sum_j g_j dg_j) / Z,
//                              Z = sum_j s[T_j]; with the sequence balance
//                              loss, every expert also gets
//                              d s_e += (a_e - sum_e' a_e' s_e' / sum s) / sum s,
//                              a_e = coef * count[seq, e].
// The balance term makes ds dense, so dx_r = ds Wr^T becomes an MFMA product
// over E: six bf16 plane products (hi, mid, lo of ds against hi, mid, lo of
// Wr, dropping the three below 2^-24 relative) in one rows-GEMM launch.
#include "common.h"
#include "kernels.h"

namespace moe {

constexpr int kRbTok = 4;  // tokens (wavefronts) per 256-thread block

__device__ __forceinline__ float sigmoid_score(float l) { return 1.f / (1.f + expf(-l)); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int msk = 32; msk > 0; msk >>= 1) v += __shfl_xor(v, msk);
    return v;  // the xor butterfly leaves the same bits in every lane
}

// hi + mid + lo == w within 2^-24 |w| (three successive bf16 roundings).
__device__ __forceinline__ void split3(float w, uint32_t& hi, uint32_t& mid, uint32_t& lo) {
    hi = f32_to_bf16(w);
    const float r1 = w - __uint_as_float(hi << 16);
    mid = f32_to_bf16(r1);
    lo = f32_to_bf16(r1 - __uint_as_float(mid << 16));
}

// Row t of ds (fp32, E wide), of ds3 (planes hi | mid | lo, each Ep wide) and,
// when ds6 is not null, of ds6 (planes hi hi hi mid mid lo, matching the
// weight planes Wh Wm Wl Wh Wm Wh of wr_split6_kernel).
template <int EPL>
__device__ __forceinline__ void store_ds_row(const float (&v)[EPL], int64_t t, int E, int Ep, int lane,
                                             float* __restrict__ ds, uint16_t* __restrict__ ds3,
                                             uint16_t* __restrict__ ds6) {
    const int64_t E3 = 3 * (int64_t)Ep, E6 = 6 * (int64_t)Ep;
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
        const int e = lane + 64 * i;
        if (e >= Ep) break;
        const float w = e < E ? v[i] : 0.f;
        if (e < E) ds[t * E + e] = w;
        uint32_t hi, mid, lo;
        split3(w, hi, mid, lo);
        ds3[t * E3 + e] = (uint16_t)hi;
        ds3[t * E3 + Ep + e] = (uint16_t)mid;
        ds3[t * E3 + 2 * Ep + e] = (uint16_t)lo;
        if (ds6 != nullptr) {
            uint16_t* r = ds6 + t * E6 + e;
            r[0] = (uint16_t)hi; r[Ep] = (uint16_t)hi; r[2 * Ep] = (uint16_t)hi;
            r[3 * Ep] = (uint16_t)mid; r[4 * Ep] = (uint16_t)mid; r[5 * Ep] = (uint16_t)lo;
        }
    }
}

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
    store_ds_row<EPL>(v, t, E, Ep, lane, ds, ds3, nullptr);
}

// Sigmoid router: one wavefront per token.  seq_counts (per sequence of T
// tokens and expert, from the balance-loss forward) null = no balance loss.
template <int EPL>
__global__ __launch_bounds__(256) void router_ds_sigmoid_kernel(
    const float* __restrict__ logits, const int32_t* __restrict__ topk_idx, const float* __restrict__ topk_gate,
    const float* __restrict__ dg, const int32_t* __restrict__ seq_counts, int64_t S, int E, int Ep, int K,
    int64_t T, float coef, float* __restrict__ ds, uint16_t* __restrict__ ds3, uint16_t* __restrict__ ds6) {
    const int lane = threadIdx.x & 63;
    const int64_t t = (int64_t)blockIdx.x * kRbTok + (threadIdx.x >> 6);
    if (t >= S) return;
    int e_l = -1;
    float g_l = 0.f, dg_l = 0.f, s_l = 0.f;
    if (lane < K) {
        e_l = topk_idx[t * K + lane];
        if (e_l < 0 || e_l >= E) e_l = -1;  // malformed index: no contribution
        g_l = topk_gate[t * K + lane];
        dg_l = dg[t * K + lane];
        s_l = e_l >= 0 ? sigmoid_score(logits[t * E + e_l]) : 0.f;
    }
    const float m = wave_sum(g_l * dg_l);
    const float Z = wave_sum(s_l);
    const float dsel_l = lane < K ? (dg_l - m) / Z : 0.f;
    float sg[EPL], v[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
        const int e = lane + 64 * i;
        sg[i] = e < E ? sigmoid_score(logits[t * E + e]) : 0.f;
        v[i] = 0.f;
    }
    for (int k = 0; k < K; ++k) {
        const int ek = __shfl(e_l, k);
        const float dk = __shfl(dsel_l, k);
        if (ek < 0) continue;
#pragma unroll
        for (int i = 0; i < EPL; ++i)
            if (lane + 64 * i == ek) v[i] = dk;
    }
    if (seq_counts != nullptr) {
        const int32_t* cnt = seq_counts + (t / T) * E;
        float part = 0.f;
#pragma unroll
        for (int i = 0; i < EPL; ++i) part += sg[i];
        const float tot = wave_sum(part);
        float a[EPL], ap = 0.f;
#pragma unroll
        for (int i = 0; i < EPL; ++i) {
            const int e = lane + 64 * i;
            a[i] = e < E ? coef * (float)cnt[e] : 0.f;
            ap += a[i] * (sg[i] / tot);
        }
        const float A = wave_sum(ap);
#pragma unroll
        for (int i = 0; i < EPL; ++i) v[i] += (a[i] - A) / tot;
    }
#pragma unroll
    for (int i = 0; i < EPL; ++i) v[i] *= sg[i] * (1.f - sg[i]);
    store_ds_row<EPL>(v, t, E, Ep, lane, ds, ds3, ds6);
}

// W6[d][p*Ep + e] = plane p of Wr[d, e], planes (hi, mid, lo, hi, mid, hi);
// columns E .. Ep-1 zero.  K-contiguous rows of 6*Ep, the transposed weight
// of the dx product.
__global__ __launch_bounds__(256) void wr_split6_kernel(const float* __restrict__ Wr, int D, int E, int Ep,
                                                        uint16_t* __restrict__ W6) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)D * Ep) return;
    const int64_t d = i / Ep;
    const int e = (int)(i - d * Ep);
    uint32_t hi, mid, lo;
    split3(e < E ? Wr[d * E + e] : 0.f, hi, mid, lo);
    uint16_t* r = W6 + d * 6 * (int64_t)Ep + e;
    r[0] = (uint16_t)hi; r[Ep] = (uint16_t)mid; r[2 * Ep] = (uint16_t)lo;
    r[3 * Ep] = (uint16_t)hi; r[4 * Ep] = (uint16_t)mid; r[5 * Ep] = (uint16_t)hi;
}

// dbias[e] = sum_t ds[t, e] in two fixed-order passes.  Pass 1: workgroup
// (column block of 64, row chunk) with 4 row lanes per column, each adding
// its rows in order (loads issued 8 at a time so they overlap), then the 4
// lanes in order.  Pass 2: one thread per column adds the chunks in order.
constexpr int kColChunkRows = 256;

static int colsum_chunks(int64_t rows) {
    int64_t n = (rows + kColChunkRows - 1) / kColChunkRows;
    return (int)(n < 1 ? 1 : (n > 64 ? 64 : n));
}

__global__ __launch_bounds__(256) void colsum_partial_kernel(const float* __restrict__ src, int64_t rows, int cols,
                                                             int64_t chunk_rows, float* __restrict__ part) {
    __shared__ float red[4][64];
    const int c = threadIdx.x & 63, q = threadIdx.x >> 6;
    const int col = blockIdx.x * 64 + c;
    const int64_t r0 = (int64_t)blockIdx.y * chunk_rows;
    const int64_t r1 = (r0 + chunk_rows) < rows ? (r0 + chunk_rows) : rows;
    float s = 0.f;
    if (col < cols) {
        int64_t r = r0 + q;
        for (; r + 28 < r1; r += 32) {
            float v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = src[(r + 4 * u) * cols + col];
#pragma unroll
            for (int u = 0; u < 8; ++u) s += v[u];
        }
        for (; r < r1; r += 4) s += src[r * cols + col];
    }
    red[q][c] = s;
    __syncthreads();
    if (q == 0 && col < cols)
        part[(int64_t)blockIdx.y * cols + col] = ((red[0][c] + red[1][c]) + red[2][c]) + red[3][c];
}

__global__ __launch_bounds__(256) void colsum_final_kernel(const float* __restrict__ part, int nchunk, int cols,
                                                           float* __restrict__ out) {
    const int col = blockIdx.x * 256 + threadIdx.x;
    if (col >= cols) return;
    float s = 0.f;
    int c = 0;
    for (; c + 8 <= nchunk; c += 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = part[(int64_t)(c + u) * cols + col];
#pragma unroll
        for (int u = 0; u < 8; ++u) s += v[u];
    }
    for (; c < nchunk; ++c) s += part[(int64_t)c * cols + col];
    out[col] = s;
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
    // the loop bound is wave-uniform, so every lane takes part in the
    // shuffles of lanes 0 .. K-1; only the column accesses are masked
    for (int cw = 0; cw < D4; cw += 64) {
        const int c = cw + lane;
        const bool on = c < D4;
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int k = 0; k < K; ++k) {
            const int ek = __shfl(e_l, k);
            const float w = __shfl(w_l, k);
            if (ek < 0 || !on) continue;
            const float4 r = WrT[(int64_t)ek * D4 + c];
            acc.x += w * r.x; acc.y += w * r.y; acc.z += w * r.z; acc.w += w * r.w;
        }
        if (on) dx[t * D4 + c] = acc;
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
    return launch_check(st);
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
    float* ds; uint16_t* ds3; float* WrT; float* part; float* colpart; uint16_t* ds6; uint16_t* W6; size_t bytes;
    int nchunk;
};

static int pad8(int e) { return (e + 7) / 8 * 8; }

// dense: room for the six-plane dx product of the sigmoid router with the
// balance loss (ds6 [S, 6 Ep], W6 [D, 6 Ep] bf16).
static RouterBwdWs router_bwd_layout(char* base, int64_t S, int D, int E, bool dense) {
    RouterBwdWs w{};
    size_t off = 0;
    auto take = [&](size_t bytes) { void* p = base ? base + off : nullptr; off += (bytes + 255) / 256 * 256; return p; };
    const int Ep = pad8(E);
    w.nchunk = wgrad_chunks(S, D, 3 * Ep);
    w.ds = (float*)take((size_t)S * E * 4);
    w.ds3 = (uint16_t*)take((size_t)S * 3 * Ep * 2);
    w.WrT = (float*)take((size_t)E * D * 4);
    w.part = (float*)take((size_t)w.nchunk * D * 3 * Ep * 4);
    w.colpart = (float*)take((size_t)colsum_chunks(S) * E * 4);
    if (dense) {
        w.ds6 = (uint16_t*)take((size_t)S * 6 * Ep * 2);
        w.W6 = (uint16_t*)take((size_t)D * 6 * Ep * 2);
    }
    w.bytes = off;
    return w;
}

size_t router_bwd_ws_bytes(int64_t S, int D, int E, bool dense) {
    return router_bwd_layout(nullptr, S, D, E, dense).bytes;
}

// dWr, dbias and dx_r from ds (and its planes) already in the workspace.
static hipError_t router_linear_bwd(const moe_bf16* x_r, const float* Wr, const int32_t* topk_idx,
                                    const float* ds, const RouterBwdWs& w, int64_t S, int D, int E, int K,
                                    float* dWr, float* dbias, float* dx_r, hipStream_t st);

hipError_t launch_router_bwd_sigmoid(const moe_bf16* x_r, const float* Wr, const float* logits,
                                     const int32_t* topk_idx, const float* topk_gate, const float* dg,
                                     const int32_t* seq_counts, int64_t seq_len, float coef, int64_t S, int D,
                                     int E, int K, float* dlogits, float* dWr, float* dbias, float* dx_r,
                                     void* ws, hipStream_t st) {
    const bool dense = seq_counts != nullptr;
    RouterBwdWs w = router_bwd_layout((char*)ws, S, D, E, dense);
    float* ds = dlogits != nullptr ? dlogits : w.ds;
    const int Ep = pad8(E);
    uint16_t* ds6 = dense && dx_r != nullptr ? w.ds6 : nullptr;
    if (S > 0) {
        const int epl = (Ep + 63) / 64;
#define MOE_DS_CASE(N)                                                                                       \
    hipLaunchKernelGGL(router_ds_sigmoid_kernel<N>, dim3(grid_for(S, kRbTok)), dim3(256), 0, st, logits,       \
                       topk_idx, topk_gate, dg, seq_counts, S, E, Ep, K, seq_len, coef, ds, w.ds3, ds6)
        if (epl <= 1) MOE_DS_CASE(1);
        else if (epl <= 2) MOE_DS_CASE(2);
        else if (epl <= 4) MOE_DS_CASE(4);
        else if (epl <= 8) MOE_DS_CASE(8);
        else MOE_DS_CASE(16);
#undef MOE_DS_CASE
        hipError_t err = launch_check(st);
        if (err != hipSuccess) return err;
    }
    if (!dense) return router_linear_bwd(x_r, Wr, topk_idx, ds, w, S, D, E, K, dWr, dbias, dx_r, st);
    hipError_t err = router_linear_bwd(x_r, Wr, topk_idx, ds, w, S, D, E, K, dWr, dbias, nullptr, st);
    if (err != hipSuccess || dx_r == nullptr || S == 0) return err;
    // dense dx_r [S, D] = ds6 [S, 6 Ep] . W6 [D, 6 Ep]^T, fp32 out
    hipLaunchKernelGGL(wr_split6_kernel, dim3(grid_for((int64_t)D * Ep, 256)), dim3(256), 0, st, Wr, D, E, Ep,
                       w.W6);
    if ((err = launch_check(st)) != hipSuccess) return err;
    return launch_grouped_rows((const moe_bf16*)ds6, 6 * (int64_t)Ep, (const moe_bf16*)w.W6, 6 * (int64_t)Ep, 0,
                               true, dx_r, D, EPI_F32, nullptr, nullptr, nullptr, 1, S, D, 6 * Ep, st);
}

hipError_t launch_router_bwd(const moe_bf16* x_r, const float* Wr, const int32_t* topk_idx, const float* topk_prob,
                             const float* dp, int64_t S, int D, int E, int K, float* dlogits, float* dWr,
                             float* dbias, float* dx_r, void* ws, hipStream_t st) {
    RouterBwdWs w = router_bwd_layout((char*)ws, S, D, E, false);
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
        if ((err = launch_check(st)) != hipSuccess) return err;
    }
    return router_linear_bwd(x_r, Wr, topk_idx, ds, w, S, D, E, K, dWr, dbias, dx_r, st);
}

static hipError_t router_linear_bwd(const moe_bf16* x_r, const float* Wr, const int32_t* topk_idx,
                                    const float* ds, const RouterBwdWs& w, int64_t S, int D, int E, int K,
                                    float* dWr, float* dbias, float* dx_r, hipStream_t st) {
    const int Ep = pad8(E);
    hipError_t err;
    // dWr [D, E] = x_r^T [hi | mid | lo](ds), fp32 partials per row chunk
    const int64_t kchunk = S > 0 ? (S + w.nchunk - 1) / w.nchunk : 1;
    if ((err = launch_chunked_wgrad(x_r, D, (const moe_bf16*)w.ds3, 3 * (int64_t)Ep, w.part, 3 * (int64_t)Ep,
                                    (int64_t)D * 3 * Ep, w.nchunk, kchunk, D, 3 * Ep, S, st)) != hipSuccess)
        return err;
    // (an empty row range contributes zero partials: the k-grouped kernel writes its zero accumulators)
    if ((err = launch_sum_planes(w.part, w.nchunk, D, E, 3, Ep, dWr, st)) != hipSuccess) return err;
    if (dbias != nullptr) {
        const int nch = colsum_chunks(S);
        const int64_t chunk_rows = (S + nch - 1) / nch;
        hipLaunchKernelGGL(colsum_partial_kernel, dim3((unsigned)((E + 63) / 64), (unsigned)nch), dim3(256), 0, st,
                           ds, S, E, chunk_rows > 0 ? chunk_rows : 1, w.colpart);
        if ((err = launch_check(st)) != hipSuccess) return err;
        hipLaunchKernelGGL(colsum_final_kernel, dim3((unsigned)((E + 255) / 256)), dim3(256), 0, st, w.colpart,
                           nch, E, dbias);
        if ((err = launch_check(st)) != hipSuccess) return err;
    }
    if (dx_r != nullptr && S > 0) {
        hipLaunchKernelGGL(transpose_f32_kernel, dim3((unsigned)((E + 31) / 32), (unsigned)((D + 31) / 32)),
                           dim3(256), 0, st, Wr, D, E, w.WrT);
        if ((err = launch_check(st)) != hipSuccess) return err;
        hipLaunchKernelGGL(router_dx_kernel, dim3(grid_for(S, kRbTok)), dim3(256), 0, st, ds, topk_idx,
                           (const float4*)w.WrT, S, D / 4, E, K, (float4*)dx_r);
        if ((err = launch_check(st)) != hipSuccess) return err;
    }
    return hipSuccess;
}

}  // namespace moe
