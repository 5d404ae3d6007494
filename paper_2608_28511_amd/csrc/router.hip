// Router logits on gfx950: logits[t, e] = sum_d x[t, d] * Wr[d, e] + bias[e]
// (the router scores every token against every expert, Section 5.2).
//
// The router weight is fp32 while x is bf16.  Each fp32 weight w is split
// into three bf16 terms, hi = bf16(w), mid = bf16(w - hi), lo = bf16(w - hi -
// mid), whose sum equals w to within 2^-24 |w|.  Products of bf16 values are
// exact in fp32, so three bf16 MFMAs (x*lo + x*mid + x*hi, accumulated in
// fp32) reproduce the fp32 product to fp32 accuracy while running on the
// matrix cores (bf16 splitting as in Henry, Tang and Heinecke, "Leveraging
// the bfloat16 artificial intelligence datatype for higher-precision
// computations", ARITH 2019).
//
// Two launches:
//   router_split_kernel   Wr [D, E] fp32 -> three bf16 planes [3][E][D]
//                         (transposed: each plane is K-contiguous like x);
//   router_logits_kernel  64 tokens x RE experts per workgroup (RE = 64, or
//                         32 when 64-wide tiles would leave compute units
//                         idle), RE / 8 waves of 32 tokens x 16 experts; x
//                         and the three planes are copied global -> LDS by a
//                         4-stage DMA ring (8 KB + 3 x RE x 128 B per 64-wide
//                         d step), every fragment is one conflict-free
//                         ds_read_b128, and every output is one fixed-order
//                         fp32 MFMA chain (lo, mid, hi per 32-wide d step),
//                         so results are deterministic.
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "tile_dma.h"

namespace moe {

constexpr int kRT = 64;                      // tokens per workgroup
constexpr int kRStages = 4;
constexpr int kRTile = 64 * BK * 2;          // the 64-token x tile of one d step: 8 KB

// ---- split: one lane per (expert, 8-wide d chunk) -------------------------
// Lanes of a wave take 64 consecutive experts, so each of the 8 loads is one
// contiguous 256-byte row segment of Wr; each lane then stores its 8 d values
// of every plane as one 16-byte chunk.  No LDS, no barrier: the launch is a
// single load-split-store step for D/8 x E lanes.
__global__ __launch_bounds__(256) void router_split_kernel(const float* __restrict__ Wr, int D, int E,
                                                           uint16_t* __restrict__ w3) {
    const int lane = threadIdx.x & 63;
    const int d = (blockIdx.x * 4 + (threadIdx.x >> 6)) * 8;
    const int e = blockIdx.y * 64 + lane;
    if (e >= E || d >= D) return;            // D is a multiple of 8: chunks are whole
    float w[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) w[q] = Wr[(int64_t)(d + q) * E + e];
    uint32_t hb[4], mb[4], lb[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        uint32_t p[3][2];
#pragma unroll
        for (int v = 0; v < 2; ++v) {
            const float x = w[2 * u + v];
            const uint32_t hi = f32_to_bf16(x);
            const float r1 = x - __uint_as_float(hi << 16);
            const uint32_t mid = f32_to_bf16(r1);
            const uint32_t lo = f32_to_bf16(r1 - __uint_as_float(mid << 16));
            p[0][v] = hi; p[1][v] = mid; p[2][v] = lo;
        }
        hb[u] = p[0][0] | (p[0][1] << 16);
        mb[u] = p[1][0] | (p[1][1] << 16);
        lb[u] = p[2][0] | (p[2][1] << 16);
    }
    const int64_t plane = (int64_t)E * D;
    uint16_t* dst = w3 + (int64_t)e * D + d;
    *(uint4*)dst = make_uint4(hb[0], hb[1], hb[2], hb[3]);
    *(uint4*)(dst + plane) = make_uint4(mb[0], mb[1], mb[2], mb[3]);
    *(uint4*)(dst + 2 * plane) = make_uint4(lb[0], lb[1], lb[2], lb[3]);
}

// ---- logits --------------------------------------------------------------
template <bool KTAIL, int RE>
__global__ __launch_bounds__(RE / 8 * 64, 1) void router_logits_kernel(const uint16_t* __restrict__ x,
                                                                       const uint16_t* __restrict__ w3,
                                                                       const float* __restrict__ bias,
                                                                       int64_t S, int D, int E,
                                                                       float* __restrict__ logits,
                                                                       bool vec_out) {
    constexpr int kW = RE / 8;                     // waves: 2 (tokens) x RE / 16 (experts)
    constexpr int kWTile = RE * BK * 2;            // one plane's RE x 64 tile
    constexpr int kStage = kRTile + 3 * kWTile;    // x, hi, mid, lo
    __shared__ __attribute__((aligned(1024))) char smem[kRStages * kStage];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / (RE / 16), wn = wave % (RE / 16);
    const int64_t t0 = (int64_t)blockIdx.x * kRT;
    const int e0 = blockIdx.y * RE;
    const int64_t plane = (int64_t)E * D;

    DmaTile<true, 64, BK, kW> dx;
    DmaTile<true, RE, BK, kW> dw[3];
    constexpr int kSX = DmaTile<true, 64, BK, kW>::kSlots, kSW = DmaTile<true, RE, BK, kW>::kSlots;
    dx.init(x, D, t0, S, 0, D, wave, lane);
#pragma unroll
    for (int s = 0; s < 3; ++s) dw[s].init(w3 + s * plane, D, e0, E, 0, D, wave, lane);

    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_char*)smem;
    auto issue = [&](int stage, int64_t rem) {
        const uint32_t b = lds0 + (uint32_t)stage * kStage;
        dx.template issue<KTAIL, 0, kSX>(b, rem, wave);
#pragma unroll
        for (int s = 0; s < 3; ++s) dw[s].template issue<KTAIL, 0, kSW>(b + kRTile + s * kWTile, rem, wave);
    };
    constexpr int kPerStage = kSX + 3 * kSW;   // copies per wave per stage

    uint32_t xb[2], wb[2];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
        xb[kk] = lds0 + row_base(wm * 32, kk, lane);
        wb[kk] = lds0 + kRTile + row_base(wn * 16, kk, lane);
    }

    f32x4 acc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
    const int nk = (D + BK - 1) / BK;

    auto step = [&](auto stage_c, int kt) {
        constexpr int S = decltype(stage_c)::value;
        if (kt + 2 < nk) wait_vmcnt<2 * kPerStage>();
        else if (kt + 1 < nk) wait_vmcnt<kPerStage>();
        else wait_vmcnt<0>();
        stage_barrier();
        if (kt + 3 < nk) issue((S + 3) % kRStages, (int64_t)D - (int64_t)(kt + 3) * BK);
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            bf16x8 af[2], wf[3];
#pragma unroll
            for (int i = 0; i < 2; ++i) af[i] = lds_b128(xb[kk] + S * kStage + i * 2048);
#pragma unroll
            for (int s = 0; s < 3; ++s) wf[s] = lds_b128(wb[kk] + S * kStage + s * kWTile);
#pragma unroll
            for (int s = 2; s >= 0; --s)   // lo, mid, hi: smaller terms first
#pragma unroll
                for (int i = 0; i < 2; ++i)
                    acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[s], af[i], acc[i], 0, 0, 0);
        }
    };

    issue(0, D);
    if (nk > 1) issue(1, (int64_t)D - BK);
    if (nk > 2) issue(2, (int64_t)D - 2 * BK);
    for (int kt = 0; kt < nk; kt += kRStages) {
        step(std::integral_constant<int, 0>{}, kt);
        if (kt + 1 < nk) step(std::integral_constant<int, 1>{}, kt + 1);
        if (kt + 2 < nk) step(std::integral_constant<int, 2>{}, kt + 2);
        if (kt + 3 < nk) step(std::integral_constant<int, 3>{}, kt + 3);
    }

    // lane holds logits[t][e .. e+3]
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int64_t t = t0 + wm * 32 + i * 16 + (lane & 15);
        if (t >= S) continue;
        const int e = e0 + wn * 16 + 4 * (lane >> 4);
        float v[4] = {acc[i][0], acc[i][1], acc[i][2], acc[i][3]};
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

size_t router_ws_bytes(int D, int E) { return ((size_t)3 * E * D * 2 + 255) / 256 * 256; }

hipError_t launch_router_logits(const moe_bf16* x, const float* Wr, const float* bias, int64_t S,
                                int D, int E, float* logits, void* ws, hipStream_t st) {
    uint16_t* w3 = (uint16_t*)ws;
    hipLaunchKernelGGL(router_split_kernel, dim3((unsigned)((D / 8 + 3) / 4), (unsigned)((E + 63) / 64)),
                       dim3(256), 0, st, Wr, D, E, w3);
    hipError_t err = launch_check(st);
    if (err != hipSuccess || S == 0) return err;
    // 16-byte output stores only where every row start is 16-byte aligned
    const bool vec_out = (E % 4) == 0 && ((uintptr_t)logits % 16) == 0;
    // 32-expert tiles when 64-wide ones would not give every compute unit a workgroup
    const int64_t wide = (int64_t)grid_for(S, kRT) * ((E + 63) / 64);
    const bool narrow = wide < cu_count();
#define MOE_ROUTER_LAUNCH(KT, RE)                                                                        \
    hipLaunchKernelGGL((router_logits_kernel<KT, RE>), dim3(grid_for(S, kRT), (unsigned)((E + RE - 1) / RE)), \
                       dim3(RE / 8 * 64), 0, st, (const uint16_t*)x, w3, bias, S, D, E, logits, vec_out)
    if (D % BK != 0) {
        if (narrow) MOE_ROUTER_LAUNCH(true, 32); else MOE_ROUTER_LAUNCH(true, 64);
    } else {
        if (narrow) MOE_ROUTER_LAUNCH(false, 32); else MOE_ROUTER_LAUNCH(false, 64);
    }
#undef MOE_ROUTER_LAUNCH
    return launch_check(st);
}

}  // namespace moe
