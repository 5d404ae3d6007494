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
//   router_logits_kernel  TM tokens x RE experts per workgroup (128 x 64 on
//                         eight waves of 32 x 32, or 64 x 64 / 64 x 32 on
//                         waves of 32 x 16 when the larger tile would leave
//                         compute units idle); x and the three planes are
//                         copied global -> LDS by a DMA ring (TM x 128 B + 3
//                         x RE x 128 B per 64-wide d step), every fragment is
//                         one conflict-free ds_read_b128, and every output is
//                         one fixed-order fp32 MFMA chain (lo, mid, hi per
//                         32-wide d step), so results are deterministic.  The
//                         128 x 64 tile re-reads the planes half as often as
//                         the 64-token tiles, and its two waves per SIMD
//                         overlap one wave's fragment reads with the other's
//                         MFMAs (four waves of 64 x 32 left each SIMD a single
//                         wave: 35 -> 31 us with the split at 256 experts x
//                         8192 tokens).
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "tile_dma.h"

namespace moe {


// ---- split: one lane per (expert, 8-wide d chunk) -------------------------
// A wave takes 8 experts x 64 d: lane l handles expert 8 * wave-slot + l / 8
// and d chunk l % 8, so the eight lanes of an expert store its 64 d of each
// plane as one contiguous 128-byte piece, and each of a lane's 8 loads reads
// 8 rows of Wr, 8 consecutive experts (32 bytes) per row.  No LDS, no
// barrier: the launch is a single load-split-store step for D/8 x E lanes.
__global__ __launch_bounds__(256) void router_split_kernel(const float* __restrict__ Wr, int D, int E,
                                                           uint16_t* __restrict__ w3) {
    const int lane = threadIdx.x & 63;
    const int d = blockIdx.x * 64 + (lane & 7) * 8;
    const int e = (blockIdx.y * 4 + (threadIdx.x >> 6)) * 8 + (lane >> 3);
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
// TM tokens x RE experts per workgroup, waves of WM tokens x WN experts.  x
// and the three planes are copied global -> LDS by a kStages-deep DMA ring;
// each wave reads its x fragments once per 32-wide d step and uses them for
// all three planes of its WN / 16 expert fragments.
template <bool KTAIL, int TM, int RE, int WM, int WN>
__global__ __launch_bounds__(TM / WM * (RE / WN) * 64, 1) void router_logits_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ w3, const float* __restrict__ bias, int64_t S,
    int D, int E, float* __restrict__ logits, bool vec_out) {
    constexpr int kWM = TM / WM, kWN = RE / WN, kW = kWM * kWN;   // waves
    constexpr int kMI = WM / 16, kNJ = WN / 16;                   // fragments per wave
    constexpr int kXTile = TM * BK * 2, kWTile = RE * BK * 2;     // one d step of x, of one plane
    constexpr int kStage = kXTile + 3 * kWTile;
    constexpr int kStages = 4 * kStage <= 160 * 1024 ? 4 : 3;
    __shared__ __attribute__((aligned(1024))) char smem[kStages * kStage];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / kWN, wn = wave % kWN;
    const int64_t t0 = (int64_t)blockIdx.x * TM;
    const int e0 = blockIdx.y * RE;
    const int64_t plane = (int64_t)E * D;

    DmaTile<true, TM, BK, kW> dx;
    DmaTile<true, RE, BK, kW> dw[3];
    constexpr int kSX = DmaTile<true, TM, BK, kW>::kSlots, kSW = DmaTile<true, RE, BK, kW>::kSlots;
    dx.init(x, D, t0, S, 0, D, wave, lane);
#pragma unroll
    for (int s = 0; s < 3; ++s) dw[s].init(w3 + s * plane, D, e0, E, 0, D, wave, lane);

    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_char*)smem;
    auto issue = [&](int stage, int64_t rem) {
        const uint32_t b = lds0 + (uint32_t)stage * kStage;
        dx.template issue<KTAIL, 0, kSX>(b, rem, wave);
#pragma unroll
        for (int s = 0; s < 3; ++s) dw[s].template issue<KTAIL, 0, kSW>(b + kXTile + s * kWTile, rem, wave);
    };
    constexpr int kPerStage = kSX + 3 * kSW;   // copies per wave per stage

    uint32_t xb[2], wb[2];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
        xb[kk] = lds0 + row_base(wm * WM, kk, lane);
        wb[kk] = lds0 + kXTile + row_base(wn * WN, kk, lane);
    }

    f32x4 acc[kMI][kNJ];
#pragma unroll
    for (int i = 0; i < kMI; ++i)
#pragma unroll
        for (int j = 0; j < kNJ; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int nk = (D + BK - 1) / BK;

    auto step = [&](auto stage_c, int kt) {
        constexpr int SL = decltype(stage_c)::value;
        // stage kt has landed once at most the later stages' copies are in flight
        if constexpr (kStages >= 4) {
            if (kt + 2 < nk) wait_vmcnt<2 * kPerStage>();
            else if (kt + 1 < nk) wait_vmcnt<kPerStage>();
            else wait_vmcnt<0>();
        } else {
            if (kt + 1 < nk) wait_vmcnt<kPerStage>();
            else wait_vmcnt<0>();
        }
        stage_barrier();
        // every fragment of the stage is read up front, so the LDS latency
        // is paid once per stage rather than before each group of products
        bf16x8 af[2][kMI], wf[2][kNJ][3];
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
            for (int i = 0; i < kMI; ++i) af[kk][i] = lds_b128(xb[kk] + SL * kStage + i * 2048);
#pragma unroll
            for (int j = 0; j < kNJ; ++j)
#pragma unroll
                for (int s = 0; s < 3; ++s)
                    wf[kk][j][s] = lds_b128(wb[kk] + SL * kStage + s * kWTile + j * 2048);
        }
        if (kt + kStages - 1 < nk)
            issue((SL + kStages - 1) % kStages, (int64_t)D - (int64_t)(kt + kStages - 1) * BK);
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
            for (int s = 2; s >= 0; --s)   // lo, mid, hi: smaller terms first
#pragma unroll
                for (int i = 0; i < kMI; ++i)
#pragma unroll
                    for (int j = 0; j < kNJ; ++j)
                        acc[i][j] =
                            __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[kk][j][s], af[kk][i], acc[i][j], 0, 0, 0);
    };

    for (int q = 0; q < kStages - 1 && q < nk; ++q) issue(q, (int64_t)D - (int64_t)q * BK);
    for (int kt = 0; kt < nk; kt += kStages) {
        step(std::integral_constant<int, 0>{}, kt);
        if (kt + 1 < nk) step(std::integral_constant<int, 1>{}, kt + 1);
        if (kt + 2 < nk) step(std::integral_constant<int, 2>{}, kt + 2);
        if constexpr (kStages >= 4)
            if (kt + 3 < nk) step(std::integral_constant<int, 3 % kStages>{}, kt + 3);
    }

    // lane holds logits[t][e .. e+3] of each fragment pair
#pragma unroll
    for (int i = 0; i < kMI; ++i) {
        const int64_t t = t0 + wm * WM + i * 16 + (lane & 15);
        if (t >= S) continue;
#pragma unroll
        for (int j = 0; j < kNJ; ++j) {
            const int e = e0 + wn * WN + j * 16 + 4 * (lane >> 4);
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

size_t router_ws_bytes(int D, int E) { return ((size_t)3 * E * D * 2 + 255) / 256 * 256; }

hipError_t launch_router_logits(const moe_bf16* x, const float* Wr, const float* bias, int64_t S,
                                int D, int E, float* logits, void* ws, hipStream_t st) {
    uint16_t* w3 = (uint16_t*)ws;
    hipLaunchKernelGGL(router_split_kernel, dim3((unsigned)((D + 63) / 64), (unsigned)((E + 31) / 32)),
                       dim3(256), 0, st, Wr, D, E, w3);
    hipError_t err = launch_check(st);
    if (err != hipSuccess || S == 0) return err;
    // 16-byte output stores only where every row start is 16-byte aligned
    const bool vec_out = (E % 4) == 0 && ((uintptr_t)logits % 16) == 0;
    // The tile whose rounds of workgroups over the compute units cost the
    // least (rounds x tile area; ties to the larger tile, which re-reads x
    // and the planes fewer times): 128 x 64, 64 x 64 or 64 x 32.
    const int64_t cus = cu_count();
    auto cost = [&](int tm, int re) {
        const int64_t wgs = (int64_t)grid_for(S, tm) * ((E + re - 1) / re);
        return (wgs + cus - 1) / cus * tm * re;
    };
    const int64_t c_l = cost(128, 64), c_w = cost(64, 64), c_n = cost(64, 32);
    const int cfg = (c_l <= c_w && c_l <= c_n) ? 2 : (c_w <= c_n ? 1 : 0);
#define MOE_ROUTER_LAUNCH(KT, TM, RE, WM, WN)                                                            \
    hipLaunchKernelGGL((router_logits_kernel<KT, TM, RE, WM, WN>),                                       \
                       dim3(grid_for(S, TM), (unsigned)((E + RE - 1) / RE)), dim3(TM / WM * (RE / WN) * 64), \
                       0, st, (const uint16_t*)x, w3, bias, S, D, E, logits, vec_out)
#define MOE_ROUTER_CFG(KT)                                  \
    if (cfg == 2) MOE_ROUTER_LAUNCH(KT, 128, 64, 32, 32);   \
    else if (cfg == 1) MOE_ROUTER_LAUNCH(KT, 64, 64, 32, 16); \
    else MOE_ROUTER_LAUNCH(KT, 64, 32, 32, 16)
    if (D % BK != 0) {
        MOE_ROUTER_CFG(true);
    } else {
        MOE_ROUTER_CFG(false);
    }
#undef MOE_ROUTER_CFG
#undef MOE_ROUTER_LAUNCH
    return launch_check(st);
}

}  // namespace moe
