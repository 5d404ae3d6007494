// Grouped bf16 GEMM on gfx950 MFMA for the routed experts (grouped GEMM over
// expert segments, Section 5.2), their backward, and the dense latent
// projections.
//
// One kernel template covers every product of the layer:
//
//   ROWS mode   C[r, n] = sum_k A[r, k] * B_e[k, n] for the rows r of expert
//               e's segment [offsets[e], offsets[e+1]) (forward up/down and
//               the two dgrads), or for all M rows when offsets is NULL
//               (dense latent projections).
//   KGRP mode   C_e[m, n] = sum_{r in segment e} A[r, m] * B[r, n]  (wgrad:
//               the contraction runs over the expert's ragged rows).
//
// Two block tiles, chosen per launch (Tile below), on 512 threads: 8
// wavefronts in a 2 x 4 grid, each (BM/2) x 64 outputs (v_mfma_f32_16x16x32_bf16):
//   128 x 256, 64 k per stage, 3-stage ring of 48 KB stages;
//   256 x 256, 32 k per stage, 4-stage ring of 32 KB stages -- one third
//   fewer operand bytes per product, for launches long enough that the
//   coarser tile count does not leave the last round of CUs half idle.
// Neither the MFMAs nor copy bandwidth bound the kernel: the per-CU
// texture-data return path reads 82% busy at 0.42 of the MFMA rate while a
// plain stream of the same copies reaches ~4x these bytes per clock, so the
// waits are on copy latency (a quarter of the operand reads miss L2); the
// 256-row tile moves a third less per flop.  One workgroup fills a CU's LDS,
// so each SIMD runs two wavefronts: one wave's address arithmetic, barrier
// and LDS latency overlap the other's MFMAs.
//
// Operands never pass through registers on their way to LDS: every 16-byte
// chunk is copied by a buffer load with an LDS destination into the LDS
// ring, all but one stage in flight while one is consumed.  Each operand
// keeps the layout it has in HBM:
//   K-contiguous source  -> LDS rows of 64 or 32 k (XOR-swizzled by row),
//                           MFMA fragments read with ds_read_b128;
//   M/N-contiguous source (weights stored [D, F] / [F, D], both wgrad
//                           operands) -> LDS k-rows of BM or BN elements
//                           (chunk pairs XOR-swizzled by k), fragments read
//                           with two ds_read_b64_tr_b16, the gfx950 LDS
//                           transpose read, so no VALU transposition at all.
// A DMA lane's LDS destination is fixed by its lane id, so the swizzles are
// applied by permuting which global chunk each lane fetches.  Lanes whose
// chunk lies outside the operand (ragged expert rows, k / n tails) fetch a
// zero chunk instead, so partial tiles need no special path.
//
// The MFMA takes the weight-side fragment as its first operand, so each
// lane's four accumulators hold four consecutive output columns of one row.
//
// ROWS mode runs persistently: one workgroup per CU walks its share of the
// output tiles, and the DMA ring runs over the flattened sequence of (tile,
// k step) pairs, so the first two k steps of a workgroup's next tile are
// already loading while it finishes the current one.  Output tiles are
// written through a 16 KB LDS slice (16 x 64 bf16 per wave) so that every
// store is 16 contiguous bytes and one store instruction covers 8 whole
// 128-byte rows; stores go through a range-checked buffer descriptor, so
// rows past the tile's end and columns past N are dropped by the hardware.
// Squared-ReLU (up projection) is fused there, and so is the dgrad's
// product with the activation derivative, whose saved pre-activation each
// lane loads at its accumulators' positions.
//
// The up projection can also read its A operand as the MX-FP8 dispatch
// payload (gemm_rows_mx_kernel): codes and block scales travel through the
// same ring and each lane decodes its fragment right before the MFMA, with a
// result identical to decoding first (see MxDma and mx_frag).
//
// KGRP mode (weight gradients) runs one workgroup per (expert, m-tile,
// n-tile) item, two m-tiles at a time across all n-tiles so that the items
// an XCD runs together keep their operand rows in its L2, and writes its fp32
// tile through LDS as whole 256-byte row pieces with non-temporal stores.
//
// Expert segments are located through device-side tile tables (expert,
// first row, end row of every 128-row and every 256-row tile, built from the
// routing offsets on the device): no host reads the routing counts.  Work item w of the
// grid-wide order is tile (m, n) of an ordering that takes 8 m-tiles at a
// time across all n-tiles, and the items a round of workgroups processes
// together on one XCD are consecutive, so they share A rows and expert
// weights in that XCD's L2.
#include <mutex>
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "schedule.h"
#include "tile_dma.h"

namespace moe {

constexpr int BN = 256;
constexpr int kGemmThreads = kWaves * 64;
constexpr int kEpiWaveBytes = 16 * 64 * 2;      // 16 x 64 bf16 staging block per wave
constexpr int kEpiBytes = kWaves * kEpiWaveBytes;  // 16 KB
constexpr int kGroupM = 8;

// Block tile BM x BN with KD contraction elements per ring stage and a ring
// of STAGES stages.  AMX: A is MX-FP8 (codes, one byte per element, and the
// stage's block scales; see MxDma) instead of bf16.
template <int BM_, int KD_, int STAGES_, bool AMX_ = false>
struct Tile {
    static constexpr int BM = BM_, KD = KD_, kStages = STAGES_;
    static constexpr bool kAmx = AMX_;
    static constexpr int MI = BM / 32;          // A fragments (16 rows) per wave: waves cover BM/2 rows
    static constexpr int kKK = KD / 32;         // MFMA k steps per stage
    static constexpr int kCodeBytes = BM * KD;  // AMX: the stage's codes, then its scale words
    static constexpr int kSclBytes = AMX_ ? kWaves * 64 * 4 : 0;
    static constexpr int kABytes = AMX_ ? kCodeBytes + kSclBytes : BM * KD * 2;
    static constexpr int kBBytes = BN * KD * 2;
    static constexpr int kStageBytes = kABytes + kBBytes;
    static constexpr int kRingBytes = kStages * kStageBytes;
    static constexpr int kFrag = 16 * KD * 2;   // bytes between 16-row fragments of the row layout
    static constexpr int kFragA = AMX_ ? 16 * KD : kFrag;
};
using TileS = Tile<128, 64, 3>;   // 144 KB ring (+16 KB epilogue staging)
using TileL = Tile<256, 32, 4>;   // 128 KB ring
using TileSX = Tile<128, 64, 3, true>;   // MX-FP8 A: 126 KB ring
using TileLX = Tile<256, 32, 4, true>;   // 104 KB ring
static_assert(TileS::kRingBytes + kEpiBytes <= 160 * 1024 && TileL::kRingBytes + kEpiBytes <= 160 * 1024 &&
                  TileSX::kRingBytes + kEpiBytes <= 160 * 1024 && TileLX::kRingBytes + kEpiBytes <= 160 * 1024,
              "LDS budget");

typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) u32x2 lds_u32x2;
typedef __attribute__((address_space(3))) u32x4 lds_u32x4;
typedef __attribute__((address_space(3))) uint8_t lds_u8;
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// MX-FP8 A operand (codes [R, Kd] uint8, E8M0 scales [R, Kd / 32] uint8):
// per stage each wave copies one 16-byte chunk of codes (rows of KD bytes,
// fp8 row layout) and one scale word.  A row's scale bytes are not 4-byte
// aligned, so every row gets a window of kLPR words starting at the aligned
// word at or below its first block of the stage; the fragment read takes its
// byte at offset (row * nb + kb) & 3 of the window.  The scale descriptor
// spans the whole array rounded up to 4 bytes: rows past R read zero, and
// rows past a tile's end (zero codes) read other rows' finite scales.
template <class T>
struct MxDma {
    static constexpr int kLPR = kWaves * 64 / T::BM;   // scale words per row
    static_assert(kLPR * T::BM == kWaves * 64 && 3 + T::kKK <= 4 * kLPR, "scale window");
    static constexpr int kSlots = 2;                     // copies per wave and stage
    DmaTile<true, T::BM, T::KD / 2, kWaves, 1> codes;    // code pairs as 16-bit elements
    static_assert(decltype(codes)::kSlots == 1, "one code chunk per wave and stage");
    i32x4 srs;       // wave-uniform
    uint32_t srow;   // (row0 + this lane's window row) * nb
    uint32_t sword;  // byte of this lane's word in the window
    uint32_t kb;     // first block of the next stage

    __device__ __forceinline__ void init(const uint8_t* q, const uint8_t* scale, uint32_t scale_bytes,
                                         int64_t row0, int64_t row_hi, int Kd, int wave, int lane) {
        codes.init((const uint16_t*)q, Kd / 2, row0, row_hi, 0, Kd / 2, wave, lane);
        srs = buf_rsrc(scale, scale_bytes);
        const int p = wave * 64 + lane;
        srow = (uint32_t)((row0 + p / kLPR) * (Kd / 32));
        sword = (uint32_t)(4 * (p % kLPR));
        kb = 0;
    }
    template <bool KTAIL, int I0, int I1>
    __device__ __forceinline__ void issue(uint32_t tile_lds, int64_t k_rem, int wave) {
        codes.template issue<KTAIL, 0, 1>(tile_lds, k_rem / 2, wave);
        dma4(srs, ((srow + kb) & ~3u) + sword, tile_lds + T::kCodeBytes + (uint32_t)wave * 256u);
        kb += T::kKK;
    }
};

// bf16 MFMA fragment of 8 MX-FP8 codes sharing one E8M0 scale byte s8:
// code * 2^(s8 - 127).  v_cvt_scalef32_pk_bf16_fp8 takes the scale from the
// exponent field of an fp32 operand; for every finite code at every scale
// byte up to 246 (the largest the encoder emits) its result equals the exact
// decode, bf16 subnormals included (checked exhaustively on gfx950).
__device__ __forceinline__ bf16x8 mx_frag(u32x2 c, uint32_t s8) {
    const float sc = __uint_as_float(s8 << 23);
    const bf16x2 p0 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(c[0], sc, false);
    const bf16x2 p1 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(c[0], sc, true);
    const bf16x2 p2 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(c[1], sc, false);
    const bf16x2 p3 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(c[1], sc, true);
    const u32x4 w = {__builtin_bit_cast(uint32_t, p0), __builtin_bit_cast(uint32_t, p1),
                     __builtin_bit_cast(uint32_t, p2), __builtin_bit_cast(uint32_t, p3)};
    return __builtin_bit_cast(bf16x8, w);
}

struct GemmArgs {
    const uint16_t* A;
    const uint16_t* B;
    void* C;
    const uint16_t* aux_in;   // EPI_DRELU2: pre-activation u, same layout as C
    uint16_t* aux_out;        // EPI_RELU2: pre-activation u (may be null)
    const int32_t* offsets;   // [E+1] expert row segments (KGRP mode)
    const int32_t* order;     // KGRP pair launch: experts by descending row count (the item order)
    const int4* tiles;        // ROWS mode: per 128-row tile {expert, row0, row_end, 0}; null = dense
    const int32_t* mtile_total;  // ROWS mode with tiles: device count of valid 128-row m-tiles
    const int4* tiles_l;      // the same for 256-row tiles
    const int32_t* mtile_total_l;
    const int32_t* a_perm;    // ROWS mode, bf16 A gathered: row r of the product is A row a_perm[r] / a_div
    int a_div;
    int64_t a_src_rows;       // rows of the gathered A
    const uint8_t* A_scale;   // MX-FP8 A: E8M0 scales [R, Kd / 32]
    uint32_t scale_bytes;     // R * Kd / 32 rounded up to a multiple of 4
    int64_t lda, ldb, ldc;
    int64_t b_stride;         // elements between experts' B (ROWS mode)
    int64_t c_stride;         // elements between experts' C (KGRP mode)
    int64_t kchunk;           // KGRP mode without offsets: group e contracts rows [e*kchunk, (e+1)*kchunk)
    int64_t M;                // dense rows (ROWS, no offsets) or output rows (KGRP)
    int64_t R;                // rows of the activation buffers: segments are clamped to [0, R)
    int N, Kd, E;
    int m_tiles, n_tiles;
    int m_tiles_l;            // ROWS mode: m-tiles of 256 rows (dense) or their static bound
    int accumulate;           // EPI_F32: C += product instead of C = product
};

// Wait until stage `cur` of `total` has landed when stages cur + 1 ..
// cur + T::kStages - 2 (those that exist) may still be in flight: copies
// complete in order, so at most that many stages' worth may be outstanding.
template <class T, int kPerStage>
__device__ __forceinline__ void wait_stage(int cur, int total) {
    const int ahead = total - 1 - cur;
    if constexpr (T::kStages >= 4) {
        if (ahead >= 2) { wait_vmcnt<2 * kPerStage>(); return; }
    }
    if constexpr (T::kStages >= 3) {
        if (ahead >= 1) { wait_vmcnt<kPerStage>(); return; }
    }
    wait_vmcnt<0>();
}

// One KD-wide stage of the main loop for stage slot S of the ring: read the
// fragments of each 32-wide k step, send the copies of the stage kStages - 1
// ahead (half of B after the second k step's reads when a stage has two),
// and accumulate.  `next` says whether there is a stage to copy; nrem is the
// contraction length left from its start.
// AMX: sb is the lane's scale byte of the stage's first block in slot 0.
template <class T, bool A_K, bool B_K, bool KTAIL, int S, class DA, class DB, int NA, int NB>
__device__ __forceinline__ void mma_stage(f32x4 (&acc)[T::MI][4], const uint32_t (&abase)[NA],
                                          const uint32_t (&bbase)[2][NB], DA& da, DB& db, bool next,
                                          int64_t nrem, uint32_t ldsA, uint32_t ldsB, int wave,
                                          uint32_t sb = 0) {
    constexpr int NS = (S + T::kStages - 1) % T::kStages;
    constexpr int kSA = DA::kSlots, kSB = DB::kSlots;
#pragma unroll
    for (int kk = 0; kk < T::kKK; ++kk) {
        bf16x8 af[T::MI], bfg[4];
#pragma unroll
        for (int i = 0; i < T::MI; ++i) {
            if constexpr (T::kAmx) {
                // volatile: the compiler would pair these reads (512 bytes
                // apart) into ds_read2st64_b64, whose two addresses per lane
                // share banks (measured: 2.6x the LDS cycles)
                const u32x2 c =
                    *(const volatile lds_u32x2*)(uintptr_t)(abase[kk] + S * T::kABytes + i * T::kFragA);
                const uint32_t s8 =
                    *(const lds_u8*)(uintptr_t)(sb + S * T::kABytes + i * 16 * 4 * MxDma<T>::kLPR + kk);
                af[i] = mx_frag(c, s8);
            } else if constexpr (A_K) {
                af[i] = lds_b128(abase[kk] + S * T::kABytes + i * T::kFrag);
            } else {
                af[i] = lds_tr_pair(abase[i] + S * T::kABytes + kk * 64 * T::BM, 8 * T::BM);
            }
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            constexpr uint32_t so = (S & 1) * T::kBBytes;
            if constexpr (B_K) bfg[j] = lds_b128(bbase[S >> 1][kk] + so + j * T::kFrag);
            else bfg[j] = lds_tr_pair(bbase[S >> 1][j] + so + kk * 64 * BN, 8 * BN);
        }
        if (next) {
            if (T::kKK == 1) {
                da.template issue<KTAIL, 0, kSA>(ldsA + NS * T::kABytes, nrem, wave);
                db.template issue<KTAIL, 0, kSB>(ldsB + NS * T::kBBytes, nrem, wave);
            } else if (kk == 0) {
                da.template issue<KTAIL, 0, kSA>(ldsA + NS * T::kABytes, nrem, wave);
                db.template issue<KTAIL, 0, kSB / 2>(ldsB + NS * T::kBBytes, nrem, wave);
            } else {
                db.template issue<KTAIL, kSB / 2, kSB>(ldsB + NS * T::kBBytes, nrem, wave);
            }
        }
#pragma unroll
        for (int i = 0; i < T::MI; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bfg[j], af[i], acc[i][j], 0, 0, 0);
    }
}

// Per-lane fragment bases of the A (BM-wide) and B (BN-wide) operands.
template <class T, bool A_K, bool B_K, int NA, int NB>
__device__ __forceinline__ void frag_bases(uint32_t (&abase)[NA], uint32_t (&bbase)[2][NB], uint32_t ldsA,
                                           uint32_t ldsB, int wm, int wn, int lane) {
#pragma unroll
    for (int i = 0; i < NA; ++i)
        abase[i] = ldsA + (T::kAmx ? mx_row_base<T::KD>(wm * (T::BM / 2), i, lane)
                           : A_K  ? row_base<T::KD>(wm * (T::BM / 2), i, lane)
                                  : col_base<T::BM>(wm * (T::BM / 2) + i * 16, lane));
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        const uint32_t o = B_K ? row_base<T::KD>(wn * 64, j, lane) : col_base<BN>(wn * 64 + j * 16, lane);
        bbase[0][j] = ldsB + o;                    // stages 0 and 1
        bbase[1][j] = ldsB + 2 * T::kBBytes + o;   // stages 2 and 3 (immediate offsets reach 64 KB)
    }
}

template <int MI>
__device__ __forceinline__ void zero_acc(f32x4 (&acc)[MI][4]) {
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
}

// Calls step(integral_constant<S>, g) for g = g0 .. g0 + kStages - 1 (those
// below total), S the ring slot of step g.
template <int kStages, class F>
__device__ __forceinline__ void ring_round(F&& step, int g0, int total) {
    step(std::integral_constant<int, 0>{}, g0);
    if (g0 + 1 < total) step(std::integral_constant<int, 1 % kStages>{}, g0 + 1);
    if constexpr (kStages >= 3)
        if (g0 + 2 < total) step(std::integral_constant<int, 2 % kStages>{}, g0 + 2);
    if constexpr (kStages >= 4)
        if (g0 + 3 < total) step(std::integral_constant<int, 3 % kStages>{}, g0 + 3);
}

// ---------------------------------------------------------------------------
// KGRP mode (wgrad): C_e[m, n] = sum over expert e's rows r of A[r, m] B[r, n],
// fp32 output.  One workgroup per (expert, m-tile, n-tile).
template <class T>
__device__ __forceinline__ void kgrp_item(const GemmArgs& p, int e, int in, char* smem);

// The pair launch's items are those of the expert order (slot r = the
// expert with the r-th most rows), each slot holding problem 0's items, then
// problem 1's.  Workgroups go to XCDs round-robin, so workgroup b is the
// (b / 8)-th of XCD b % 8, and every XCD runs its items in the order below:
//   heavy slots (the leading ones, at most 8, whose expert holds more than
//   R / 16 rows: its two gradients are then over half an XCD's fair share)
//   are cut into chunks of kKgChunk consecutive items, chunk c going to XCD
//   c % 8, so every XCD holds an equal share of the longest contractions
//   (whole units left the XCD with the busiest experts of a Zipf routing
//   at ~1.2x its share);
//   the other slots' units (one expert, one problem) follow whole, dealt
//   in rounds of 8 that alternate direction (unit 8k + i to XCD i, or 7 - i
//   when k is odd, counted from the XCD after the last heavy chunk), so
//   the units' decreasing sizes even out across XCDs, and the items an XCD
//   runs together keep one expert's operand rows in its L2 (cutting them
//   too cost 2.6% on a balanced routing).
// Each XCD's share is padded to the same length; the padding comes last.
constexpr int kKgChunk = 8;

struct KgItem {
    int r, q, in;   // slot, problem, item; r < 0: padding
};

// Slots whose expert holds more than R / 16 rows: a prefix of the order.
__device__ __forceinline__ int heavy_slots(const GemmArgs& p) {
    typedef const __attribute__((address_space(4))) int32_t* cptr;
    const cptr ord = (cptr)p.order, off = (cptr)p.offsets;
    const int n = p.E < kXcds ? p.E : kXcds;
    const int R = (int)p.R;
    int h = 0;
    for (; h < n; ++h) {
        int e = ord[h];
        e = (e >= 0 && e < p.E) ? e : h;
        int lo = off[e], hi = off[e + 1];
        lo = lo < 0 ? 0 : (lo > R ? R : lo);
        hi = hi < lo ? lo : (hi > R ? R : hi);
        if ((int64_t)(hi - lo) * 16 <= p.R) break;
    }
    return h;
}

__device__ __forceinline__ KgItem kg_item(unsigned b, int E, int per0, int per1, int H) {
    const int per = per0 + per1, perm = per0 > per1 ? per0 : per1;
    const int64_t heavy = (int64_t)H * per;
    const int n_hc = (int)((heavy + kKgChunk - 1) / kKgChunk);
    const int x = (int)(b % kXcds), j = (int)(b / kXcds);
    const int nhx = n_hc > x ? (n_hc - x + kXcds - 1) / kXcds : 0;   // heavy chunks on XCD x
    KgItem it{-1, 0, 0};
    if (perm == 0) return it;
    if (j < nhx * kKgChunk) {
        const int64_t g = (int64_t)(x + kXcds * (j / kKgChunk)) * kKgChunk + j % kKgChunk;
        if (g >= heavy) return it;
        it.r = (int)(g / per);
        const int rem = (int)(g - (int64_t)it.r * per);
        it.q = rem >= per0 ? 1 : 0;
        it.in = rem - it.q * per0;
        return it;
    }
    const int jj = j - nhx * kKgChunk, k = jj / perm;
    const int xp = ((x - n_hc) % kXcds + kXcds) % kXcds;
    const int u = kXcds * k + ((k & 1) ? kXcds - 1 - xp : xp);
    const int r = H + u / 2, q = u & 1, in = jj - k * perm;
    if (r >= E || in >= (q ? per1 : per0)) return it;
    return KgItem{r, q, in};
}

// The pair launch's grid: every XCD's longest possible share (8 heavy slots).
inline int64_t kg_grid(int E, int64_t per0, int64_t per1) {
    const int64_t per = per0 + per1, perm = per0 > per1 ? per0 : per1;
    const int64_t n_hc = ((E < kXcds ? E : kXcds) * per + kKgChunk - 1) / kKgChunk;
    return kXcds * ((n_hc + kXcds - 1) / kXcds * kKgChunk + (2 * (int64_t)E + kXcds - 1) / kXcds * perm);
}

// One launch: (row chunk, m-tile, n-tile) items, item `in` of chunk e.  Each
// XCD takes a contiguous range of chunks, so a chunk's items run
// consecutively on one XCD and share its rows in that XCD's L2.
template <class T>
__global__ __launch_bounds__(kGemmThreads, 1) void gemm_kgrp_kernel(GemmArgs p) {
    __shared__ __attribute__((aligned(1024))) char smem[T::kRingBytes];
    const int per = p.m_tiles * p.n_tiles;
    const int lid = xcd_remap(blockIdx.x, gridDim.x);
    const int e = lid / per;
    const int in = lid - e * per;
    kgrp_item<T>(p, e, in, smem);
}

// Two weight gradients over the same expert segments in one launch, items
// placed as above, so each gradient's long contractions overlap the other's
// instead of each launch ending on its own tail.
template <class T>
__global__ __launch_bounds__(kGemmThreads, 1) void gemm_kgrp2_kernel(GemmArgs p0, GemmArgs p1) {
    __shared__ __attribute__((aligned(1024))) char smem[T::kRingBytes];
    const KgItem it = kg_item(blockIdx.x, p0.E, p0.m_tiles * p0.n_tiles, p1.m_tiles * p1.n_tiles, heavy_slots(p0));
    if (it.r < 0) return;
    const GemmArgs& p = it.q ? p1 : p0;
    const int eo = ((const __attribute__((address_space(4))) int32_t*)p0.order)[it.r];
    const int e = (eo >= 0 && eo < p0.E) ? eo : it.r;
    kgrp_item<T>(p, e, it.in, smem);
}

// Item `in` (an m-tile, n-tile pair) of expert (or row chunk) e.
template <class T>
__device__ __forceinline__ void kgrp_item(const GemmArgs& p, int e, int in, char* smem) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar LDS offsets
    const int wm = wave >> 2, wn = wave & 3;
    // Two m-tiles at a time across all n-tiles: the ~32 items an XCD runs
    // together then share two m-tiles of A rows and a run of n-tiles of B
    // rows, which fit its L2 (all m-tiles at a time did not: the 31.5B
    // shape's wgrad 3286 -> ~3100 us; groups of 4 and 8 fell in between).
    constexpr int kKgM = 2;
    const int width = kKgM * p.n_tiles;
    const int grp = in / width, first_m = grp * kKgM;
    const int gsz = (p.m_tiles - first_m) < kKgM ? (p.m_tiles - first_m) : kKgM;
    const int in2 = in - grp * width;
    const int mt = first_m + in2 % gsz, nt = in2 / gsz;
    const int64_t row0 = (int64_t)mt * T::BM;
    const int64_t row_hi = (row0 + T::BM) < p.M ? (row0 + T::BM) : p.M;
    int64_t k_begin = p.offsets != nullptr ? (int64_t)p.offsets[e] : (int64_t)e * p.kchunk;
    int64_t k_end = p.offsets != nullptr ? (int64_t)p.offsets[e + 1] : k_begin + p.kchunk;
    k_begin = k_begin < 0 ? 0 : (k_begin > p.R ? p.R : k_begin);
    k_end = k_end < k_begin ? k_begin : (k_end > p.R ? p.R : k_end);
    const int64_t n0 = (int64_t)nt * BN;

    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_char*)smem;
    const uint32_t ldsB = lds0, ldsA = lds0 + T::kStages * T::kBBytes;

    DmaTile<false, T::BM, T::KD> da;
    DmaTile<false, BN, T::KD> db;
    da.init(p.A, p.lda, row0, row_hi, k_begin, k_end, wave, lane);
    db.init(p.B, p.ldb, n0, (int64_t)p.N, k_begin, k_end, wave, lane);
    constexpr int kSA = DmaTile<false, T::BM, T::KD>::kSlots, kSB = DmaTile<false, BN, T::KD>::kSlots;
    constexpr int kPerStage = kSA + kSB;

    uint32_t abase[T::MI], bbase[2][4];
    frag_bases<T, false, false>(abase, bbase, ldsA, ldsB, wm, wn, lane);

    f32x4 acc[T::MI][4];
    zero_acc(acc);

    const int64_t klen = k_end - k_begin;
    const int nk = (int)((klen + T::KD - 1) / T::KD);

    auto step = [&](auto stage_c, int kt) {
        constexpr int S = decltype(stage_c)::value;
        wait_stage<T, kPerStage>(kt, nk);
        stage_barrier();
        mma_stage<T, false, false, true, S>(acc, abase, bbase, da, db, kt + T::kStages - 1 < nk,
                                            klen - (int64_t)(kt + T::kStages - 1) * T::KD, ldsA, ldsB, wave);
    };

    if (nk > 0) {
        for (int q = 0; q < T::kStages - 1 && q < nk; ++q) {
            da.template issue<true, 0, kSA>(ldsA + q * T::kABytes, klen - (int64_t)q * T::KD, wave);
            db.template issue<true, 0, kSB>(ldsB + q * T::kBBytes, klen - (int64_t)q * T::KD, wave);
        }
        for (int kt = 0; kt < nk; kt += T::kStages) ring_round<T::kStages>(step, kt, nk);
    }

    // Epilogue through LDS (the ring is free once every wave has passed the
    // barrier): per 16-row block the wave's 16 x 64 fp32 go to its 4 KB
    // slice (16-byte chunk c of row r at c ^ r) and come back as whole
    // 256-byte row pieces, 4 rows per store instruction, written
    // non-temporally: the gradient is not read here, and full lines keep the
    // bypassing writes efficient while the operand rows stay in L2.
    __syncthreads();
    const int64_t c_base = (int64_t)e * p.c_stride;
    const uint32_t ep = lds0 + (uint32_t)wave * 4096u;
    const int r = lane & 15;
    const int rq = lane >> 4, c = lane & 15;
    const int64_t ncol = n0 + wn * 64 + c * 4;
#pragma unroll
    for (int i = 0; i < T::MI; ++i) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int ch = (j * 4 + (lane >> 4)) ^ r;
            *(__attribute__((address_space(3))) f32x4*)(uintptr_t)(ep + (uint32_t)(r * 256 + ch * 16)) = acc[i][j];
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int rr = q * 4 + rq;
            const f32x4 v =
                *(const __attribute__((address_space(3))) f32x4*)(uintptr_t)(ep + (uint32_t)(rr * 256 + ((c ^ rr) * 16)));
            const int64_t m = row0 + wm * (T::BM / 2) + i * 16 + rr;
            if (m < row_hi && ncol < p.N)
                __builtin_nontemporal_store(v, (f32x4*)((float*)p.C + c_base + m * p.ldc + ncol));
        }
    }
}

// ---------------------------------------------------------------------------
// ROWS mode, persistent.

struct RowsTile {
    int e, row0, row_hi, n0;  // rows and columns are below 2^31
};

static_assert(kSchedGroupM == kGroupM, "schedule runs and dense groups take the same m-tiles");

template <int BM>
__device__ __forceinline__ RowsTile rows_tile(const GemmArgs& p, const int4* tiles, int m_count, int w,
                                              int m_base) {
    typedef const __attribute__((address_space(4))) int32_t* cptr;
    // item w of the m-tiles [m_base, m_base + m_count) x all n-tiles, taken a
    // group of m-tiles at a time across all n-tiles: with a tile table the
    // groups are its runs of one expert's m-tiles (cut at the share's ends),
    // dense rows take kGroupM m-tiles at a time
    int mt, nt;
    if (tiles != nullptr) {
        // item w lies in the run that holds m-tile m_base + w / n_tiles (a
        // run of s m-tiles covers s * n_tiles consecutive items); the table
        // is written by an earlier launch and read-only here: scalar loads
        // through the constant address space
        const int q = m_base + w / p.n_tiles;
        const int packed = ((cptr)(tiles + q))[3];
        int a = packed >> 4, b = a + (packed & 15);
        a = a > m_base ? a : m_base;
        b = b < m_base + m_count ? b : m_base + m_count;
        if (a > q || b <= q) { a = q; b = q + 1; }   // an entry that does not hold q: take q alone
        const int s = b - a;
        const int in = w - (a - m_base) * p.n_tiles;
        mt = a + in % s;
        nt = in / s;
        nt = nt < p.n_tiles ? nt : p.n_tiles - 1;
    } else {
        const int width = kGroupM * p.n_tiles;
        const int group = w / width;
        const int first_m = group * kGroupM;
        const int gsz = (m_count - first_m) < kGroupM ? (m_count - first_m) : kGroupM;
        const int in = w - group * width;
        mt = m_base + first_m + in % gsz;
        nt = in / gsz;
    }
    mt = __builtin_amdgcn_readfirstlane(mt);
    RowsTile t;
    if (tiles != nullptr) {
        const __attribute__((address_space(4))) int32_t* ti =
            (const __attribute__((address_space(4))) int32_t*)(tiles + mt);
        t.e = ti[0];
        t.row0 = ti[1];
        t.row_hi = ti[2];
    } else {
        t.e = 0;
        t.row0 = mt * BM;
        t.row_hi = (t.row0 + BM) < p.M ? (t.row0 + BM) : (int)p.M;
    }
    t.n0 = nt * BN;
    return t;
}

// Buffer descriptor over rows [row0, row0 + nrows) of a row-major bf16 matrix:
// accesses at byte offsets >= nrows * ldc * 2 are dropped (stores) or read as
// zero (loads) by the hardware.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rows_rsrc(const void* base, int64_t row0, int64_t nrows,
                                                            int64_t ldc) {
    const uint16_t* b = (const uint16_t*)base + row0 * ldc;
    const int32_t bytes = nrows > 0 ? (int32_t)(nrows * ldc * 2) : 0;
    return __builtin_amdgcn_make_buffer_rsrc((void*)b, 0, bytes, 0x00020000);
}

constexpr uint32_t kDropOffset = 0x80000000u;  // beyond any descriptor's range

// Staged epilogue of one 64 x 64 wave tile (EPI_BF16 / EPI_RELU2 /
// EPI_DRELU2): per 16-row block, the accumulators go to the wave's LDS slice
// as bf16 (chunk c of row r at c ^ (r & 7)), come back as 16-byte row pieces
// and leave as two buffer_store_dwordx4 of 8 rows x 128 bytes each.  OUT:
// 0 = the product (squared-ReLU applied for EPI_RELU2; times 2 max(u, 0),
// u from uu at the accumulators' positions, for EPI_DRELU2), 1 = the raw
// product (pre-activation).
template <int EPI, int OUT, int MI>
__device__ __forceinline__ void staged_store(const f32x4 (&acc)[MI][4], void* C, int64_t ldc, int N,
                                             int64_t rbase, int64_t nrows, int64_t cbase,
                                             uint32_t ep, int lane, const u32x2 (*uu)[4] = nullptr) {
    const __amdgpu_buffer_rsrc_t rs = rows_rsrc(C, rbase, nrows, ldc);
    const int r = lane & 15;
    const uint32_t wr = ep + (uint32_t)(r * 128 + (lane >> 4 & 1) * 8);
    const int rr0 = lane >> 3, c = lane & 7;
    const bool col_ok = cbase + c * 8 < N;
#pragma unroll
    for (int i = 0; i < MI; ++i) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const f32x4 a = acc[i][j];
            float v0 = a[0], v1 = a[1], v2 = a[2], v3 = a[3];
            if constexpr (EPI == EPI_RELU2 && OUT == 0) {
                v0 = relu_f32(v0); v1 = relu_f32(v1); v2 = relu_f32(v2); v3 = relu_f32(v3);
                v0 *= v0; v1 *= v1; v2 *= v2; v3 *= v3;
            }
            if constexpr (EPI == EPI_DRELU2) {
                const u32x2 u = uu[i][j];
                v0 = v0 * 2.f * relu_f32(bf16_lo(u[0]));
                v1 = v1 * 2.f * relu_f32(bf16_hi(u[0]));
                v2 = v2 * 2.f * relu_f32(bf16_lo(u[1]));
                v3 = v3 * 2.f * relu_f32(bf16_hi(u[1]));
            }
            const int ch = 2 * j + (lane >> 5);
            const u32x2 w = {pack_bf16x2(v0, v1), pack_bf16x2(v2, v3)};
            *(lds_u32x2*)(uintptr_t)(wr + (uint32_t)((ch ^ (r & 7)) * 16)) = w;
        }
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int rr = q * 8 + rr0;
            const u32x4 v = *(const lds_u32x4*)(uintptr_t)(ep + (uint32_t)(rr * 128 + ((c ^ (rr & 7)) * 16)));
            const int64_t row = i * 16 + rr;
            const uint32_t off = (row < nrows && col_ok) ? (uint32_t)((row * ldc + cbase + c * 8) * 2) : kDropOffset;
            __builtin_amdgcn_raw_buffer_store_b128(v, rs, off, 0, 0);
        }
    }
}

// dgrad epilogue: C = bf16(acc * 2 max(u, 0)) with u read from aux_in at the
// accumulators' own positions (8 bytes per lane and fragment), written by
// staged_store.  The sixteen u loads are issued by drelu2_load at the tile's
// first k step (right after its barrier, before that step's operand
// copies), so they have long completed when the epilogue uses them: its
// waits never reach the copies in flight at the tile's end.
template <int MI>
__device__ __forceinline__ void drelu2_load(u32x2 (&uu)[MI][4], const uint16_t* aux_in, int64_t ldc, int N,
                                            int64_t rbase, int64_t nrows, int64_t cbase, int lane) {
    const __amdgpu_buffer_rsrc_t ru = rows_rsrc(aux_in, rbase, nrows, ldc);
#pragma unroll
    for (int i = 0; i < MI; ++i) {
        const int64_t row = i * 16 + (lane & 15);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t col = cbase + j * 16 + 4 * (lane >> 4);
            const uint32_t off = (row < nrows && col < N) ? (uint32_t)((row * ldc + col) * 2) : kDropOffset;
            uu[i][j] = __builtin_amdgcn_raw_buffer_load_b64(ru, off, 0, 0);
        }
    }
}

// fp32 epilogue: each lane's four accumulators of a fragment are four
// consecutive columns of one row, stored as one 16-byte buffer store (with
// `accumulate`, added to what C holds there).  The descriptor spans only this
// wave's rows, so rows past the tile and columns past N are dropped.
template <int MI>
__device__ __forceinline__ void f32_store(const f32x4 (&acc)[MI][4], float* C, int64_t ldc, int N,
                                          int64_t rbase, int64_t nrows, int64_t cbase, bool accumulate,
                                          int lane) {
    const int64_t rows = nrows < MI * 16 ? nrows : MI * 16;
    const int32_t bytes = rows > 0 ? (int32_t)(rows * ldc * 4) : 0;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc((void*)(C + rbase * ldc), 0, bytes,
                                                                        0x00020000);
#pragma unroll
    for (int i = 0; i < MI; ++i) {
        const int64_t row = i * 16 + (lane & 15);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t col = cbase + j * 16 + 4 * (lane >> 4);
            const uint32_t off = (row < rows && col < N) ? (uint32_t)((row * ldc + col) * 4) : kDropOffset;
            f32x4 v = acc[i][j];
            if (accumulate) {
                const u32x4 o = __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0);
                v[0] += __uint_as_float(o[0]);
                v[1] += __uint_as_float(o[1]);
                v[2] += __uint_as_float(o[2]);
                v[3] += __uint_as_float(o[3]);
            }
            const u32x4 w = {__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]),
                             __float_as_uint(v[3])};
            __builtin_amdgcn_raw_buffer_store_b128(w, rs, off, 0, 0);
        }
    }
}

// C[r, n] = sum_k A[r, k] B_e[k, n] over the grid-wide list of output tiles
// (expert segments from the tile table `tiles` with m_total valid m-tiles,
// or all M rows when it is null), in tiles of T::BM rows.  A is K-contiguous
// (ROW layout); B is N-contiguous (B_K false: weights stored [Kd, N]) or
// K-contiguous (B_K true: transposed weights of the dgrads).  KTAIL: Kd is
// not a multiple of 64.
template <class T, bool B_K, int EPI, bool KTAIL>
__device__ __forceinline__ void rows_body(const GemmArgs& p, char* smem, const int4* tiles, int m_total) {
    constexpr int BM = T::BM, MI = T::MI, KD = T::KD, kStages = T::kStages;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 2, wn = wave & 3;

    // Each XCD's G / 8 workgroups (workgroups go to XCDs round-robin) take a
    // contiguous eighth of the m-tiles, all n-tiles, in group-M order; this
    // workgroup takes items w = lx + j * (G / 8) of its XCD's share.  The
    // tile list is expert-major, so an expert's weights stream through one
    // XCD's L2 (two where a share boundary splits the expert) instead of
    // every XCD whose m-tile groups touch it.
    const int G = gridDim.x;   // a multiple of kXcds
    const int Gx = G / kXcds;
    const int xcd = (int)(blockIdx.x % kXcds), lx = (int)(blockIdx.x / kXcds);
    const int m_base = (int)((int64_t)m_total * xcd / kXcds);
    const int m_count = (int)((int64_t)m_total * (xcd + 1) / kXcds) - m_base;
    const int n_work = m_count * p.n_tiles;
    const int n_mine = lx < n_work ? (n_work - lx + Gx - 1) / Gx : 0;
    const int nk = (p.Kd + KD - 1) / KD;
    const int g_total = n_mine * nk;  // (tile, k step) pairs
    if (g_total == 0) return;

    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_char*)smem;
    const uint32_t ldsB = lds0, ldsA = lds0 + kStages * T::kBBytes;
    const uint32_t ep = lds0 + T::kRingBytes + (uint32_t)wave * kEpiWaveBytes;

    using DA = std::conditional_t<T::kAmx, MxDma<T>, DmaTile<true, BM, KD>>;
    DA da;
    DmaTile<B_K, BN, KD> db;
    constexpr int kSA = DA::kSlots, kSB = DmaTile<B_K, BN, KD>::kSlots;
    constexpr int kPerStage = kSA + kSB;
    auto dma_tile = [&](int j) {
        const RowsTile t = rows_tile<BM>(p, tiles, m_count, lx + j * Gx, m_base);
        if constexpr (T::kAmx)
            da.init((const uint8_t*)p.A, p.A_scale, p.scale_bytes, t.row0, t.row_hi, p.Kd, wave, lane);
        else if (p.a_perm != nullptr)
            da.init_gather(p.A, p.lda, p.a_perm, p.a_div, p.a_src_rows, t.row0, t.row_hi, wave, lane);
        else
            da.init(p.A, p.lda, t.row0, t.row_hi, 0, p.Kd, wave, lane);
        db.init(p.B + (int64_t)t.e * p.b_stride, p.ldb, t.n0, (int64_t)p.N, 0, p.Kd, wave, lane);
    };

    constexpr int kNB = B_K ? T::kKK : 4;
    uint32_t abase[T::kKK], bbase[2][kNB];
    frag_bases<T, true, B_K>(abase, bbase, ldsA, ldsB, wm, wn, lane);

    f32x4 acc[MI][4];
    zero_acc(acc);

    // AMX: the lane's rows are r0 + 16 i; their scale windows sit 4 * kLPR
    // bytes apart, and all share the in-window byte offset (row * nb + kb) & 3.
    const int nb = p.Kd / 32;
    const int r0_lane = wm * (BM / 2) + (lane & 15);
    uint32_t sbase = 0, rnb = 0;
    if constexpr (T::kAmx) {
        sbase = ldsA + T::kCodeBytes + (uint32_t)r0_lane * 4u * MxDma<T>::kLPR;
        rnb = (uint32_t)(r0_lane * nb);
    }

    // DMA of the first kStages - 1 steps; kd / jd track the next step to send.
    int kd = 0, jd = 0;
    for (int q = 0; q < kStages - 1 && q < g_total; ++q) {
        if (kd == 0) dma_tile(jd);
        const int rem = p.Kd - kd * KD;
        da.template issue<KTAIL, 0, kSA>(ldsA + q * T::kABytes, rem, wave);
        db.template issue<KTAIL, 0, kSB>(ldsB + q * T::kBBytes, rem, wave);
        if (++kd == nk) { kd = 0; ++jd; }
    }

    int kc = 0;   // k step of the tile being computed
    int jc = 0;   // its index in this workgroup's list
    RowsTile cur = rows_tile<BM>(p, tiles, m_count, lx, m_base);
    u32x2 uu[MI][4];   // dgrad: the tile's pre-activations

    auto step = [&](auto stage_c, int g) {
        constexpr int S = decltype(stage_c)::value;
        // Stages g .. g + kStages - 2 are in flight and stage g must have
        // landed.  Stores of an epilogue may still be in flight; they are
        // not counted, so the wait covers this stage's copies whichever way
        // they complete (loads complete in order among themselves).
        wait_stage<T, kPerStage>(g, g_total);
        stage_barrier();
        if constexpr (EPI == EPI_DRELU2 && MI <= 4)   // with taller tiles: loaded in the epilogue
            if (kc == 0)
                drelu2_load(uu, p.aux_in, p.ldc, p.N, cur.row0 + wm * (BM / 2),
                            cur.row_hi - (cur.row0 + wm * (BM / 2)), cur.n0 + wn * 64, lane);
        const bool next = g + kStages - 1 < g_total;
        if (next && kd == 0) dma_tile(jd);
        uint32_t sb = 0;
        if constexpr (T::kAmx) sb = sbase + (((uint32_t)(cur.row0 * nb + kc * T::kKK) + rnb) & 3u);
        mma_stage<T, true, B_K, KTAIL, S>(acc, abase, bbase, da, db, next, p.Kd - kd * KD, ldsA, ldsB, wave,
                                          sb);
        if (++kd == nk) { kd = 0; ++jd; }
        if (kc == nk - 1) {
            const int rbase = cur.row0 + wm * (BM / 2);
            const int nrows = cur.row_hi - rbase;
            const int cbase = cur.n0 + wn * 64;
            if constexpr (EPI == EPI_DRELU2) {
                if constexpr (MI > 4) drelu2_load(uu, p.aux_in, p.ldc, p.N, rbase, nrows, cbase, lane);
                staged_store<EPI, 0, MI>(acc, p.C, p.ldc, p.N, rbase, nrows, cbase, ep, lane, uu);
            } else if constexpr (EPI == EPI_F32) {
                f32_store(acc, (float*)p.C, p.ldc, p.N, rbase, nrows, cbase, p.accumulate != 0, lane);
            } else {
                staged_store<EPI, 0, MI>(acc, p.C, p.ldc, p.N, rbase, nrows, cbase, ep, lane);
                if constexpr (EPI == EPI_RELU2)
                    if (p.aux_out != nullptr)
                        staged_store<EPI, 1, MI>(acc, p.aux_out, p.ldc, p.N, rbase, nrows, cbase, ep, lane);
            }
            zero_acc(acc);
            kc = 0;
            ++jc;
            if (jc < n_mine) cur = rows_tile<BM>(p, tiles, m_count, lx + jc * Gx, m_base);
        } else {
            ++kc;
        }
    };

    for (int g = 0; g < g_total; g += kStages) ring_round<kStages>(step, g, g_total);
}

// Relative time of one 256-row tile against two 128-row tiles: the tall tile
// moves a third fewer operand bytes per product (measured 0.91 over the five
// layer shapes' real routing counts).
constexpr int kTallTileCostPct = 91;

// The tile height of a launch, from the m-tile counts of both heights: the
// busiest XCD's rounds of each (ceil(m / 8) m-tiles times n_tiles items over
// G / 8 workgroups), tall tiles when their rounds cost less.  Every
// workgroup reads the same counts, so the whole grid takes the same body.
__device__ __forceinline__ bool take_tall_tiles(int m_small, int m_tall, int n_tiles, int G) {
    const int Gx = G / kXcds;
    const int r_small = ((m_small + kXcds - 1) / kXcds * n_tiles + Gx - 1) / Gx;
    const int r_tall = ((m_tall + kXcds - 1) / kXcds * n_tiles + Gx - 1) / Gx;
    return 2 * r_tall * kTallTileCostPct < 100 * r_small;
}

constexpr int kRowsSmemBytes =
    (TileS::kRingBytes > TileL::kRingBytes ? TileS::kRingBytes : TileL::kRingBytes) + kEpiBytes;

// The ROWS launch: one body per tile height, chosen on the device from the
// tile schedule's counts (known only after routing).  Products with k-major
// weights (the dgrads) always take 128-row tiles: measured on the same five
// shapes, the tall tile never won for them.
template <bool B_K, int EPI, bool KTAIL>
__global__ __launch_bounds__(kGemmThreads, 1) void gemm_rows_kernel(GemmArgs p) {
    __shared__ __attribute__((aligned(1024))) char smem[kRowsSmemBytes];
    typedef const __attribute__((address_space(4))) int32_t* cnt_ptr;
    // the table's count, never beyond the table (the builder caps it too)
    const int m_small = p.mtile_total != nullptr ? min(*(cnt_ptr)p.mtile_total, p.m_tiles) : p.m_tiles;
    if constexpr (!B_K) {
        const int m_tall = p.mtile_total_l != nullptr ? min(*(cnt_ptr)p.mtile_total_l, p.m_tiles_l) : p.m_tiles_l;
        if (take_tall_tiles(m_small, m_tall, p.n_tiles, (int)gridDim.x)) {
            rows_body<TileL, B_K, EPI, KTAIL>(p, smem, p.tiles_l, m_tall);
            return;
        }
    }
    rows_body<TileS, B_K, EPI, KTAIL>(p, smem, p.tiles, m_small);
}

constexpr int kRowsMxSmemBytes =
    (TileSX::kRingBytes > TileLX::kRingBytes ? TileSX::kRingBytes : TileLX::kRingBytes) + kEpiBytes;

// The ROWS launch over an MX-FP8 A (the up projection reading the dispatch
// payload as sent): the same bodies with the codes and scales in the ring
// and the decode in the fragment read; the tile height is chosen as above.
template <int EPI, bool KTAIL>
__global__ __launch_bounds__(kGemmThreads, 1) void gemm_rows_mx_kernel(GemmArgs p) {
    __shared__ __attribute__((aligned(1024))) char smem[kRowsMxSmemBytes];
    typedef const __attribute__((address_space(4))) int32_t* cnt_ptr;
    // the table's count, never beyond the table (the builder caps it too)
    const int m_small = p.mtile_total != nullptr ? min(*(cnt_ptr)p.mtile_total, p.m_tiles) : p.m_tiles;
    const int m_tall = p.mtile_total_l != nullptr ? min(*(cnt_ptr)p.mtile_total_l, p.m_tiles_l) : p.m_tiles_l;
    if (take_tall_tiles(m_small, m_tall, p.n_tiles, (int)gridDim.x)) {
        rows_body<TileLX, false, EPI, KTAIL>(p, smem, p.tiles_l, m_tall);
        return;
    }
    rows_body<TileSX, false, EPI, KTAIL>(p, smem, p.tiles, m_small);
}

static_assert(kSchedBM[0] == TileS::BM && kSchedBM[1] == TileL::BM, "schedule tile heights");

__global__ __launch_bounds__(1024) void tile_schedule_kernel(const int32_t* __restrict__ offsets, int E, int R,
                                                              SchedPart small, SchedPart large) {
    build_tile_schedule(offsets, E, R, small, large);
}

int gemm_tile_m() { return TileS::BM; }

size_t gemm_schedule_bytes(int E, int64_t R) {
    return sched_part_bytes(E, R, TileS::BM) + sched_part_bytes(E, R, TileL::BM);
}

// Compute units of the current device, read once per device.
int cu_count() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    static std::once_flag once[64];
    static int cus[64];
    std::call_once(once[dev], [dev] {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
            n = 256;
        cus[dev] = n;
    });
    return cus[dev];
}

// The persistent grid: one workgroup per CU (a multiple of the XCD count).
static int64_t persistent_grid() {
    int64_t G = (cu_count() / kXcds) * kXcds;
    return G < kXcds ? kXcds : G;
}

// Workgroups of a ROWS launch: never more than the static bound on the
// number of output tiles (0: nothing to do).
static int64_t rows_grid(const GemmArgs& a) {
    const int64_t bound = (int64_t)a.m_tiles * a.n_tiles;
    if (bound <= 0) return 0;
    const int64_t G = persistent_grid();
    const int64_t need = (bound + kXcds - 1) / kXcds * kXcds;
    return need < G ? need : G;
}

template <bool B_K, int EPI>
static hipError_t launch_rows(const GemmArgs& a, hipStream_t st) {
    const int64_t G = rows_grid(a);
    if (G == 0) return hipSuccess;
    if (a.Kd % TileS::KD != 0)
        hipLaunchKernelGGL((gemm_rows_kernel<B_K, EPI, true>), dim3((unsigned)G), dim3(kGemmThreads), 0, st, a);
    else
        hipLaunchKernelGGL((gemm_rows_kernel<B_K, EPI, false>), dim3((unsigned)G), dim3(kGemmThreads), 0, st, a);
    return launch_check(st);
}

template <int EPI>
static hipError_t launch_rows_mx(const GemmArgs& a, hipStream_t st) {
    const int64_t G = rows_grid(a);
    if (G == 0) return hipSuccess;
    if (a.Kd % TileS::KD != 0)
        hipLaunchKernelGGL((gemm_rows_mx_kernel<EPI, true>), dim3((unsigned)G), dim3(kGemmThreads), 0, st, a);
    else
        hipLaunchKernelGGL((gemm_rows_mx_kernel<EPI, false>), dim3((unsigned)G), dim3(kGemmThreads), 0, st, a);
    return launch_check(st);
}

static hipError_t launch_rows_epi(const GemmArgs& a, bool b_kmajor, int epi, hipStream_t st) {
    if (!b_kmajor) {
        if (epi == EPI_BF16) return launch_rows<false, EPI_BF16>(a, st);
        if (epi == EPI_RELU2) return launch_rows<false, EPI_RELU2>(a, st);
        if (epi == EPI_F32) return launch_rows<false, EPI_F32>(a, st);
    } else {
        if (epi == EPI_BF16) return launch_rows<true, EPI_BF16>(a, st);
        if (epi == EPI_DRELU2) return launch_rows<true, EPI_DRELU2>(a, st);
        if (epi == EPI_F32) return launch_rows<true, EPI_F32>(a, st);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_tile_schedule(const int32_t* offsets, int E, int64_t R, void* sched, hipStream_t st) {
    hipLaunchKernelGGL(tile_schedule_kernel, dim3(1), dim3(1024), 0, st, offsets, E, (int)R,
                       sched_part(sched, E, R, false), sched_part(sched, E, R, true));
    return launch_check(st);
}

// The operand-independent part of a ROWS launch: B, C, sizes and both tile
// heights' schedule tables (the kernel picks one from their counts).
static void rows_args(GemmArgs& a, const moe_bf16* B, int64_t ldb, int64_t b_stride, void* C, int64_t ldc,
                      moe_bf16* aux_out, const void* sched, int E, int64_t R, int N, int Kd) {
    a.B = B; a.C = C; a.aux_out = aux_out;
    a.ldb = ldb; a.ldc = ldc; a.b_stride = b_stride;
    a.M = R; a.R = R; a.N = N; a.Kd = Kd; a.E = E;
    a.n_tiles = (N + BN - 1) / BN;
    if (sched != nullptr) {
        const SchedPart ss = sched_part((void*)sched, E, R, false), sl = sched_part((void*)sched, E, R, true);
        a.tiles = ss.tiles;
        a.mtile_total = ss.mtile_start + E;  // mtile_start[E]
        a.m_tiles = ss.max_tiles;
        a.tiles_l = sl.tiles;
        a.mtile_total_l = sl.mtile_start + E;
        a.m_tiles_l = sl.max_tiles;
    } else {
        a.m_tiles = (int)((R + TileS::BM - 1) / TileS::BM);
        a.m_tiles_l = (int)((R + TileL::BM - 1) / TileL::BM);
    }
}

hipError_t launch_grouped_rows(const moe_bf16* A, int64_t lda, const moe_bf16* B, int64_t ldb,
                               int64_t b_stride, bool b_kmajor, void* C, int64_t ldc, int epi,
                               const moe_bf16* aux_in, moe_bf16* aux_out, const void* sched,
                               int E, int64_t R, int N, int Kd, hipStream_t st, bool accumulate) {
    if (R == 0) return hipSuccess;
    // the DMA descriptor of an N-contiguous B spans its whole contraction
    if (!b_kmajor && (int64_t)Kd * ldb * 2 >= kMaxDmaBytes) return hipErrorInvalidValue;
    GemmArgs a{};
    a.A = A; a.aux_in = aux_in;
    a.accumulate = accumulate ? 1 : 0;
    a.lda = lda;
    rows_args(a, B, ldb, b_stride, C, ldc, aux_out, sched, E, R, N, Kd);
    return launch_rows_epi(a, b_kmajor, epi, st);
}

hipError_t launch_grouped_rows_gather(const moe_bf16* X, int64_t ldx, int64_t x_rows, const int32_t* perm, int div,
                                      const moe_bf16* B, int64_t ldb, int64_t b_stride, void* C, int64_t ldc, int epi,
                                      moe_bf16* aux_out, const void* sched, int E, int64_t R, int N, int Kd,
                                      hipStream_t st) {
    if (R == 0) return hipSuccess;
    if ((int64_t)Kd * ldb * 2 >= kMaxDmaBytes || x_rows * ldx * 2 >= kMaxDmaBytes || div < 1)
        return hipErrorInvalidValue;
    GemmArgs a{};
    a.A = X;
    a.lda = ldx;
    a.a_perm = perm;
    a.a_div = div;
    a.a_src_rows = x_rows;
    rows_args(a, B, ldb, b_stride, C, ldc, aux_out, sched, E, R, N, Kd);
    return launch_rows_epi(a, false, epi, st);
}

hipError_t launch_grouped_rows_mx(const uint8_t* Aq, const uint8_t* A_scale, const moe_bf16* B, int64_t ldb,
                                  int64_t b_stride, void* C, int64_t ldc, int epi, moe_bf16* aux_out,
                                  const void* sched, int E, int64_t R, int N, int Kd, hipStream_t st) {
    if (R == 0) return hipSuccess;
    if (Kd <= 0 || Kd % 32 != 0 || ((uintptr_t)Aq & 15u) != 0) return hipErrorInvalidValue;
    if ((int64_t)Kd * ldb * 2 >= kMaxDmaBytes) return hipErrorInvalidValue;
    const int64_t scale_bytes = (R * (Kd / 32) + 3) / 4 * 4;
    if (scale_bytes >= kMaxDmaBytes) return hipErrorInvalidValue;
    GemmArgs a{};
    a.A = (const uint16_t*)Aq;
    a.A_scale = A_scale;
    a.scale_bytes = (uint32_t)scale_bytes;
    a.lda = Kd;
    rows_args(a, B, ldb, b_stride, C, ldc, aux_out, sched, E, R, N, Kd);
    if (epi == EPI_BF16) return launch_rows_mx<EPI_BF16>(a, st);
    if (epi == EPI_RELU2) return launch_rows_mx<EPI_RELU2>(a, st);
    return hipErrorInvalidValue;
}


// KGRP launches: tall tiles when there are enough workgroups to fill the
// device a few times over.
static hipError_t launch_kgrp(GemmArgs a, int64_t groups, hipStream_t st) {
    const int64_t nt = (a.N + BN - 1) / BN;
    const int64_t mt_l = (a.M + TileL::BM - 1) / TileL::BM;
    const bool large = groups * mt_l * nt >= 2 * persistent_grid();
    a.m_tiles = (int)(large ? mt_l : (a.M + TileS::BM - 1) / TileS::BM);
    a.n_tiles = (int)nt;
    const int64_t n_wg = groups * a.m_tiles * a.n_tiles;
    if (n_wg <= 0) return hipSuccess;
    if (n_wg > 0x7fffffff) return hipErrorInvalidConfiguration;
    if (large)
        hipLaunchKernelGGL(gemm_kgrp_kernel<TileL>, dim3((unsigned)n_wg), dim3(kGemmThreads), 0, st, a);
    else
        hipLaunchKernelGGL(gemm_kgrp_kernel<TileS>, dim3((unsigned)n_wg), dim3(kGemmThreads), 0, st, a);
    return launch_check(st);
}

// Both weight gradients of the expert FFN in one launch (gemm_kgrp2_kernel),
// items of the experts with the most rows first.
hipError_t launch_grouped_wgrad2(const moe_bf16* A0, int64_t lda0, const moe_bf16* B0, int64_t ldb0, float* C0,
                                 int64_t ldc0, int64_t c_stride0, int M0, int N0, const moe_bf16* A1, int64_t lda1,
                                 const moe_bf16* B1, int64_t ldb1, float* C1, int64_t ldc1, int64_t c_stride1, int M1,
                                 int N1, const int32_t* offsets, const int32_t* order, int E, int64_t R,
                                 hipStream_t st) {
    if (R * (lda0 > ldb0 ? lda0 : ldb0) * 2 >= kMaxDmaBytes || R * (lda1 > ldb1 ? lda1 : ldb1) * 2 >= kMaxDmaBytes)
        return hipErrorInvalidValue;
    if (order == nullptr || E < 1) return hipErrorInvalidValue;
    GemmArgs a[2] = {};
    const moe_bf16* As[2] = {A0, A1};
    const moe_bf16* Bs[2] = {B0, B1};
    float* Cs[2] = {C0, C1};
    const int64_t lda[2] = {lda0, lda1}, ldb[2] = {ldb0, ldb1}, ldc[2] = {ldc0, ldc1}, cs[2] = {c_stride0, c_stride1};
    const int Ms[2] = {M0, M1}, Ns[2] = {N0, N1};
    int64_t items_l = 0;
    for (int q = 0; q < 2; ++q) {
        a[q].A = As[q]; a[q].B = Bs[q]; a[q].C = Cs[q]; a[q].offsets = offsets; a[q].order = order;
        a[q].lda = lda[q]; a[q].ldb = ldb[q]; a[q].ldc = ldc[q]; a[q].c_stride = cs[q];
        a[q].M = Ms[q]; a[q].R = R; a[q].N = Ns[q]; a[q].E = E;
        items_l += (int64_t)E * ((Ms[q] + TileL::BM - 1) / TileL::BM) * ((Ns[q] + BN - 1) / BN);
    }
    // tall tiles when both gradients have enough items to fill the device a few times over
    const bool large = items_l >= 4 * persistent_grid();
    for (int q = 0; q < 2; ++q) {
        a[q].m_tiles = (int)((Ms[q] + (large ? TileL::BM : TileS::BM) - 1) / (large ? TileL::BM : TileS::BM));
        a[q].n_tiles = (Ns[q] + BN - 1) / BN;
    }
    const int64_t n_wg =
        kg_grid(E, (int64_t)a[0].m_tiles * a[0].n_tiles, (int64_t)a[1].m_tiles * a[1].n_tiles);
    if (n_wg > 0x7fffffff) return hipErrorInvalidConfiguration;
    if (large)
        hipLaunchKernelGGL(gemm_kgrp2_kernel<TileL>, dim3((unsigned)n_wg), dim3(kGemmThreads), 0, st, a[0], a[1]);
    else
        hipLaunchKernelGGL(gemm_kgrp2_kernel<TileS>, dim3((unsigned)n_wg), dim3(kGemmThreads), 0, st, a[0], a[1]);
    return launch_check(st);
}

hipError_t launch_chunked_wgrad(const moe_bf16* A, int64_t lda, const moe_bf16* B, int64_t ldb, float* C,
                                int64_t ldc, int64_t c_stride, int nchunk, int64_t kchunk, int M, int N,
                                int64_t R, hipStream_t st) {
    GemmArgs a{};
    a.A = A; a.B = B; a.C = C; a.offsets = nullptr; a.kchunk = kchunk;
    a.lda = lda; a.ldb = ldb; a.ldc = ldc; a.c_stride = c_stride;
    a.M = M; a.R = R; a.N = N; a.E = nchunk;
    if (R * (lda > ldb ? lda : ldb) * 2 >= kMaxDmaBytes) return hipErrorInvalidValue;
    return launch_kgrp(a, nchunk, st);
}

// Experts ranked by row count, most first (ties to the lower index):
// order[rank] = e.  One workgroup; each thread counts, for its experts, the
// experts that come before them.
__global__ __launch_bounds__(1024) void expert_order_kernel(const int32_t* __restrict__ offsets, int E, int R,
                                                            int32_t* __restrict__ order) {
    __shared__ int32_t cnt[1024];
    for (int e = threadIdx.x; e < E; e += 1024) {
        int lo = offsets[e], hi = offsets[e + 1];
        lo = lo < 0 ? 0 : (lo > R ? R : lo);
        hi = hi < lo ? lo : (hi > R ? R : hi);
        cnt[e] = hi - lo;
    }
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += 1024) {
        const int c = cnt[e];
        int rank = 0;
        for (int f = 0; f < E; ++f) rank += (cnt[f] > c || (cnt[f] == c && f < e)) ? 1 : 0;
        order[rank] = e;
    }
}

hipError_t launch_expert_order(const int32_t* offsets, int E, int64_t R, int32_t* order, hipStream_t st) {
    hipLaunchKernelGGL(expert_order_kernel, dim3(1), dim3(1024), 0, st, offsets, E, (int)R, order);
    return launch_check(st);
}


}  // namespace moe
