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
// Tiles are BM x BN x BK = 128 x 128 x 64 on 256 threads (4 wavefronts in a
// 2 x 2 grid, 64 x 64 outputs each, 16 v_mfma_f32_16x16x32_bf16 per 32-wide k
// step).  Both operands live in LDS as "rows of K-contiguous 16-byte chunks"
// with an XOR swizzle on the chunk index, which is the layout the MFMA
// operand reads want.  An operand whose source is K-contiguous is copied
// straight in; one whose source is M/N-contiguous (weights stored [D, F] or
// [F, D], and both wgrad operands) is read as 4x8 bf16 blocks with 16-byte
// loads and transposed in registers before the LDS write.  LDS is double
// buffered with the next tile's global loads issued before the current
// tile's MFMAs.
//
// The MFMA is issued with the weight tile as its first operand, so each
// lane's four accumulators hold four consecutive output columns of one row:
// the epilogue stores 8 bytes (bf16) or 16 bytes (fp32) per lane directly,
// after fusing squared-ReLU (up), its derivative (dgrad), or nothing.
//
// Workgroups of one expert segment are found from a device-side tile
// schedule (prefix sum of per-expert tile counts), so no host ever reads the
// routing counts; workgroup ids are remapped so that consecutive tiles land
// on the same XCD and share its L2.
#include "common.h"
#include "kernels.h"

namespace moe {

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int kGemmThreads = 256;
constexpr int kChunks = BK / 8;     // 16-byte chunks per LDS row
constexpr int kGroupM = 8;          // m-tiles per scheduling group
constexpr int kXcds = 8;

enum { MODE_ROWS = 0, MODE_KGRP = 1 };

struct GemmArgs {
    const uint16_t* A;
    const uint16_t* B;
    void* C;
    const uint16_t* aux_in;   // EPI_DRELU2: pre-activation u, same layout as C
    uint16_t* aux_out;        // EPI_RELU2: pre-activation u (may be null)
    const int32_t* offsets;   // [E+1] expert row segments; null = one dense segment
    const int32_t* mtile_start;  // [E+1] ROWS mode with offsets
    int64_t lda, ldb, ldc;
    int64_t b_stride;         // elements between experts' B (ROWS mode)
    int64_t c_stride;         // elements between experts' C (KGRP mode)
    int64_t M;                // dense rows (ROWS, no offsets) or output rows (KGRP)
    int64_t R;                // rows of the activation buffers: segments are clamped to [0, R)
    int N, Kd, E;
    int m_tiles, n_tiles;
};

__device__ __forceinline__ int swz(int row) { return (row ^ (row >> 3)) & (kChunks - 1); }

// Byte offset of chunk c of LDS row r.
__device__ __forceinline__ int lds_off(int r, int c) { return (r * kChunks + (c ^ swz(r))) * 16; }

// Tile rows [r0, r0+ROWS) x k [k0, k0+BK) from a K-contiguous source:
// element (r, k) at src[r*ld + k]; rows >= r_hi and k >= k_hi read as zero.
template <int ROWS>
struct KMajorTile {
    static constexpr int kPer = ROWS * kChunks / kGemmThreads;
    uint4 v[kPer];
    __device__ __forceinline__ void load(const uint16_t* __restrict__ src, int64_t ld, int64_t r0,
                                         int64_t r_hi, int64_t k0, int64_t k_hi, int tid) {
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            const int q = tid + kGemmThreads * i;
            const int r = q / kChunks, c = q % kChunks;
            const int64_t gr = r0 + r, gk = k0 + c * 8;
            if (gr < r_hi && gk < k_hi)
                v[i] = *(const uint4*)(src + gr * ld + gk);
            else
                v[i] = make_uint4(0, 0, 0, 0);
        }
    }
    __device__ __forceinline__ void store(char* lds, int tid) const {
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            const int q = tid + kGemmThreads * i;
            const int r = q / kChunks, c = q % kChunks;
            *(uint4*)(lds + lds_off(r, c)) = v[i];
        }
    }
};

// Tile rows [r0, r0+ROWS) x k [k0, k0+BK) from a row(M/N)-contiguous source:
// element (r, k) at src[k*ld + r].  Each thread loads a 4(k) x 8(r) block
// with four 16-byte loads and writes it transposed as eight 8-byte pieces.
template <int ROWS>
struct MNMajorTile {
    static constexpr int kRB = ROWS / 8;                       // 8-row blocks
    static constexpr int kBlocks = (BK / 4) * kRB;
    static constexpr int kPer = kBlocks / kGemmThreads;
    uint4 v[kPer][4];
    __device__ __forceinline__ void load(const uint16_t* __restrict__ src, int64_t ld, int64_t r0,
                                         int64_t r_hi, int64_t k0, int64_t k_hi, int tid) {
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            const int b = tid + kGemmThreads * i;
            const int kb = b / kRB, rb = b % kRB;
            const int64_t gr = r0 + rb * 8;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int64_t gk = k0 + kb * 4 + q;
                if (gr < r_hi && gk < k_hi)
                    v[i][q] = *(const uint4*)(src + gk * ld + gr);
                else
                    v[i][q] = make_uint4(0, 0, 0, 0);
            }
        }
    }
    __device__ __forceinline__ void store(char* lds, int tid) const {
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            const int b = tid + kGemmThreads * i;
            const int kb = b / kRB, rb = b % kRB;
            const uint32_t* w0 = (const uint32_t*)&v[i][0];
            const uint32_t* w1 = (const uint32_t*)&v[i][1];
            const uint32_t* w2 = (const uint32_t*)&v[i][2];
            const uint32_t* w3 = (const uint32_t*)&v[i][3];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int wd = j >> 1;
                uint32_t lo, hi;
                if (j & 1) {
                    lo = (w0[wd] >> 16) | (w1[wd] & 0xffff0000u);
                    hi = (w2[wd] >> 16) | (w3[wd] & 0xffff0000u);
                } else {
                    lo = (w0[wd] & 0xffffu) | (w1[wd] << 16);
                    hi = (w2[wd] & 0xffffu) | (w3[wd] << 16);
                }
                const int r = rb * 8 + j;
                *(uint2*)(lds + lds_off(r, kb >> 1) + (kb & 1) * 8) = make_uint2(lo, hi);
            }
        }
    }
};

template <bool KMAJOR, int ROWS>
struct TileSel;
template <int ROWS>
struct TileSel<true, ROWS> {
    using type = KMajorTile<ROWS>;
};
template <int ROWS>
struct TileSel<false, ROWS> {
    using type = MNMajorTile<ROWS>;
};

__device__ __forceinline__ int xcd_remap(int pid, int n) {
    const int q = n / kXcds, r = n % kXcds;
    const int xcd = pid % kXcds, local = pid / kXcds;
    return xcd < r ? xcd * (q + 1) + local : r * (q + 1) + (xcd - r) * q + local;
}

template <int MODE, bool A_K, bool B_K, int EPI>
__global__ __launch_bounds__(kGemmThreads, 2) void gemm_kernel(GemmArgs p) {
    __shared__ __attribute__((aligned(16))) char smem[2 * (BM + BN) * BK * 2];
    char* const As0 = smem;
    char* const Bs0 = smem + BM * BK * 2;
    constexpr int kBufBytes = (BM + BN) * BK * 2;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int lid = xcd_remap(blockIdx.x, gridDim.x);

    int e = 0, mt, nt;
    int64_t row0, row_hi, k_begin, k_end;
    if (MODE == MODE_ROWS) {
        const int width = kGroupM * p.n_tiles;
        const int group = lid / width;
        const int first_m = group * kGroupM;
        const int gsz = (p.m_tiles - first_m) < kGroupM ? (p.m_tiles - first_m) : kGroupM;
        const int in = lid - group * width;
        mt = first_m + in % gsz;
        nt = in / gsz;
        if (p.offsets != nullptr) {
            if (mt >= p.mtile_start[p.E]) return;
            int lo = 0, hi = p.E;  // last e with mtile_start[e] <= mt
            while (hi - lo > 1) {
                const int mid = (lo + hi) >> 1;
                if (p.mtile_start[mid] <= mt) lo = mid; else hi = mid;
            }
            e = lo;
            row0 = (int64_t)p.offsets[e] + (int64_t)(mt - p.mtile_start[e]) * BM;
            if (row0 < 0 || row0 >= p.R) return;
            int64_t seg_end = p.offsets[e + 1];
            if (seg_end > p.R) seg_end = p.R;
            row_hi = (row0 + BM) < seg_end ? (row0 + BM) : seg_end;
        } else {
            row0 = (int64_t)mt * BM;
            if (row0 >= p.M) return;
            row_hi = (row0 + BM) < p.M ? (row0 + BM) : p.M;
        }
        k_begin = 0;
        k_end = p.Kd;
    } else {
        const int per = p.m_tiles * p.n_tiles;
        e = lid / per;
        const int in = lid - e * per;
        mt = in % p.m_tiles;
        nt = in / p.m_tiles;
        row0 = (int64_t)mt * BM;
        row_hi = (row0 + BM) < p.M ? (row0 + BM) : p.M;
        k_begin = p.offsets[e];
        k_end = p.offsets[e + 1];
        k_begin = k_begin < 0 ? 0 : (k_begin > p.R ? p.R : k_begin);
        k_end = k_end < k_begin ? k_begin : (k_end > p.R ? p.R : k_end);
    }
    const int64_t n0 = (int64_t)nt * BN;
    const uint16_t* Bsrc = p.B + (MODE == MODE_ROWS ? (int64_t)e * p.b_stride : 0);

    typename TileSel<A_K, BM>::type ta;
    typename TileSel<B_K, BN>::type tb;

    f32x4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int64_t klen = k_end - k_begin;
    const int nk = (int)((klen + BK - 1) / BK);

    // Row ranges of the two operand tiles: A rows are activation rows (ROWS)
    // or output rows m (KGRP); B rows are output columns n.
    auto load_tiles = [&](int kt) {
        const int64_t k0 = k_begin + (int64_t)kt * BK;
        if (MODE == MODE_ROWS) {
            ta.load(p.A, p.lda, row0, row_hi, k0, k_end, tid);
        } else {
            ta.load(p.A, p.lda, row0, row_hi, k0, k_end, tid);
        }
        tb.load(Bsrc, p.ldb, n0, (int64_t)p.N, k0, k_end, tid);
    };

    if (nk > 0) {
        load_tiles(0);
        ta.store(As0, tid);
        tb.store(Bs0, tid);
        __syncthreads();
        for (int kt = 0; kt < nk; ++kt) {
            const int cur = kt & 1;
            if (kt + 1 < nk) load_tiles(kt + 1);
            const char* As = As0 + cur * kBufBytes;
            const char* Bs = Bs0 + cur * kBufBytes;
#pragma unroll
            for (int kk = 0; kk < BK / 32; ++kk) {
                const int c = kk * 4 + (lane >> 4);
                bf16x8 af[4], bfg[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int r = wm * 64 + i * 16 + (lane & 15);
                    af[i] = *(const bf16x8*)(As + lds_off(r, c));
                }
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int r = wn * 64 + j * 16 + (lane & 15);
                    bfg[j] = *(const bf16x8*)(Bs + lds_off(r, c));
                }
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bfg[j], af[i], acc[i][j], 0, 0, 0);
            }
            if (kt + 1 < nk) {
                ta.store(As0 + (cur ^ 1) * kBufBytes, tid);
                tb.store(Bs0 + (cur ^ 1) * kBufBytes, tid);
            }
            __syncthreads();
        }
    }

    // Epilogue: lane holds C[m][n .. n+3] for each (i, j).
    const int64_t c_base = (MODE == MODE_KGRP) ? (int64_t)e * p.c_stride : 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t m = row0 + wm * 64 + i * 16 + (lane & 15);
        if (m >= row_hi) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t n = n0 + wn * 64 + j * 16 + 4 * (lane >> 4);
            if (n >= p.N) continue;
            const f32x4 a = acc[i][j];
            const int64_t off = c_base + m * p.ldc + n;
            if (EPI == EPI_F32) {
                *(float4*)((float*)p.C + off) = make_float4(a[0], a[1], a[2], a[3]);
            } else if (EPI == EPI_BF16) {
                *(uint2*)((uint16_t*)p.C + off) = make_uint2(pack_bf16x2(a[0], a[1]), pack_bf16x2(a[2], a[3]));
            } else if (EPI == EPI_RELU2) {
                const float r0 = fmaxf(a[0], 0.f), r1 = fmaxf(a[1], 0.f);
                const float r2 = fmaxf(a[2], 0.f), r3 = fmaxf(a[3], 0.f);
                *(uint2*)((uint16_t*)p.C + off) =
                    make_uint2(pack_bf16x2(r0 * r0, r1 * r1), pack_bf16x2(r2 * r2, r3 * r3));
                if (p.aux_out != nullptr)
                    *(uint2*)(p.aux_out + off) = make_uint2(pack_bf16x2(a[0], a[1]), pack_bf16x2(a[2], a[3]));
            } else {  // EPI_DRELU2
                const uint2 u = *(const uint2*)(p.aux_in + off);
                const float g0 = a[0] * 2.f * fmaxf(bf16_lo(u.x), 0.f);
                const float g1 = a[1] * 2.f * fmaxf(bf16_hi(u.x), 0.f);
                const float g2 = a[2] * 2.f * fmaxf(bf16_lo(u.y), 0.f);
                const float g3 = a[3] * 2.f * fmaxf(bf16_hi(u.y), 0.f);
                *(uint2*)((uint16_t*)p.C + off) = make_uint2(pack_bf16x2(g0, g1), pack_bf16x2(g2, g3));
            }
        }
    }
}

// mtile_start[0] = 0, mtile_start[e+1] = sum_{e' <= e} ceil(count[e'] / BM).
__global__ __launch_bounds__(1024) void tile_schedule_kernel(const int32_t* __restrict__ offsets, int E,
                                                              int32_t* __restrict__ mtile_start) {
    __shared__ int32_t s[1024];
    const int tid = threadIdx.x;
    s[tid] = tid < E ? (offsets[tid + 1] - offsets[tid] + BM - 1) / BM : 0;
    __syncthreads();
    for (int d = 1; d < 1024; d <<= 1) {
        const int add = tid >= d ? s[tid - d] : 0;
        __syncthreads();
        s[tid] += add;
        __syncthreads();
    }
    if (tid < E) mtile_start[tid + 1] = s[tid];
    if (tid == 0) mtile_start[0] = 0;
}

int gemm_tile_m() { return BM; }

size_t gemm_schedule_bytes(int E) { return (size_t)((E + 1) * 4 + 255) / 256 * 256; }

static int64_t mtiles_bound(int64_t R, int E) {
    // sum_e ceil(c_e / BM) <= ceil(R / BM) + (number of non-empty experts)
    const int64_t nonempty = R < E ? R : E;
    return (R + BM - 1) / BM + nonempty;
}

template <int MODE, bool A_K, bool B_K, int EPI>
static hipError_t launch(const GemmArgs& a, int64_t n_wg, hipStream_t st) {
    if (n_wg <= 0) return hipSuccess;
    if (n_wg > 0x7fffffff) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((gemm_kernel<MODE, A_K, B_K, EPI>), dim3((unsigned)n_wg), dim3(kGemmThreads), 0,
                       st, a);
    return hipGetLastError();
}

hipError_t launch_tile_schedule(const int32_t* offsets, int E, int32_t* mtile_start, hipStream_t st) {
    hipLaunchKernelGGL(tile_schedule_kernel, dim3(1), dim3(1024), 0, st, offsets, E, mtile_start);
    return hipGetLastError();
}

hipError_t launch_grouped_rows(const moe_bf16* A, int64_t lda, const moe_bf16* B, int64_t ldb,
                               int64_t b_stride, bool b_kmajor, void* C, int64_t ldc, int epi,
                               const moe_bf16* aux_in, moe_bf16* aux_out, const int32_t* offsets,
                               const int32_t* mtile_start, int E, int64_t R, int N, int Kd,
                               hipStream_t st) {
    GemmArgs a{};
    a.A = A; a.B = B; a.C = C; a.aux_in = aux_in; a.aux_out = aux_out;
    a.offsets = offsets; a.mtile_start = mtile_start;
    a.lda = lda; a.ldb = ldb; a.ldc = ldc; a.b_stride = b_stride;
    a.M = R; a.R = R; a.N = N; a.Kd = Kd; a.E = E;
    a.n_tiles = (N + BN - 1) / BN;
    a.m_tiles = (int)(offsets ? mtiles_bound(R, E) : (R + BM - 1) / BM);
    const int64_t n_wg = (int64_t)a.m_tiles * a.n_tiles;
    if (R == 0) return hipSuccess;
    if (!b_kmajor) {
        if (epi == EPI_BF16) return launch<MODE_ROWS, true, false, EPI_BF16>(a, n_wg, st);
        if (epi == EPI_RELU2) return launch<MODE_ROWS, true, false, EPI_RELU2>(a, n_wg, st);
    } else {
        if (epi == EPI_BF16) return launch<MODE_ROWS, true, true, EPI_BF16>(a, n_wg, st);
        if (epi == EPI_DRELU2) return launch<MODE_ROWS, true, true, EPI_DRELU2>(a, n_wg, st);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_grouped_wgrad(const moe_bf16* A, int64_t lda, const moe_bf16* B, int64_t ldb,
                                float* C, int64_t ldc, int64_t c_stride, const int32_t* offsets,
                                int E, int M, int N, int64_t R, hipStream_t st) {
    GemmArgs a{};
    a.A = A; a.B = B; a.C = C; a.offsets = offsets;
    a.lda = lda; a.ldb = ldb; a.ldc = ldc; a.c_stride = c_stride;
    a.M = M; a.R = R; a.N = N; a.E = E;
    a.m_tiles = (M + BM - 1) / BM;
    a.n_tiles = (N + BN - 1) / BN;
    const int64_t n_wg = (int64_t)E * a.m_tiles * a.n_tiles;
    return launch<MODE_KGRP, false, false, EPI_F32>(a, n_wg, st);
}

}  // namespace moe
