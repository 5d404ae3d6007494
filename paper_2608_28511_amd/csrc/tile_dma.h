// Building blocks shared by the gfx950 MFMA kernels (grouped GEMM, router
// logits): the direct global -> LDS copy ring, the LDS operand layouts and
// their MFMA fragment reads.
//
// A workgroup has kWaves = 8 wavefronts and contracts BK = 64 elements per
// ring stage.  An operand tile lives in LDS in one of two layouts:
//   row layout  [rows][64 k], from a K-contiguous source, fragments read with
//               ds_read_b128;
//   col layout  [64 k][cols], from an M/N-contiguous source, fragments read
//               with the gfx950 LDS transpose read ds_read_b64_tr_b16.
#pragma once

#include "common.h"

namespace moe {

constexpr int BK = 64;
constexpr int kWaves = 8;
constexpr int kXcds = 8;

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef short v8i16 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
typedef __attribute__((address_space(3))) char lds_char;

// One zero chunk: the source of every out-of-range DMA lane.
static __device__ __attribute__((aligned(16))) uint4 g_zero_chunk[1];

// ---- row layout: [rows][64 k], 8 chunks per row; chunk c of row r stored at
// c ^ (r & 7).  The fragments of rows r and r + 16 then sit a constant 2 KB
// apart (an immediate offset).  A ds_read_b128 of 16 consecutive rows is
// conflict-free with this swizzle: rows r and r + 8 (1 KB apart) already fall
// in different banks on gfx950, and XOR-ing r >> 3 into the chunk as well
// measured as a 2-way conflict (LDS bank-conflict counter, 16-row fragment
// read pattern).
__device__ __forceinline__ int rswz(int r) { return r & 7; }

// ---- col layout: [64 k][cols], cols/8 chunks per k-row; chunk pairs XOR-swizzled
// so the 8 rows {k..k+3, k+8..k+11} read together by ds_read_b64_tr_b16 hit
// distinct 32-byte bank groups.  cswz depends on k mod 16 only, so rows k + 4
// and k + 32 sit constant offsets away.
__device__ __forceinline__ int cswz(int k) { return 2 * ((k & 3) | (((k >> 3) & 1) << 2)); }

// 16-byte global -> LDS copy for the whole wave: lane l's chunk lands at LDS
// byte lds_addr + 16*l (lds_addr wave-uniform).  Issued as inline assembly so
// that the compiler does not treat it as an LDS write that every later LDS
// read must wait for; the kernel orders it with explicit vmcnt waits and
// barriers instead.
__device__ __forceinline__ void dma16(const void* g, uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 :
                 : "v"(g), "s"(lds_addr)
                 : "memory", "m0");
}

// Workgroup barrier without the memory fence of __syncthreads (whose release
// fence would drain every in-flight DMA stage).  Callers wait for their own
// DMA stage with wait_vmcnt first; every LDS read of the previous stage has
// been consumed by an MFMA before a wave can arrive here.
__device__ __forceinline__ void stage_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    if constexpr (N == 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    else if constexpr (N == 4) asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
    else if constexpr (N == 6) asm volatile("s_waitcnt vmcnt(6)" ::: "memory");
    else if constexpr (N == 8) asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
    else static_assert(N == 0, "unsupported vmcnt");
}

// Per-lane DMA slots of one operand tile.  Slot i of a wave covers LDS bytes
// [(wave*kSlots + i)*1024, +1024) of the tile; each lane's 16-byte chunk has a
// fixed global row / column for the whole k loop, so its pointer advances by
// one k tile per stage (by zero for chunks outside the operand, which keep
// pointing at the zero chunk).  Only a tile that crosses the end of the
// contraction re-checks the k coordinate.
//
// Row layout (K-contiguous source, element (r, k) at src[r*ld + k]).
// Col layout (M/N-contiguous source, element (k, c) at src[k*ld + c]).
template <bool ROWL, int EXT>
struct DmaTile {
    static constexpr int kCPR = ROWL ? 8 : EXT / 8;       // chunks per LDS row
    static constexpr int kSlots = EXT * 8 / 64 / kWaves;  // 1 KB slots per wave
    const uint16_t* ptr[kSlots];
    int64_t step[kSlots];
    int kpos[kSlots];      // k offset of the chunk inside the tile
    bool ok[kSlots];

    __device__ __forceinline__ void init(const uint16_t* __restrict__ src, int64_t ld, int64_t x0,
                                         int64_t x_hi, int64_t k_begin, int wave, int lane) {
#pragma unroll
        for (int i = 0; i < kSlots; ++i) {
            const int p = (wave * kSlots + i) * 64 + lane;
            const int row = p / kCPR;
            int c = p % kCPR;
            if (ROWL) {
                c ^= rswz(row);
                ok[i] = x0 + row < x_hi;
                kpos[i] = c * 8;
                ptr[i] = ok[i] ? src + (x0 + row) * ld + k_begin + c * 8 : (const uint16_t*)g_zero_chunk;
                step[i] = ok[i] ? (int64_t)BK : 0;
            } else {
                c ^= cswz(row);
                ok[i] = x0 + c * 8 < x_hi;
                kpos[i] = row;
                ptr[i] = ok[i] ? src + (k_begin + row) * ld + x0 + c * 8 : (const uint16_t*)g_zero_chunk;
                step[i] = ok[i] ? (int64_t)BK * ld : 0;
            }
        }
    }
    // Issue this wave's slots [I0, I1) of the next tile in k order, then
    // advance.  KTAIL: the contraction length may end inside a tile, so chunks
    // at or past k_rem are replaced by the zero chunk.
    template <bool KTAIL, int I0, int I1>
    __device__ __forceinline__ void issue(uint32_t tile_lds, int64_t k_rem, int wave) {
#pragma unroll
        for (int i = I0; i < I1; ++i) {
            const uint32_t dst = tile_lds + (uint32_t)(wave * kSlots + i) * 1024u;
            if constexpr (KTAIL)
                dma16(kpos[i] < k_rem ? (const void*)ptr[i] : (const void*)g_zero_chunk, dst);
            else
                dma16(ptr[i], dst);
            ptr[i] += step[i];
        }
    }
};

// Fragment addressing.  A fragment is 16 rows x 8 k per lane group; the lane
// base offsets below are computed once, everything else is an immediate.
//
// Row layout: lane reads row (row0 + lane%16), chunk (4*kk + lane/16) ^ rswz.
__device__ __forceinline__ uint32_t row_base(int row0, int kk, int lane) {
    const int r = row0 + (lane & 15);
    const int c = kk * 4 + (lane >> 4);
    return (uint32_t)((r * 8 + (c ^ rswz(r))) * 16);
}
// Col layout: lane 16g + 4r + q points at k-row 8g + r (+32 kk, +4 for the
// second read), columns col0 + 4q .. +3; each 16-lane group then receives one
// column each from ds_read_b64_tr_b16.
template <int COLS>
__device__ __forceinline__ uint32_t col_base(int col0, int lane) {
    constexpr int kCPR = COLS / 8;
    const int g = lane >> 4, rq = (lane >> 2) & 3, q = lane & 3;
    const int k = g * 8 + rq;
    const int c = (col0 >> 3) + (q >> 1);
    return (uint32_t)((k * kCPR + (c ^ cswz(k))) * 16 + (q & 1) * 8);
}

typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;

__device__ __forceinline__ bf16x8 lds_b128(uint32_t addr) { return *(const lds_bf16x8*)(uintptr_t)addr; }

__device__ __forceinline__ bf16x8 lds_tr_pair(uint32_t addr, uint32_t hi_off) {
    const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(uintptr_t)addr);
    const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(uintptr_t)(addr + hi_off));
    const v8i16 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8, v);
}

__device__ __forceinline__ int xcd_remap(int pid, int n) {
    const int q = n / kXcds, r = n % kXcds;
    const int xcd = pid % kXcds, local = pid / kXcds;
    return xcd < r ? xcd * (q + 1) + local : r * (q + 1) + (xcd - r) * q + local;
}


}  // namespace moe
