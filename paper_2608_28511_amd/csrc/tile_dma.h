// Building blocks shared by the gfx950 MFMA kernels (grouped GEMM, router
// logits): the direct global -> LDS copy ring, the LDS operand layouts and
// their MFMA fragment reads.
//
// A workgroup has kWaves = 8 wavefronts and contracts KD = 64 (default) or 32
// elements per ring stage.  An operand tile lives in LDS in one of two layouts:
//   row layout  [rows][KD k], from a K-contiguous source, fragments read with
//               ds_read_b128;
//   col layout  [KD k][cols], from an M/N-contiguous source, fragments read
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

typedef int i32x4 __attribute__((ext_vector_type(4)));

// ---- row layout: [rows][64 k], 8 chunks per row; chunk c of row r stored at
// c ^ (r & 7).  The fragments of rows r and r + 16 then sit a constant 2 KB
// apart (an immediate offset).  A ds_read_b128 of 16 consecutive rows is
// conflict-free with this swizzle: rows r and r + 8 (1 KB apart) already fall
// in different banks on gfx950, and XOR-ing r >> 3 into the chunk as well
// measured as a 2-way conflict (LDS bank-conflict counter, 16-row fragment
// read pattern).
__device__ __forceinline__ int rswz(int r) { return r & 7; }
// For 32 k per row (64-byte rows, 4 chunks) the conflict-free swizzle of the
// same 16-row fragment read is chunk c of row r at c ^ ((r >> 1) & 3): the
// eight 16-byte reads of rows r .. r+1 and r+8 .. r+9 land in distinct bank
// groups (measured with the LDS bank-conflict counter).
template <int KD>
__device__ __forceinline__ int rswz_k(int r) { return KD == 64 ? (r & 7) : ((r >> 1) & 3); }

// ---- fp8 row layout: [rows][KDB bytes] of MX-FP8 codes (KDB = 64 or 32:
// 4 or 2 chunks of 16 codes); a lane's fragment is 8 codes, read with
// ds_read_b64.  Chunk c of row r is stored at c ^ mxswz<KDB>(r), so that the
// 16 rows x 2 eight-byte pieces each half-wave reads fall in distinct banks.
template <int KDB>
__device__ __forceinline__ int mxswz(int r) { return KDB == 64 ? ((r >> 2) & 3) : ((r >> 3) & 1); }

// ---- col layout: [64 k][cols], cols/8 chunks per k-row; chunk pairs XOR-swizzled
// so the 8 rows {k..k+3, k+8..k+11} read together by ds_read_b64_tr_b16 hit
// distinct 32-byte bank groups.  cswz depends on k mod 16 only, so rows k + 4
// and k + 32 sit constant offsets away.
__device__ __forceinline__ int cswz(int k) { return 2 * ((k & 3) | (((k >> 3) & 1) << 2)); }

// Range-checked buffer descriptor over [base, base + bytes): every access at
// or past `bytes` reads as zero without touching memory.  bytes < 2^31.
__device__ __forceinline__ i32x4 buf_rsrc(const void* base, uint32_t bytes) {
    const uint64_t a = (uint64_t)(uintptr_t)base;
    return i32x4{(int)(uint32_t)a, (int)((uint32_t)(a >> 32) & 0xffffu), (int)bytes, 0x00020000};
}

// An offset beyond every descriptor's range, with room to advance by a whole
// operand (< 2^31 bytes) without wrapping.
constexpr uint32_t kDmaDrop = 0x80000000u;
constexpr int64_t kMaxDmaBytes = (int64_t)1 << 31;  // descriptor ranges stay below this

// 16-byte buffer -> LDS copy for the whole wave: lane l's chunk (byte offset
// `off` in the descriptor's range, zero if outside it) lands at LDS byte
// lds_addr + 16*l (lds_addr wave-uniform).  Issued as inline assembly so
// that the compiler does not treat it as an LDS write that every later LDS
// read must wait for; the kernels order it with explicit vmcnt waits and
// barriers instead.
__device__ __forceinline__ void dma16(const i32x4& rs, uint32_t off, uint32_t lds_addr) {
    // descriptor and LDS base are wave-uniform: pin them to scalar registers
    const i32x4 srs = {__builtin_amdgcn_readfirstlane(rs[0]), __builtin_amdgcn_readfirstlane(rs[1]),
                       __builtin_amdgcn_readfirstlane(rs[2]), __builtin_amdgcn_readfirstlane(rs[3])};
    const uint32_t sdst = __builtin_amdgcn_readfirstlane(lds_addr);
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
                 :
                 : "v"(off), "s"(srs), "s"(sdst)
                 : "memory", "m0");
}

// 4-byte buffer -> LDS copy for the whole wave: lane l's dword lands at
// lds_addr + 4*l (same ordering rules as dma16).
__device__ __forceinline__ void dma4(const i32x4& rs, uint32_t off, uint32_t lds_addr) {
    const i32x4 srs = {__builtin_amdgcn_readfirstlane(rs[0]), __builtin_amdgcn_readfirstlane(rs[1]),
                       __builtin_amdgcn_readfirstlane(rs[2]), __builtin_amdgcn_readfirstlane(rs[3])};
    const uint32_t sdst = __builtin_amdgcn_readfirstlane(lds_addr);
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dword %0, %1, 0 offen lds"
                 :
                 : "v"(off), "s"(srs), "s"(sdst)
                 : "memory", "m0");
}

// Workgroup barrier without the memory fence of __syncthreads (whose release
// fence would drain every in-flight DMA stage).  Callers wait for their own
// DMA stage with wait_vmcnt first; every LDS read of the previous stage has
// been consumed by an MFMA before a wave can arrive here.
__device__ __forceinline__ void stage_barrier() {
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0), visible to the compiler's wait tracking
    asm volatile("s_barrier" ::: "memory");
}

// Wait until at most N vector-memory operations of this wave are in flight
// (an immediate operand: N < 64).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt out of range");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Per-lane DMA slots of one operand tile.  Slot i of a wave covers LDS bytes
// [(wave*kSlots + i)*1024, +1024) of the tile; each lane's 16-byte chunk has a
// fixed row / column for the whole k loop, so its byte offset advances by one
// k tile per stage.  The descriptor spans only the tile's part of the operand,
// so chunks past its rows (ragged expert segments, the end of the contraction
// for the column layout) read as zero; chunks past its columns start at
// kDmaDrop.
//
// Row layout (K-contiguous source, element (r, k) at src[r*ld + k]): rows
//   [x0, min(x_hi, x0 + EXT)), k from k_begin.  A contraction that ends inside
//   a k tile (KTAIL) is cut per chunk at issue time.  SW = 1: the fp8 row
//   swizzle (rows of 2*KD code bytes) instead of the bf16 one.
// Col layout (M/N-contiguous source, element (k, c) at src[k*ld + c]): k rows
//   [k_begin, k_end), columns [x0, x_hi).
template <bool ROWL, int EXT, int KD = BK, int WAVES = kWaves, int SW = 0>
struct DmaTile {
    static constexpr int kCPR = ROWL ? KD / 8 : EXT / 8;       // chunks per LDS row
    static constexpr int kSlots = EXT * KD * 2 / 1024 / WAVES;  // 1 KB slots per wave
    static_assert(kSlots * WAVES * 1024 == EXT * KD * 2, "the tile must split into whole slots per wave");
    i32x4 rs;                // wave-uniform
    uint32_t kstep;          // bytes per k tile, wave-uniform
    uint32_t off[kSlots];
    int kpos[kSlots];        // row layout: k offset of the chunk inside the tile

    __device__ __forceinline__ void init(const uint16_t* __restrict__ src, int64_t ld, int64_t x0,
                                         int64_t x_hi, int64_t k_begin, int64_t k_end, int wave, int lane) {
        if (ROWL) {
            const int64_t x_end = (x0 + EXT) < x_hi ? (x0 + EXT) : x_hi;
            const int64_t rows = x_end > x0 ? x_end - x0 : 0;
            rs = buf_rsrc(src + x0 * ld + k_begin, (uint32_t)(rows * ld * 2));
            kstep = KD * 2;
        } else {
            const int64_t krows = k_end > k_begin ? k_end - k_begin : 0;
            rs = buf_rsrc(src + k_begin * ld + x0, (uint32_t)(krows > 0 ? krows * ld * 2 - x0 * 2 : 0));
            kstep = (uint32_t)(KD * ld * 2);
        }
#pragma unroll
        for (int i = 0; i < kSlots; ++i) {
            const int p = (wave * kSlots + i) * 64 + lane;
            const int row = p / kCPR;
            int c = p % kCPR;
            if (ROWL) {
                c ^= SW ? mxswz<KD * 2>(row) : rswz_k<KD>(row);
                kpos[i] = c * 8;
                off[i] = (uint32_t)((row * ld + c * 8) * 2);
            } else {
                c ^= cswz(row);
                kpos[i] = row;
                off[i] = x0 + c * 8 < x_hi ? (uint32_t)((row * ld + c * 8) * 2) : kDmaDrop;
            }
        }
    }
    // Row layout with gathered rows (the permutation fused into the copy):
    // tile row r of [x0, x_hi) is source row rows_idx[x0 + r] / div of a
    // K-contiguous source of src_rows rows (the token of routed row x0 + r),
    // k from 0; rows past x_hi, or whose index is out of range, read as zero.
    // The descriptor spans the whole source (src_rows * ld * 2 < 2^31).
    __device__ __forceinline__ void init_gather(const uint16_t* __restrict__ src, int64_t ld,
                                                const int32_t* __restrict__ rows_idx, int div, int64_t src_rows,
                                                int64_t x0, int64_t x_hi, int wave, int lane) {
        static_assert(ROWL, "gathered rows need the row layout");
        rs = buf_rsrc(src, (uint32_t)(src_rows * ld * 2));
        kstep = KD * 2;
#pragma unroll
        for (int i = 0; i < kSlots; ++i) {
            const int p = (wave * kSlots + i) * 64 + lane;
            const int row = p / kCPR;
            const int c = (p % kCPR) ^ (SW ? mxswz<KD * 2>(row) : rswz_k<KD>(row));
            kpos[i] = c * 8;
            off[i] = kDmaDrop;
            if (x0 + row < x_hi) {
                const int tok = rows_idx[x0 + row] / div;
                if (tok >= 0 && tok < src_rows) off[i] = (uint32_t)((tok * ld + c * 8) * 2);
            }
        }
    }
    // Issue this wave's slots [I0, I1) of the next tile in k order, then
    // advance.  KTAIL (row layout): chunks at or past k_rem, the contraction
    // left from this tile's start, read as zero.
    template <bool KTAIL, int I0, int I1>
    __device__ __forceinline__ void issue(uint32_t tile_lds, int64_t k_rem, int wave) {
#pragma unroll
        for (int i = I0; i < I1; ++i) {
            const uint32_t dst = tile_lds + (uint32_t)(wave * kSlots + i) * 1024u;
            uint32_t o = off[i];
            if constexpr (KTAIL && ROWL) o = kpos[i] < k_rem ? o : kDmaDrop;
            dma16(rs, o, dst);
            off[i] += kstep;
        }
    }
};

// Fragment addressing.  A fragment is 16 rows x 8 k per lane group; the lane
// base offsets below are computed once, everything else is an immediate.
//
// Row layout: lane reads row (row0 + lane%16), chunk (4*kk + lane/16) ^ rswz.
template <int KD = BK>
__device__ __forceinline__ uint32_t row_base(int row0, int kk, int lane) {
    const int r = row0 + (lane & 15);
    const int c = kk * 4 + (lane >> 4);
    return (uint32_t)((r * (KD / 8) + (c ^ rswz_k<KD>(r))) * 16);
}
// fp8 row layout: lane reads row (row0 + lane%16), codes
// [32*kk + 8*(lane/16), +8) of a KDB-byte row.
template <int KDB>
__device__ __forceinline__ uint32_t mx_row_base(int row0, int kk, int lane) {
    const int r = row0 + (lane & 15);
    const int g = kk * 4 + (lane >> 4);   // 8-byte piece of the row
    return (uint32_t)(r * KDB + (((g >> 1) ^ mxswz<KDB>(r)) * 16) + (g & 1) * 8);
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
