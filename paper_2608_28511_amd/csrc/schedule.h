// Device-side tile schedules of the grouped GEMM (internal to the library).
//
// For expert segments offsets[0..E] (clamped to [0, R)) and each tile height
// BM in {128, 256}:
//   mtile_start[0] = 0, mtile_start[e+1] = min(sum_{e' <= e} ceil(count[e'] / BM), max_tiles)
//   tiles[mt] = {e, row0, row_end, 16 * g0 + gs} for every BM-row tile mt of
//               expert e, {-1, 0, 0, 0} for mt in [total, max_tiles) (the
//               static grid bound).  g0 and gs place mt in its group: an
//               expert's m-tiles are cut, from its first, into runs of at
//               most kSchedGroupM; mt's run is [g0, g0 + gs).  The GEMM walks
//               each run across all n-tiles before the next, so the workgroups
//               of an XCD that run together share one expert's weight panels
//               and row tiles in its L2.
// Routing offsets are monotone, so the tile count never exceeds max_tiles;
// malformed offsets (segments that overlap after clamping) could ask for
// more, and the cap keeps every reader of the table inside it.
// The buffer holds the 128-row part, then the 256-row part; each part is
// mtile_start [E+1] int32, then (16-byte aligned) the tile table, and is
// 256-byte aligned.  The tables are built either by one workgroup of any
// size (a multiple of 64 threads: its own launch, or an extra workgroup of a
// launch that runs after the routing), or a slice per workgroup by several
// workgroups that each hold the segment bounds (sched_fill_slice).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moe {

constexpr int kSchedBM[2] = {128, 256};
constexpr int kSchedGroupM = 8;   // m-tiles per run of one expert

struct SchedPart {
    int32_t* mtile_start;
    int4* tiles;
    int max_tiles;
};

// sum_e ceil(c_e / BM) <= ceil(R / BM) + (number of non-empty experts)
inline int64_t mtiles_bound(int64_t R, int E, int BMr) {
    const int64_t nonempty = R < E ? R : E;
    return (R + BMr - 1) / BMr + nonempty;
}
inline size_t sched_table_offset(int E) { return (size_t)((E + 1) * 4 + 15) / 16 * 16; }
inline size_t sched_part_bytes(int E, int64_t R, int BMr) {
    return (sched_table_offset(E) + (size_t)mtiles_bound(R, E, BMr) * 16 + 255) / 256 * 256;
}
inline SchedPart sched_part(void* sched, int E, int64_t R, bool large) {
    char* base = (char*)sched + (large ? sched_part_bytes(E, R, kSchedBM[0]) : 0);
    return SchedPart{(int32_t*)base, (int4*)(base + sched_table_offset(E)),
                     (int)mtiles_bound(R, E, kSchedBM[large ? 1 : 0])};
}

// One tile height's tables from the segments in LDS; cnt is LDS scratch of E
// entries.  Every thread of the workgroup calls it.
__device__ __forceinline__ void sched_fill_part(const int32_t* seg_lo, const int32_t* seg_hi, int32_t* cnt,
                                                int E, int BMr, const SchedPart& sp) {
    const int tid = threadIdx.x, nt = blockDim.x;
    for (int e = tid; e < E; e += nt) cnt[e] = (seg_hi[e] - seg_lo[e] + BMr - 1) / BMr;
    __syncthreads();
    if (tid < 64) {   // the first wave: inclusive scan over E in 64 contiguous chunks
        const int per = (E + 63) / 64;
        const int e0 = tid * per, e1 = e0 + per < E ? e0 + per : E;
        int local = 0;
        for (int e = e0; e < e1; ++e) local += cnt[e];
        int incl = local;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int o = __shfl_up(incl, d);
            if (tid >= d) incl += o;
        }
        int run = incl - local;
        for (int e = e0; e < e1; ++e) {
            run += cnt[e];
            cnt[e] = run;
        }
    }
    __syncthreads();
    for (int e = tid; e < E; e += nt) sp.mtile_start[e + 1] = cnt[e] < sp.max_tiles ? cnt[e] : sp.max_tiles;
    if (tid == 0) sp.mtile_start[0] = 0;
    const int total = cnt[E - 1] < sp.max_tiles ? cnt[E - 1] : sp.max_tiles;
    for (int mt = tid; mt < sp.max_tiles; mt += nt) {
        int4 v = make_int4(-1, 0, 0, 0);
        if (mt < total) {
            int a = 0, b = E - 1;  // first e with cnt[e] > mt
            while (a < b) {
                const int m = (a + b) >> 1;
                if (cnt[m] > mt) b = m; else a = m + 1;
            }
            const int first = a ? cnt[a - 1] : 0;
            const int row0 = seg_lo[a] + (mt - first) * BMr;
            const int row_end = row0 + BMr < seg_hi[a] ? row0 + BMr : seg_hi[a];
            const int g0 = first + (mt - first) / kSchedGroupM * kSchedGroupM;
            const int gs = cnt[a] - g0 < kSchedGroupM ? cnt[a] - g0 : kSchedGroupM;
            v = make_int4(a, row0, row_end, 16 * g0 + gs);
        }
        sp.tiles[mt] = v;
    }
    __syncthreads();   // cnt is reused by the next part
}

// Entries [mt0, mt1) of one tile height's table (and, with starts, its
// mtile_start array) from segments seg_lo / seg_hi and the inclusive prefix
// sums incl[e] of their tile counts, all in LDS: lets every workgroup of a
// launch write its own slice.
__device__ __forceinline__ void sched_fill_slice(const int32_t* seg_lo, const int32_t* seg_hi, const int32_t* incl,
                                                 int E, int BMr, const SchedPart& sp, int mt0, int mt1,
                                                 bool starts) {
    const int tid = threadIdx.x, nt = blockDim.x;
    if (starts) {
        for (int e = tid; e < E; e += nt) sp.mtile_start[e + 1] = incl[e] < sp.max_tiles ? incl[e] : sp.max_tiles;
        if (tid == 0) sp.mtile_start[0] = 0;
    }
    const int total = incl[E - 1] < sp.max_tiles ? incl[E - 1] : sp.max_tiles;
    mt1 = mt1 < sp.max_tiles ? mt1 : sp.max_tiles;
    for (int mt = mt0 + tid; mt < mt1; mt += nt) {
        int4 v = make_int4(-1, 0, 0, 0);
        if (mt < total) {
            int a = 0, b = E - 1;  // first e with incl[e] > mt
            while (a < b) {
                const int m = (a + b) >> 1;
                if (incl[m] > mt) b = m; else a = m + 1;
            }
            const int first = a ? incl[a - 1] : 0;
            const int row0 = seg_lo[a] + (mt - first) * BMr;
            const int row_end = row0 + BMr < seg_hi[a] ? row0 + BMr : seg_hi[a];
            const int g0 = first + (mt - first) / kSchedGroupM * kSchedGroupM;
            const int gs = incl[a] - g0 < kSchedGroupM ? incl[a] - g0 : kSchedGroupM;
            v = make_int4(a, row0, row_end, 16 * g0 + gs);
        }
        sp.tiles[mt] = v;
    }
}

// Both tile heights' tables for segments offsets[0..E] (1 <= E <= 1024).
__device__ __forceinline__ void build_tile_schedule(const int32_t* __restrict__ offsets, int E, int R,
                                                    const SchedPart& small, const SchedPart& large) {
    __shared__ int32_t seg_lo[1024], seg_hi[1024], cnt[1024];
    for (int e = threadIdx.x; e < E; e += blockDim.x) {
        int lo = offsets[e], hi = offsets[e + 1];
        lo = lo < 0 ? 0 : (lo > R ? R : lo);
        hi = hi < lo ? lo : (hi > R ? R : hi);
        seg_lo[e] = lo;
        seg_hi[e] = hi;
    }
    __syncthreads();
    sched_fill_part(seg_lo, seg_hi, cnt, E, kSchedBM[0], small);
    sched_fill_part(seg_lo, seg_hi, cnt, E, kSchedBM[1], large);
}

}  // namespace moe
