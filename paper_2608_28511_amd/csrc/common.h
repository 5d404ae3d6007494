// Internal helpers shared by the gfx950 kernels of the MoE layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "moe.h"

namespace moe {

constexpr int kWave = 64;  // CDNA wavefront width

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
    return __uint_as_float(bits16 << 16);
}

// Low / high bf16 of a packed dword as fp32.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16 bits, round to nearest even (gfx950 converts in hardware).
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
    __bf16 b = (__bf16)f;
    return (uint32_t)__builtin_bit_cast(uint16_t, b);
}

// 16-byte load with the non-temporal hint, for rows that are read once:
// under a cold last-level cache it lets a gather or a row copy stream from HBM
// near the copy ceiling (measured on the 256-expert layer's combine: 4.95 TB/s
// against 2.86 TB/s with plain loads).
__device__ __forceinline__ uint4 ld_nt(const uint4* p) {
    const u32x4 q = __builtin_nontemporal_load((const u32x4*)p);
    return make_uint4(q[0], q[1], q[2], q[3]);
}

// Two fp32 -> one dword holding (lo, hi) bf16, both rounded to nearest even
// by one v_cvt_pk_bf16_f32 (converting them one at a time costs a shift and
// an or per pair on top of two conversions).
typedef __bf16 bf16x2_cvt __attribute__((ext_vector_type(2)));
typedef float f32x2_cvt __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_cvt){lo, hi}, bf16x2_cvt));
}

// max(x, 0) as one integer max of the bit pattern: every negative value and
// -0 map to +0, non-negative values pass unchanged (a NaN with the sign bit
// clear passes too).  fmaxf costs a NaN-quieting max on top.
__device__ __forceinline__ float relu_f32(float x) { return __int_as_float(max(__float_as_int(x), 0)); }

// MOE_DEBUG_SYNC=1 in the environment (read once per process).
bool debug_sync_enabled();

// Status of the launches just enqueued on st: the launch error, and with
// MOE_DEBUG_SYNC also the outcome of running them (the stream is
// synchronised, so a fault surfaces at the entry point that enqueued it).
// A stream that is being captured into a graph is never synchronised.
inline hipError_t launch_check(hipStream_t st) {
    hipError_t e = hipGetLastError();
    if (e == hipSuccess && debug_sync_enabled()) {
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        if (hipStreamIsCapturing(st, &cs) != hipSuccess) {
            (void)hipGetLastError();   // e.g. the null stream under a global capture: do not synchronise
            return hipSuccess;
        }
        if (cs == hipStreamCaptureStatusNone) {
            e = hipStreamSynchronize(st);
            if (e == hipSuccess) e = hipGetLastError();
        }
    }
    return e;
}

// Sizes handed to every launch: grid dimension from an element count.
inline unsigned grid_for(int64_t n, int per_block) {
    return (unsigned)((n + per_block - 1) / per_block);
}

}  // namespace moe
