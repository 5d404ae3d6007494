// Host side of the C ABI in include/moe.h: synchronous argument validation,
// workspace sizing and carving, and stream-ordered launch of the kernels.
// Nothing here allocates, frees or synchronises device memory.
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>

#include <hip/hip_runtime_api.h>

#include "moe.h"
#include "kernels.h"

namespace {

constexpr int kMaxE = 1024;
constexpr int kMaxK = 32;
constexpr int kMaxDim = 65536;
constexpr int64_t kMaxRows = (int64_t)1 << 31;

bool misaligned(const void* p, size_t a) { return ((uintptr_t)p) % a != 0; }

// A pointer that must address `bytes` bytes: NULL is allowed only for an empty range.
int need(const void* p, uint64_t bytes, size_t align) {
    if (bytes == 0) return MOE_OK;
    if (p == nullptr) return MOE_ERR_NULL;
    if (misaligned(p, align)) return MOE_ERR_ALIGN;
    return MOE_OK;
}

int opt(const void* p, size_t align) {
    if (p != nullptr && misaligned(p, align)) return MOE_ERR_ALIGN;
    return MOE_OK;
}

bool dim_ok(int32_t d) { return d >= 8 && d <= kMaxDim && d % 8 == 0; }

// The grouped GEMM copies operands through buffer descriptors whose range is
// below 2^31 bytes: one expert's (or the dense) [Kd, N] bf16 weight, and for
// the weight gradients each operand's rows.
constexpr int64_t kMaxOperandBytes = (int64_t)1 << 31;
bool weight_ok(int64_t kd, int64_t n) { return kd * n * 2 < kMaxOperandBytes; }

int check_route_shape(int64_t S, int32_t E, int32_t K) {
    if (S < 0) return MOE_ERR_SHAPE;
    if (E < 1 || E > kMaxE) return MOE_ERR_SHAPE;
    if (K < 1 || K > E || K > kMaxK) return MOE_ERR_SHAPE;
    if (S * (int64_t)K >= kMaxRows) return MOE_ERR_SHAPE;
    return MOE_OK;
}

int hip_status(hipError_t e) { return e == hipSuccess ? MOE_OK : MOE_ERR_HIP; }

size_t align256(size_t b) { return (b + 255) / 256 * 256; }

#define MOE_TRY(expr)                 \
    do {                              \
        const int _s = (expr);        \
        if (_s != MOE_OK) return _s;  \
    } while (0)

#define MOE_HIP(expr)                           \
    do {                                        \
        const hipError_t _e = (expr);           \
        if (_e != hipSuccess) return MOE_ERR_HIP; \
    } while (0)

}  // namespace

namespace moe {

bool debug_sync_enabled() {
    static std::once_flag once;
    static bool on = false;
    std::call_once(once, [] {
        const char* v = getenv("MOE_DEBUG_SYNC");
        on = v != nullptr && v[0] != '\0' && strcmp(v, "0") != 0;
    });
    return on;
}

}  // namespace moe

extern "C" {

int moe_abi_version(void) { return MOE_ABI_VERSION; }

const char* moe_status_string(int status) {
    switch (status) {
        case MOE_OK: return "ok";
        case MOE_ERR_NULL: return "a required pointer is NULL";
        case MOE_ERR_SHAPE: return "a size is out of range or inconsistent";
        case MOE_ERR_ALIGN: return "a pointer violates its alignment";
        case MOE_ERR_WORKSPACE: return "workspace missing or too small";
        case MOE_ERR_HIP: return "a HIP launch failed";
        case MOE_ERR_UNSUPPORTED: return "request not supported by this build";
        default: return "unknown status";
    }
}

uint64_t moe_payload_bytes(int64_t S, int32_t K, int32_t D) {
    if (S < 0 || K < 0 || D < 0) return 0;
    return (uint64_t)S * (uint64_t)K * ((uint64_t)D * 2u + 4u);
}

uint64_t moe_mx_payload_bytes(int64_t S, int32_t K, int32_t D) {
    if (S < 0 || K < 0 || D < 0 || D % 32 != 0) return 0;
    return (uint64_t)S * (uint64_t)K * ((uint64_t)D + (uint64_t)D / 32u + 4u);
}

int moe_dispatch_mxfp8(const moe_bf16* x, const float* topk_prob, const int32_t* inv_perm, int64_t S, int32_t D,
                       int32_t K, uint8_t* x_q, uint8_t* x_scale, float* p_disp, hipStream_t stream) {
    if (S < 0 || !dim_ok(D) || D % 32 != 0 || K < 1 || K > kMaxK || S * (int64_t)K >= kMaxRows)
        return MOE_ERR_SHAPE;
    if ((topk_prob == nullptr) != (p_disp == nullptr)) return MOE_ERR_NULL;
    const uint64_t R = (uint64_t)S * K;
    MOE_TRY(need(x, (uint64_t)S * D * 2, 16));
    MOE_TRY(need(inv_perm, R * 4, 4));
    MOE_TRY(need(x_q, R * D, 8));
    MOE_TRY(need(x_scale, R * (D / 32), 1));
    MOE_TRY(opt(topk_prob, 4));
    MOE_TRY(opt(p_disp, 4));
    return hip_status(moe::launch_dispatch_mx(x, topk_prob, inv_perm, S, D, K, x_q, x_scale, p_disp, stream));
}

int moe_mxfp8_dequant(const uint8_t* x_q, const uint8_t* x_scale, int64_t R, int32_t D, moe_bf16* out,
                      hipStream_t stream) {
    if (R < 0 || R >= kMaxRows || !dim_ok(D) || D % 32 != 0) return MOE_ERR_SHAPE;
    MOE_TRY(need(x_q, (uint64_t)R * D, 8));
    MOE_TRY(need(x_scale, (uint64_t)R * (D / 32), 1));
    MOE_TRY(need(out, (uint64_t)R * D * 2, 16));
    return hip_status(moe::launch_dequant_mx(x_q, x_scale, R, D, out, stream));
}

size_t moe_router_logits_workspace_bytes(int32_t D, int32_t E) {
    if (!dim_ok(D) || E < 1 || E > kMaxE) return 0;
    return moe::router_ws_bytes(D, E);
}

int moe_router_logits(const moe_bf16* x_r, const float* Wr, const float* bias, int64_t S, int32_t D,
                      int32_t E, float* logits, void* ws, size_t ws_bytes, hipStream_t stream) {
    if (S < 0 || !dim_ok(D) || E < 1 || E > kMaxE) return MOE_ERR_SHAPE;
    MOE_TRY(need(x_r, (uint64_t)S * D * 2, 16));
    MOE_TRY(need(Wr, (uint64_t)D * E * 4, 4));
    MOE_TRY(opt(bias, 4));
    MOE_TRY(need(logits, (uint64_t)S * E * 4, 4));
    if (ws == nullptr || ws_bytes < moe::router_ws_bytes(D, E)) return MOE_ERR_WORKSPACE;
    MOE_TRY(opt(ws, 16));
    return hip_status(moe::launch_router_logits(x_r, Wr, bias, S, D, E, logits, ws, stream));
}

size_t moe_route_workspace_bytes(int64_t S, int32_t E, int32_t K) {
    if (check_route_shape(S, E, K) != MOE_OK) return 0;
    return moe::route_ws_bytes(S, E);
}

int moe_route_topk(const float* logits, int64_t S, int32_t E, int32_t K, int32_t* topk_idx,
                   float* topk_prob, int32_t* counts, int32_t* offsets, int32_t* perm,
                   int32_t* inv_perm, void* ws, size_t ws_bytes, hipStream_t stream) {
    MOE_TRY(check_route_shape(S, E, K));
    const uint64_t R = (uint64_t)S * K;
    MOE_TRY(need(logits, (uint64_t)S * E * 4, 4));
    MOE_TRY(need(topk_idx, R * 4, 4));
    MOE_TRY(need(topk_prob, R * 4, 4));
    MOE_TRY(need(counts, (uint64_t)E * 4, 4));
    MOE_TRY(need(offsets, (uint64_t)(E + 1) * 4, 4));
    MOE_TRY(need(perm, R * 4, 4));
    MOE_TRY(need(inv_perm, R * 4, 4));
    const size_t wsn = moe::route_ws_bytes(S, E);
    if (wsn > 0 && (ws == nullptr || ws_bytes < wsn)) return MOE_ERR_WORKSPACE;
    MOE_TRY(opt(ws, 16));
    return hip_status(moe::launch_route(logits, S, E, K, topk_idx, topk_prob, counts, offsets, perm,
                                        inv_perm, ws, stream));
}

int moe_dispatch(const moe_bf16* x, const float* topk_prob, const int32_t* inv_perm, int64_t S,
                 int32_t D, int32_t K, moe_bf16* x_disp, float* p_disp, hipStream_t stream) {
    if (S < 0 || !dim_ok(D) || K < 1 || K > kMaxK || S * (int64_t)K >= kMaxRows) return MOE_ERR_SHAPE;
    if ((topk_prob == nullptr) != (p_disp == nullptr)) return MOE_ERR_NULL;
    const uint64_t R = (uint64_t)S * K;
    MOE_TRY(need(x, (uint64_t)S * D * 2, 16));
    MOE_TRY(need(inv_perm, R * 4, 4));
    MOE_TRY(need(x_disp, R * D * 2, 16));
    MOE_TRY(opt(topk_prob, 4));
    MOE_TRY(opt(p_disp, 4));
    return hip_status(moe::launch_dispatch(x, topk_prob, inv_perm, S, D, K, x_disp, p_disp, stream));
}

int moe_combine(const moe_bf16* y_disp, const float* p_disp, const int32_t* inv_perm, int64_t S,
                int32_t D, int32_t K, moe_bf16* y, hipStream_t stream) {
    if (S < 0 || !dim_ok(D) || K < 1 || K > kMaxK || S * (int64_t)K >= kMaxRows) return MOE_ERR_SHAPE;
    const uint64_t R = (uint64_t)S * K;
    MOE_TRY(need(y_disp, R * D * 2, 16));
    MOE_TRY(opt(p_disp, 4));
    MOE_TRY(need(inv_perm, R * 4, 4));
    MOE_TRY(need(y, (uint64_t)S * D * 2, 16));
    return hip_status(moe::launch_combine(y_disp, p_disp, inv_perm, S, D, K, nullptr, y, stream));
}

size_t moe_grouped_ffn_workspace_bytes(int32_t E, int64_t R, int32_t D, int32_t F) {
    if (E < 1 || E > kMaxE || R < 0 || R >= kMaxRows || !dim_ok(D) || !dim_ok(F)) return 0;
    return moe::gemm_schedule_bytes(E, R);
}

static int check_ffn(const moe_bf16* x_disp, const int32_t* offsets, int32_t E, int64_t R, int32_t D,
                     int32_t F, const moe_bf16* W1, const moe_bf16* W2) {
    if (E < 1 || E > kMaxE || R < 0 || R >= kMaxRows || !dim_ok(D) || !dim_ok(F)) return MOE_ERR_SHAPE;
    if (!weight_ok(D, F)) return MOE_ERR_UNSUPPORTED;
    MOE_TRY(need(x_disp, (uint64_t)R * D * 2, 16));
    MOE_TRY(need(offsets, (uint64_t)(E + 1) * 4, 4));
    MOE_TRY(need(W1, (uint64_t)E * D * F * 2, 16));
    MOE_TRY(need(W2, (uint64_t)E * F * D * 2, 16));
    return MOE_OK;
}

int moe_grouped_ffn(const moe_bf16* x_disp, const int32_t* offsets, int32_t E, int64_t R, int32_t D,
                    int32_t F, const moe_bf16* W1, const moe_bf16* W2, moe_bf16* h, moe_bf16* u_save,
                    moe_bf16* y_disp, void* ws, size_t ws_bytes, hipStream_t stream) {
    MOE_TRY(check_ffn(x_disp, offsets, E, R, D, F, W1, W2));
    MOE_TRY(need(h, (uint64_t)R * F * 2, 16));
    MOE_TRY(opt(u_save, 16));
    MOE_TRY(need(y_disp, (uint64_t)R * D * 2, 16));
    const size_t wsn = moe::gemm_schedule_bytes(E, R);
    if (ws == nullptr || ws_bytes < wsn) return MOE_ERR_WORKSPACE;
    MOE_TRY(opt(ws, 16));
    if (R == 0) return MOE_OK;
    MOE_HIP(moe::launch_tile_schedule(offsets, E, R, ws, stream));
    MOE_HIP(moe::launch_grouped_rows(x_disp, D, W1, F, (int64_t)D * F, false, h, F, moe::EPI_RELU2,
                                     nullptr, u_save, ws, E, R, F, D, stream));
    MOE_HIP(moe::launch_grouped_rows(h, F, W2, D, (int64_t)F * D, false, y_disp, D, moe::EPI_BF16,
                                     nullptr, nullptr, ws, E, R, D, F, stream));
    return MOE_OK;
}

static_assert(moe::kStaticScratchBytes == MOE_STATIC_SCRATCH_BYTES, "static scratch size");

int moe_grouped_ffn_static(const moe_bf16* x_disp, const int32_t* offsets, int32_t E, int64_t R, int32_t D,
                           int32_t F, const moe_bf16* W1, const moe_bf16* W2, moe_bf16* h, moe_bf16* u_save,
                           moe_bf16* y_disp, hipStream_t stream) {
    MOE_TRY(check_ffn(x_disp, offsets, E, R, D, F, W1, W2));
    MOE_TRY(need(h, (uint64_t)R * F * 2, 16));
    MOE_TRY(opt(u_save, 16));
    MOE_TRY(need(y_disp, (uint64_t)R * D * 2, 16));
    if (R >= MOE_STATIC_MAX_ROWS || moe::gemm_schedule_bytes(E, R) > moe::kStaticScratchBytes)
        return MOE_ERR_WORKSPACE;
    if (R == 0) return MOE_OK;
    void* sched = nullptr;
    MOE_HIP(moe::static_scratch(&sched));
    MOE_HIP(moe::launch_tile_schedule(offsets, E, R, sched, stream));
    MOE_HIP(moe::launch_grouped_rows(x_disp, D, W1, F, (int64_t)D * F, false, h, F, moe::EPI_RELU2,
                                     nullptr, u_save, sched, E, R, F, D, stream));
    MOE_HIP(moe::launch_grouped_rows(h, F, W2, D, (int64_t)F * D, false, y_disp, D, moe::EPI_BF16,
                                     nullptr, nullptr, sched, E, R, D, F, stream));
    return MOE_OK;
}

size_t moe_grouped_schedule_bytes(int32_t E, int64_t R) {
    if (E < 1 || E > kMaxE || R < 0 || R >= kMaxRows) return 0;
    return moe::gemm_schedule_bytes(E, R);
}

int moe_grouped_schedule(const int32_t* offsets, int32_t E, int64_t R, void* sched, size_t sched_bytes,
                         hipStream_t stream) {
    if (E < 1 || E > kMaxE || R < 0 || R >= kMaxRows) return MOE_ERR_SHAPE;
    MOE_TRY(need(offsets, (uint64_t)(E + 1) * 4, 4));
    if (sched == nullptr || sched_bytes < moe::gemm_schedule_bytes(E, R)) return MOE_ERR_WORKSPACE;
    MOE_TRY(opt(sched, 16));
    return hip_status(moe::launch_tile_schedule(offsets, E, R, sched, stream));
}

int moe_grouped_gemm(const moe_bf16* A, const void* sched, int32_t E, int64_t R, int32_t Kd, int32_t N,
                     const moe_bf16* W, int32_t epilogue, moe_bf16* C, moe_bf16* u_save,
                     hipStream_t stream) {
    if (E < 1 || E > kMaxE || R < 0 || R >= kMaxRows || !dim_ok(Kd) || !dim_ok(N)) return MOE_ERR_SHAPE;
    if (epilogue != 0 && epilogue != 1) return MOE_ERR_UNSUPPORTED;
    if (!weight_ok(Kd, N)) return MOE_ERR_UNSUPPORTED;
    if (epilogue == 0 && u_save != nullptr) return MOE_ERR_SHAPE;
    MOE_TRY(need(A, (uint64_t)R * Kd * 2, 16));
    if (sched == nullptr) return MOE_ERR_NULL;
    MOE_TRY(opt(sched, 16));
    MOE_TRY(need(W, (uint64_t)E * Kd * N * 2, 16));
    MOE_TRY(need(C, (uint64_t)R * N * 2, 16));
    MOE_TRY(opt(u_save, 16));
    if (R == 0) return MOE_OK;
    return hip_status(moe::launch_grouped_rows(A, Kd, W, N, (int64_t)Kd * N, false, C, N,
                                               epilogue == 1 ? moe::EPI_RELU2 : moe::EPI_BF16, nullptr,
                                               u_save, sched, E, R, N, Kd, stream));
}

int moe_grouped_gemm_gather(const moe_bf16* x, const int32_t* perm, int64_t S, int32_t K, const void* sched,
                            int32_t E, int64_t R, int32_t Kd, int32_t N, const moe_bf16* W, int32_t epilogue,
                            moe_bf16* C, moe_bf16* u_save, hipStream_t stream) {
    if (E < 1 || E > kMaxE || R < 0 || R >= kMaxRows || !dim_ok(Kd) || !dim_ok(N)) return MOE_ERR_SHAPE;
    if (S < 0 || K < 1 || K > kMaxK || S * (int64_t)K != R) return MOE_ERR_SHAPE;
    if (epilogue != 0 && epilogue != 1) return MOE_ERR_UNSUPPORTED;
    if (!weight_ok(Kd, N) || !weight_ok(S, Kd)) return MOE_ERR_UNSUPPORTED;
    if (epilogue == 0 && u_save != nullptr) return MOE_ERR_SHAPE;
    MOE_TRY(need(x, (uint64_t)S * Kd * 2, 16));
    MOE_TRY(need(perm, (uint64_t)R * 4, 4));
    if (sched == nullptr) return MOE_ERR_NULL;
    MOE_TRY(opt(sched, 16));
    MOE_TRY(need(W, (uint64_t)E * Kd * N * 2, 16));
    MOE_TRY(need(C, (uint64_t)R * N * 2, 16));
    MOE_TRY(opt(u_save, 16));
    if (R == 0) return MOE_OK;
    return hip_status(moe::launch_grouped_rows_gather(x, Kd, S, perm, K, W, N, (int64_t)Kd * N, C, N,
                                                      epilogue == 1 ? moe::EPI_RELU2 : moe::EPI_BF16, u_save, sched,
                                                      E, R, N, Kd, stream));
}

uint64_t moe_mx_scale_alloc_bytes(int64_t R, int32_t D) {
    if (R < 0 || D < 32 || D % 32 != 0) return 0;
    return ((uint64_t)R * (uint64_t)(D / 32) + 3) / 4 * 4;
}

int moe_grouped_gemm_mxfp8(const uint8_t* x_q, const uint8_t* x_scale, const void* sched, int32_t E, int64_t R,
                           int32_t Kd, int32_t N, const moe_bf16* W, int32_t epilogue, moe_bf16* C,
                           moe_bf16* u_save, hipStream_t stream) {
    if (E < 1 || E > kMaxE || R < 0 || R >= kMaxRows || !dim_ok(Kd) || !dim_ok(N) || Kd % 32 != 0)
        return MOE_ERR_SHAPE;
    if (epilogue != 0 && epilogue != 1) return MOE_ERR_UNSUPPORTED;
    if (!weight_ok(Kd, N)) return MOE_ERR_UNSUPPORTED;
    if ((int64_t)moe_mx_scale_alloc_bytes(R, Kd) >= kMaxOperandBytes) return MOE_ERR_UNSUPPORTED;
    if (epilogue == 0 && u_save != nullptr) return MOE_ERR_SHAPE;
    MOE_TRY(need(x_q, (uint64_t)R * Kd, 16));
    MOE_TRY(need(x_scale, moe_mx_scale_alloc_bytes(R, Kd), 1));
    if (sched == nullptr) return MOE_ERR_NULL;
    MOE_TRY(opt(sched, 16));
    MOE_TRY(need(W, (uint64_t)E * Kd * N * 2, 16));
    MOE_TRY(need(C, (uint64_t)R * N * 2, 16));
    MOE_TRY(opt(u_save, 16));
    if (R == 0) return MOE_OK;
    return hip_status(moe::launch_grouped_rows_mx(x_q, x_scale, W, N, (int64_t)Kd * N, C, N,
                                                  epilogue == 1 ? moe::EPI_RELU2 : moe::EPI_BF16, u_save, sched,
                                                  E, R, N, Kd, stream));
}

int moe_latent_proj(const moe_bf16* A, const moe_bf16* W, int64_t M, int32_t Kd, int32_t N, moe_bf16* C,
                    hipStream_t stream) {
    if (M < 0 || M >= kMaxRows || !dim_ok(Kd) || !dim_ok(N)) return MOE_ERR_SHAPE;
    if (!weight_ok(Kd, N)) return MOE_ERR_UNSUPPORTED;
    MOE_TRY(need(A, (uint64_t)M * Kd * 2, 16));
    MOE_TRY(need(W, (uint64_t)Kd * N * 2, 16));
    MOE_TRY(need(C, (uint64_t)M * N * 2, 16));
    return hip_status(moe::launch_grouped_rows(A, Kd, W, N, 0, false, C, N, moe::EPI_BF16, nullptr,
                                               nullptr, nullptr, 1, M, N, Kd, stream));
}

// ---------------------------------------------------------------------------
// Whole layer
// ---------------------------------------------------------------------------

namespace {

struct Carve {
    char* base;
    size_t used;
    void* take(size_t bytes) {
        void* p = base ? base + used : nullptr;
        used += align256(bytes);
        return p;
    }
};

// coeff * E / (K T^2 B): the balance loss and its gradient per routed count.
double aux_coef(float coeff, int64_t S, int32_t E, int32_t K, int64_t T) {
    const double B = (double)(S / T);
    return (double)coeff * E / ((double)K * (double)T * (double)T * B);
}

int shared_fwd(const moe_bf16* x, const moe_bf16* Ws1, const moe_bf16* Ws2, int64_t S, int32_t D, int32_t Fs,
               moe_bf16* h_s, moe_bf16* u_s, float* y_s, hipStream_t stream) {
    // h_s = bf16(max(x Ws1, 0)^2) (u_s = bf16(x Ws1) if wanted), y_s = h_s Ws2 in fp32
    MOE_HIP(moe::launch_grouped_rows(x, D, Ws1, Fs, 0, false, h_s, Fs, moe::EPI_RELU2, nullptr, u_s, nullptr, 1,
                                     S, Fs, D, stream));
    MOE_HIP(moe::launch_grouped_rows(h_s, Fs, Ws2, D, 0, false, y_s, D, moe::EPI_F32, nullptr, nullptr, nullptr,
                                     1, S, D, Fs, stream));
    return MOE_OK;
}

// The caller's arguments in the full layout: a base-layout struct (the
// fields through ws_bytes) reads as zero / NULL beyond them.
int widen_args(const moe_layer_fwd_args* in, moe_layer_fwd_args* out) {
    if (in == nullptr) return MOE_ERR_NULL;
    const uint32_t n = in->struct_size;
    if (n != sizeof(moe_layer_fwd_args) && n != MOE_LAYER_FWD_ARGS_BASE_SIZE) return MOE_ERR_SHAPE;
    memset(out, 0, sizeof *out);
    memcpy(out, in, n);
    out->struct_size = sizeof *out;
    return MOE_OK;
}

int check_layer_args(const moe_layer_fwd_args* a) {
    MOE_TRY(check_route_shape(a->S, a->E, a->K));
    if (!dim_ok(a->D) || !dim_ok(a->F)) return MOE_ERR_SHAPE;
    if (a->H != 0 && !dim_ok(a->H)) return MOE_ERR_SHAPE;
    if (!weight_ok(a->D, a->F) || (a->H != 0 && !weight_ok(a->H, a->D))) return MOE_ERR_UNSUPPORTED;
    if (a->score_fn != MOE_SCORE_SOFTMAX && a->score_fn != MOE_SCORE_SIGMOID) return MOE_ERR_SHAPE;
    if (a->score_fn == MOE_SCORE_SOFTMAX && a->sel_bias != nullptr) return MOE_ERR_SHAPE;
    if (a->seq_len < 0 || (a->seq_len > 0 && (a->score_fn != MOE_SCORE_SIGMOID || a->S % a->seq_len != 0)))
        return MOE_ERR_SHAPE;
    if (a->Fs != 0) {
        if (!dim_ok(a->Fs)) return MOE_ERR_SHAPE;
        if (a->H != 0 || !weight_ok(a->D, a->Fs)) return MOE_ERR_UNSUPPORTED;
    }
    if (a->payload != MOE_PAYLOAD_BF16 && a->payload != MOE_PAYLOAD_MXFP8) return MOE_ERR_SHAPE;
    if (a->payload == MOE_PAYLOAD_MXFP8 && a->D % 32 != 0) return MOE_ERR_SHAPE;
    return MOE_OK;
}

// The bf16 payload with x_disp not exported: the route also writes p_disp
// and the tile tables, and the up projection gathers its rows from the
// router input through perm, so no dispatch kernel runs and the dispatched
// rows are never materialised (Section 5.2's permute fusion).  The gather's
// descriptor spans the router input, so it must stay below 2^31 bytes.
bool fused_dispatch(const moe_layer_fwd_args* a) {
    return a->payload == MOE_PAYLOAD_BF16 && a->x_disp == nullptr &&
           a->S * (int64_t)a->D * 2 < kMaxOperandBytes;
}

// Lays the non-exported intermediates out in the workspace (or, with base
// == nullptr, only counts the bytes).  Pointers the caller exported win.
struct LayerBufs {
    moe_bf16* x_lat; float* logits; int32_t* topk_idx; float* topk_prob; int32_t* counts;
    int32_t* offsets; int32_t* perm; int32_t* inv_perm; moe_bf16* x_disp; float* p_disp;
    moe_bf16* h; moe_bf16* y_disp; moe_bf16* y_lat; void* route_ws; void* sched; void* router_ws;
    void* aux_ws; int32_t* seq_counts; moe_bf16* h_s; float* y_s; uint8_t* x_q; uint8_t* x_scale;
};

size_t layer_layout(const moe_layer_fwd_args* a, char* base, LayerBufs* b) {
    Carve c{base, 0};
    const int64_t S = a->S, R = S * a->K;
    const int D = a->D, E = a->E, F = a->F;
    auto pick = [&](auto* user, size_t bytes) -> decltype(user) {
        if (user != nullptr) return user;
        return (decltype(user))c.take(bytes);
    };
    b->x_lat = a->H ? pick(a->x_lat, (size_t)S * D * 2) : nullptr;
    b->logits = pick(a->logits, (size_t)S * E * 4);
    b->topk_idx = pick(a->topk_idx, (size_t)R * 4);
    b->topk_prob = pick(a->topk_prob, (size_t)R * 4);
    b->counts = pick(a->counts, (size_t)E * 4);
    b->offsets = pick(a->offsets, (size_t)(E + 1) * 4);
    b->perm = pick(a->perm, (size_t)R * 4);
    b->inv_perm = pick(a->inv_perm, (size_t)R * 4);
    const bool mx = a->payload == MOE_PAYLOAD_MXFP8;
    // the MX payload feeds the up projection as sent, and with the bf16
    // payload the up projection gathers its rows from the router input
    // (permutation fused into its operand copy): x_disp (the decode, or the
    // dispatched rows) exists only when the caller exports it
    b->x_disp = (mx || fused_dispatch(a)) ? a->x_disp : pick(a->x_disp, (size_t)R * D * 2);
    b->p_disp = pick(a->p_disp, (size_t)R * 4);
    b->h = pick(a->h, (size_t)R * F * 2);
    b->y_disp = pick(a->y_disp, (size_t)R * D * 2);
    b->y_lat = a->H ? pick(a->y_lat, (size_t)S * D * 2) : nullptr;
    b->route_ws = c.take(moe::route_ws_bytes(S, E));
    b->sched = c.take(moe::gemm_schedule_bytes(E, R));
    b->router_ws = c.take(moe::router_ws_bytes(D, E));
    b->aux_ws = nullptr;
    b->seq_counts = nullptr;
    if (a->seq_len > 0) {
        b->aux_ws = c.take(moe::seq_aux_ws_bytes(S, E, a->seq_len));
        b->seq_counts = pick(a->seq_counts, (size_t)(S / a->seq_len) * E * 4);
    }
    b->x_q = mx ? pick(a->x_q, (size_t)R * D) : nullptr;
    b->x_scale = mx ? pick(a->x_scale, (size_t)moe_mx_scale_alloc_bytes(R, D)) : nullptr;
    b->h_s = a->Fs ? pick(a->h_s, (size_t)S * a->Fs * 2) : nullptr;
    b->y_s = a->Fs ? pick(a->y_s, (size_t)S * D * 4) : nullptr;
    return c.used;
}

}  // namespace

size_t moe_layer_fwd_workspace_bytes(const moe_layer_fwd_args* args) {
    moe_layer_fwd_args full;
    if (widen_args(args, &full) != MOE_OK) return 0;
    const moe_layer_fwd_args* a = &full;
    if (check_layer_args(a) != MOE_OK) return 0;
    LayerBufs b;
    return layer_layout(a, nullptr, &b);
}

int moe_layer_fwd(const moe_layer_fwd_args* args, hipStream_t stream) {
    moe_layer_fwd_args full;
    MOE_TRY(widen_args(args, &full));
    const moe_layer_fwd_args* a = &full;
    MOE_TRY(check_layer_args(a));
    const int64_t S = a->S, R = S * a->K;
    const int H = a->H, D = a->D, E = a->E, K = a->K, F = a->F;
    const int in_w = H ? H : D;
    MOE_TRY(need(a->x, (uint64_t)S * in_w * 2, 16));
    MOE_TRY(need(a->Wr, (uint64_t)D * E * 4, 4));
    MOE_TRY(opt(a->router_bias, 4));
    MOE_TRY(need(a->W1, (uint64_t)E * D * F * 2, 16));
    MOE_TRY(need(a->W2, (uint64_t)E * F * D * 2, 16));
    MOE_TRY(need(a->y, (uint64_t)S * in_w * 2, 16));
    if (H) {
        MOE_TRY(need(a->Wdown, (uint64_t)H * D * 2, 16));
        MOE_TRY(need(a->Wup, (uint64_t)D * H * 2, 16));
    } else if (a->Wdown != nullptr || a->Wup != nullptr) {
        return MOE_ERR_SHAPE;
    }
    if (a->Fs) {
        MOE_TRY(need(a->Ws1, (uint64_t)D * a->Fs * 2, 16));
        MOE_TRY(need(a->Ws2, (uint64_t)a->Fs * D * 2, 16));
    } else if (a->Ws1 != nullptr || a->Ws2 != nullptr) {
        return MOE_ERR_SHAPE;
    }
    if (a->seq_len > 0) MOE_TRY(need(a->aux_loss, 4, 4));
    const void* bf16_ptrs[] = {a->x_lat, a->x_disp, a->h, a->u_save, a->y_disp, a->y_lat, a->h_s, a->u_s,
                               a->y_s, a->x_q};
    for (const void* p : bf16_ptrs) MOE_TRY(opt(p, 16));
    const void* word_ptrs[] = {a->logits, a->topk_idx, a->topk_prob, a->counts, a->offsets,
                               a->perm, a->inv_perm, a->p_disp, a->sel_bias, a->seq_counts};
    for (const void* p : word_ptrs) MOE_TRY(opt(p, 4));

    LayerBufs b;
    const size_t need_ws = layer_layout(a, nullptr, &b);
    if (a->ws == nullptr || a->ws_bytes < need_ws) return MOE_ERR_WORKSPACE;
    MOE_TRY(opt(a->ws, 256));
    layer_layout(a, (char*)a->ws, &b);

    const moe_bf16* x_r = a->x;
    if (H) {
        MOE_HIP(moe::launch_grouped_rows(a->x, H, a->Wdown, D, 0, false, b.x_lat, D, moe::EPI_BF16,
                                         nullptr, nullptr, nullptr, 1, S, D, H, stream));
        x_r = b.x_lat;
    }
    MOE_HIP(moe::launch_router_logits(x_r, a->Wr, a->router_bias, S, D, E, b.logits, b.router_ws, stream));
    const bool sig = a->score_fn == MOE_SCORE_SIGMOID;
    const bool fused = fused_dispatch(a);
    MOE_HIP(moe::launch_route(b.logits, S, E, K, b.topk_idx, b.topk_prob, b.counts, b.offsets, b.perm,
                              b.inv_perm, b.route_ws, stream, sig, a->sel_bias, fused ? b.p_disp : nullptr,
                              fused && R > 0 ? b.sched : nullptr));
    if (a->seq_len > 0) {
        MOE_HIP(moe::launch_seq_aux_loss(b.logits, b.topk_idx, S, E, K, a->seq_len,
                                         aux_coef(a->aux_coeff, S, E, K, a->seq_len), a->aux_loss,
                                         b.seq_counts, b.aux_ws, stream));
    }
    // the dispatch launch also builds the grouped GEMM's tile tables
    const bool mx = a->payload == MOE_PAYLOAD_MXFP8;
    if (mx) {
        MOE_HIP(moe::launch_dispatch_mx(x_r, b.topk_prob, b.inv_perm, S, D, K, b.x_q, b.x_scale, b.p_disp, stream,
                                        R > 0 ? b.offsets : nullptr, E, R > 0 ? b.sched : nullptr));
        if (b.x_disp != nullptr) MOE_HIP(moe::launch_dequant_mx(b.x_q, b.x_scale, R, D, b.x_disp, stream));
    } else if (!fused) {
        MOE_HIP(moe::launch_dispatch(x_r, b.topk_prob, b.inv_perm, S, D, K, b.x_disp, b.p_disp, stream,
                                     R > 0 ? b.offsets : nullptr, E, R > 0 ? b.sched : nullptr));
    }
    if (R > 0) {
        if (mx)
            MOE_HIP(moe::launch_grouped_rows_mx(b.x_q, b.x_scale, a->W1, F, (int64_t)D * F, b.h, F, moe::EPI_RELU2,
                                                a->u_save, b.sched, E, R, F, D, stream));
        else if (fused)
            MOE_HIP(moe::launch_grouped_rows_gather(x_r, D, S, b.perm, K, a->W1, F, (int64_t)D * F, b.h, F,
                                                    moe::EPI_RELU2, a->u_save, b.sched, E, R, F, D, stream));
        else
            MOE_HIP(moe::launch_grouped_rows(b.x_disp, D, a->W1, F, (int64_t)D * F, false, b.h, F,
                                             moe::EPI_RELU2, nullptr, a->u_save, b.sched, E, R, F, D, stream));
        MOE_HIP(moe::launch_grouped_rows(b.h, F, a->W2, D, (int64_t)F * D, false, b.y_disp, D,
                                         moe::EPI_BF16, nullptr, nullptr, b.sched, E, R, D, F, stream));
    }
    if (a->Fs && S > 0) MOE_TRY(shared_fwd(a->x, a->Ws1, a->Ws2, S, D, a->Fs, b.h_s, a->u_s, b.y_s, stream));
    moe_bf16* comb_out = H ? b.y_lat : a->y;
    MOE_HIP(moe::launch_combine(b.y_disp, b.p_disp, b.inv_perm, S, D, K, b.y_s, comb_out, stream));
    if (H) {
        MOE_HIP(moe::launch_grouped_rows(b.y_lat, D, a->Wup, H, 0, false, a->y, H, moe::EPI_BF16,
                                         nullptr, nullptr, nullptr, 1, S, H, D, stream));
    }
    return MOE_OK;
}

// ---------------------------------------------------------------------------
// Backward
// ---------------------------------------------------------------------------

int moe_combine_bwd(const moe_bf16* dy, const moe_bf16* y_disp, const float* p_disp,
                    const int32_t* inv_perm, int64_t S, int32_t D, int32_t K, moe_bf16* dy_disp,
                    float* dp, hipStream_t stream) {
    if (S < 0 || !dim_ok(D) || K < 1 || K > kMaxK || S * (int64_t)K >= kMaxRows) return MOE_ERR_SHAPE;
    const uint64_t R = (uint64_t)S * K;
    MOE_TRY(need(dy, (uint64_t)S * D * 2, 16));
    MOE_TRY(need(y_disp, R * D * 2, 16));
    MOE_TRY(opt(p_disp, 4));
    MOE_TRY(need(inv_perm, R * 4, 4));
    MOE_TRY(need(dy_disp, R * D * 2, 16));
    MOE_TRY(opt(dp, 4));
    return hip_status(moe::launch_combine_bwd(dy, y_disp, p_disp, inv_perm, S, D, K, dy_disp, dp, stream));
}

size_t moe_grouped_ffn_bwd_workspace_bytes(int32_t E, int64_t R, int32_t D, int32_t F) {
    if (E < 1 || E > kMaxE || R < 0 || R >= kMaxRows || !dim_ok(D) || !dim_ok(F)) return 0;
    return align256((size_t)R * F * 2) + moe::gemm_schedule_bytes(E, R) + align256((size_t)E * 4);
}

int moe_grouped_ffn_bwd(const moe_bf16* x_disp, const moe_bf16* u_save, const moe_bf16* h,
                        const moe_bf16* dy_disp, const int32_t* offsets, int32_t E, int64_t R, int32_t D,
                        int32_t F, const moe_bf16* W1, const moe_bf16* W2, moe_bf16* dx_disp,
                        float* dW1, float* dW2, void* ws, size_t ws_bytes, hipStream_t stream) {
    MOE_TRY(check_ffn(x_disp, offsets, E, R, D, F, W1, W2));
    if (!weight_ok(R, D > F ? D : F)) return MOE_ERR_UNSUPPORTED;  // wgrad operand rows
    MOE_TRY(need(u_save, (uint64_t)R * F * 2, 16));
    MOE_TRY(need(h, (uint64_t)R * F * 2, 16));
    MOE_TRY(need(dy_disp, (uint64_t)R * D * 2, 16));
    MOE_TRY(need(dx_disp, (uint64_t)R * D * 2, 16));
    MOE_TRY(need(dW1, (uint64_t)E * D * F * 4, 16));
    MOE_TRY(need(dW2, (uint64_t)E * F * D * 4, 16));
    const size_t du_bytes = align256((size_t)R * F * 2);
    const size_t sched_bytes = moe::gemm_schedule_bytes(E, R);
    const size_t wsn = du_bytes + sched_bytes + align256((size_t)E * 4);
    if (ws == nullptr || ws_bytes < wsn) return MOE_ERR_WORKSPACE;
    MOE_TRY(opt(ws, 256));
    moe_bf16* du = (moe_bf16*)ws;
    void* sched = (char*)ws + du_bytes;
    int32_t* order = (int32_t*)((char*)ws + du_bytes + sched_bytes);
    MOE_HIP(moe::launch_expert_order(offsets, E, R, order, stream));
    if (R > 0) {
        MOE_HIP(moe::launch_tile_schedule(offsets, E, R, sched, stream));
        // du = (dy_disp @ W2[e]^T) * 2 max(u, 0): W2[e] is [F, D], read K(=D)-contiguous
        MOE_HIP(moe::launch_grouped_rows(dy_disp, D, W2, D, (int64_t)F * D, true, du, F, moe::EPI_DRELU2,
                                         u_save, nullptr, sched, E, R, F, D, stream));
        // dx_disp = du @ W1[e]^T: W1[e] is [D, F], read K(=F)-contiguous
        MOE_HIP(moe::launch_grouped_rows(du, F, W1, F, (int64_t)D * F, true, dx_disp, D, moe::EPI_BF16,
                                         nullptr, nullptr, sched, E, R, D, F, stream));
    }
    // dW2[e] = h_e^T @ dy_disp_e  ([F, D]);  dW1[e] = x_disp_e^T @ du_e  ([D, F])
    // both in one launch, the experts with the most rows first
    MOE_HIP(moe::launch_grouped_wgrad2(h, F, dy_disp, D, dW2, D, (int64_t)F * D, F, D, x_disp, D, du, F, dW1, F,
                                       (int64_t)D * F, D, F, offsets, order, E, R, stream));
    return MOE_OK;
}

int moe_dispatch_bwd(const moe_bf16* dx_disp, const int32_t* inv_perm, int64_t S, int32_t D, int32_t K,
                     moe_bf16* dx, hipStream_t stream) {
    if (S < 0 || !dim_ok(D) || K < 1 || K > kMaxK || S * (int64_t)K >= kMaxRows) return MOE_ERR_SHAPE;
    const uint64_t R = (uint64_t)S * K;
    MOE_TRY(need(dx_disp, R * D * 2, 16));
    MOE_TRY(need(inv_perm, R * 4, 4));
    MOE_TRY(need(dx, (uint64_t)S * D * 2, 16));
    return hip_status(moe::launch_combine(dx_disp, nullptr, inv_perm, S, D, K, nullptr, dx, stream));
}

int moe_dispatch_bwd_add(const moe_bf16* dx_disp, const int32_t* inv_perm, const float* dx_add, int64_t S,
                         int32_t D, int32_t K, moe_bf16* dx, hipStream_t stream) {
    if (S < 0 || !dim_ok(D) || K < 1 || K > kMaxK || S * (int64_t)K >= kMaxRows) return MOE_ERR_SHAPE;
    const uint64_t R = (uint64_t)S * K;
    MOE_TRY(need(dx_disp, R * D * 2, 16));
    MOE_TRY(need(inv_perm, R * 4, 4));
    MOE_TRY(need(dx_add, (uint64_t)S * D * 4, 16));
    MOE_TRY(need(dx, (uint64_t)S * D * 2, 16));
    return hip_status(moe::launch_combine(dx_disp, nullptr, inv_perm, S, D, K, dx_add, dx, stream));
}

size_t moe_router_bwd_workspace_bytes(int64_t S, int32_t D, int32_t E) {
    if (S < 0 || S >= kMaxRows || !dim_ok(D) || E < 1 || E > kMaxE) return 0;
    return moe::router_bwd_ws_bytes(S, D, E);
}

int moe_router_bwd(const moe_bf16* x_r, const float* Wr, const int32_t* topk_idx, const float* topk_prob,
                   const float* dp, int64_t S, int32_t D, int32_t E, int32_t K, float* dlogits, float* dWr,
                   float* dbias, float* dx_r, void* ws, size_t ws_bytes, hipStream_t stream) {
    MOE_TRY(check_route_shape(S, E, K));
    if (!dim_ok(D)) return MOE_ERR_SHAPE;
    const int32_t E3 = 3 * ((E + 7) / 8 * 8);  // the three bf16 planes of dlogits, rows padded to 8
    if (!weight_ok(S, D > E3 ? D : E3)) return MOE_ERR_UNSUPPORTED;  // dWr operand rows
    const uint64_t R = (uint64_t)S * K;
    MOE_TRY(need(x_r, (uint64_t)S * D * 2, 16));
    MOE_TRY(need(Wr, (uint64_t)D * E * 4, 4));
    MOE_TRY(need(topk_idx, R * 4, 4));
    MOE_TRY(need(topk_prob, R * 4, 4));
    MOE_TRY(need(dp, R * 4, 4));
    MOE_TRY(opt(dlogits, 4));
    MOE_TRY(need(dWr, (uint64_t)D * E * 4, 4));
    MOE_TRY(opt(dbias, 4));
    MOE_TRY(opt(dx_r, 16));
    if (ws == nullptr || ws_bytes < moe::router_bwd_ws_bytes(S, D, E)) return MOE_ERR_WORKSPACE;
    MOE_TRY(opt(ws, 256));
    return hip_status(moe::launch_router_bwd(x_r, Wr, topk_idx, topk_prob, dp, S, D, E, K, dlogits, dWr,
                                             dbias, dx_r, ws, stream));
}

size_t moe_latent_proj_bwd_workspace_bytes(int64_t M, int32_t Kd, int32_t N) {
    if (M < 0 || M >= kMaxRows || !dim_ok(Kd) || !dim_ok(N)) return 0;
    return align256((size_t)moe::wgrad_chunks(M, Kd, N) * Kd * N * 4);
}

int moe_latent_proj_bwd(const moe_bf16* x_in, const moe_bf16* W, const moe_bf16* dout, int64_t M, int32_t Kd,
                        int32_t N, moe_bf16* dx_in, float* dW, void* ws, size_t ws_bytes, hipStream_t stream) {
    if (M < 0 || M >= kMaxRows || !dim_ok(Kd) || !dim_ok(N)) return MOE_ERR_SHAPE;
    if (!weight_ok(Kd, N)) return MOE_ERR_UNSUPPORTED;
    if (dW != nullptr && !weight_ok(M, Kd > N ? Kd : N)) return MOE_ERR_UNSUPPORTED;
    MOE_TRY(need(dout, (uint64_t)M * N * 2, 16));
    if (dx_in != nullptr) {
        MOE_TRY(need(W, (uint64_t)Kd * N * 2, 16));
        MOE_TRY(need(dx_in, (uint64_t)M * Kd * 2, 16));
    }
    if (dW != nullptr) {
        MOE_TRY(need(x_in, (uint64_t)M * Kd * 2, 16));
        MOE_TRY(need(dW, (uint64_t)Kd * N * 4, 4));
        if (ws == nullptr || ws_bytes < moe_latent_proj_bwd_workspace_bytes(M, Kd, N)) return MOE_ERR_WORKSPACE;
        MOE_TRY(opt(ws, 256));
    }
    if (dx_in != nullptr && M > 0) {
        // dx_in[m, kd] = sum_n dout[m, n] W[kd, n]: W read N-contiguous per output column
        MOE_HIP(moe::launch_grouped_rows(dout, N, W, N, 0, true, dx_in, Kd, moe::EPI_BF16, nullptr, nullptr,
                                         nullptr, 1, M, Kd, N, stream));
    }
    if (dW != nullptr) {
        const int nch = moe::wgrad_chunks(M, Kd, N);
        const int64_t kchunk = M > 0 ? (M + nch - 1) / nch : 1;
        float* part = (float*)ws;
        MOE_HIP(moe::launch_chunked_wgrad(x_in, Kd, dout, N, part, N, (int64_t)Kd * N, nch, kchunk, Kd, N, M,
                                          stream));
        MOE_HIP(moe::launch_sum_planes(part, nch, Kd, N, 1, N, dW, stream));
    }
    return MOE_OK;
}

// ---------------------------------------------------------------------------
// Production router (sigmoid scores, selection-only bias, balance loss) and
// the shared expert
// ---------------------------------------------------------------------------

int moe_route_sigmoid(const float* logits, const float* sel_bias, int64_t S, int32_t E, int32_t K,
                      int32_t* topk_idx, float* topk_gate, int32_t* counts, int32_t* offsets, int32_t* perm,
                      int32_t* inv_perm, void* ws, size_t ws_bytes, hipStream_t stream) {
    MOE_TRY(check_route_shape(S, E, K));
    const uint64_t R = (uint64_t)S * K;
    MOE_TRY(need(logits, (uint64_t)S * E * 4, 4));
    MOE_TRY(opt(sel_bias, 4));
    MOE_TRY(need(topk_idx, R * 4, 4));
    MOE_TRY(need(topk_gate, R * 4, 4));
    MOE_TRY(need(counts, (uint64_t)E * 4, 4));
    MOE_TRY(need(offsets, (uint64_t)(E + 1) * 4, 4));
    MOE_TRY(need(perm, R * 4, 4));
    MOE_TRY(need(inv_perm, R * 4, 4));
    const size_t wsn = moe::route_ws_bytes(S, E);
    if (wsn > 0 && (ws == nullptr || ws_bytes < wsn)) return MOE_ERR_WORKSPACE;
    MOE_TRY(opt(ws, 16));
    return hip_status(moe::launch_route(logits, S, E, K, topk_idx, topk_gate, counts, offsets, perm, inv_perm,
                                        ws, stream, true, sel_bias));
}

size_t moe_seq_aux_loss_workspace_bytes(int64_t S, int32_t E, int64_t seq_len) {
    if (S < 0 || S >= kMaxRows || E < 1 || E > kMaxE || seq_len < 1 || S % seq_len != 0) return 0;
    return moe::seq_aux_ws_bytes(S, E, seq_len);
}

int moe_seq_aux_loss(const float* logits, const int32_t* topk_idx, int64_t S, int32_t E, int32_t K,
                     int64_t seq_len, float coeff, float* loss, int32_t* seq_counts, void* ws, size_t ws_bytes,
                     hipStream_t stream) {
    MOE_TRY(check_route_shape(S, E, K));
    if (seq_len < 1 || S % seq_len != 0) return MOE_ERR_SHAPE;
    MOE_TRY(need(logits, (uint64_t)S * E * 4, 4));
    MOE_TRY(need(topk_idx, (uint64_t)S * K * 4, 4));
    MOE_TRY(need(loss, 4, 4));
    MOE_TRY(opt(seq_counts, 4));
    const size_t wsn = moe::seq_aux_ws_bytes(S, E, seq_len);
    if (wsn > 0 && (ws == nullptr || ws_bytes < wsn)) return MOE_ERR_WORKSPACE;
    MOE_TRY(opt(ws, 16));
    return hip_status(moe::launch_seq_aux_loss(logits, topk_idx, S, E, K, seq_len, aux_coef(coeff, S, E, K, seq_len),
                                               loss, seq_counts, ws, stream));
}

size_t moe_router_bwd_sigmoid_workspace_bytes(int64_t S, int32_t D, int32_t E) {
    if (S < 0 || S >= kMaxRows || !dim_ok(D) || E < 1 || E > kMaxE) return 0;
    return moe::router_bwd_ws_bytes(S, D, E, true);
}

int moe_router_bwd_sigmoid(const moe_bf16* x_r, const float* Wr, const float* logits, const int32_t* topk_idx,
                           const float* topk_gate, const float* dg, const int32_t* seq_counts, int64_t seq_len,
                           float coeff, int64_t S, int32_t D, int32_t E, int32_t K, float* dlogits, float* dWr,
                           float* dbias, float* dx_r, void* ws, size_t ws_bytes, hipStream_t stream) {
    MOE_TRY(check_route_shape(S, E, K));
    if (!dim_ok(D)) return MOE_ERR_SHAPE;
    if (seq_counts != nullptr && (seq_len < 1 || S % seq_len != 0)) return MOE_ERR_SHAPE;
    const int32_t E6 = 6 * ((E + 7) / 8 * 8);  // widest bf16 plane rows of dlogits
    if (!weight_ok(S, D > E6 ? D : E6)) return MOE_ERR_UNSUPPORTED;
    const uint64_t R = (uint64_t)S * K;
    MOE_TRY(need(x_r, (uint64_t)S * D * 2, 16));
    MOE_TRY(need(Wr, (uint64_t)D * E * 4, 4));
    MOE_TRY(need(logits, (uint64_t)S * E * 4, 4));
    MOE_TRY(need(topk_idx, R * 4, 4));
    MOE_TRY(need(topk_gate, R * 4, 4));
    MOE_TRY(need(dg, R * 4, 4));
    MOE_TRY(opt(seq_counts, 4));
    MOE_TRY(opt(dlogits, 4));
    MOE_TRY(need(dWr, (uint64_t)D * E * 4, 4));
    MOE_TRY(opt(dbias, 4));
    MOE_TRY(opt(dx_r, 16));
    if (ws == nullptr || ws_bytes < moe::router_bwd_ws_bytes(S, D, E, true)) return MOE_ERR_WORKSPACE;
    MOE_TRY(opt(ws, 256));
    const float coef = seq_counts != nullptr ? (float)aux_coef(coeff, S, E, K, seq_len) : 0.f;
    return hip_status(moe::launch_router_bwd_sigmoid(x_r, Wr, logits, topk_idx, topk_gate, dg, seq_counts,
                                                     seq_counts != nullptr ? seq_len : 1, coef, S, D, E, K,
                                                     dlogits, dWr, dbias, dx_r, ws, stream));
}

int moe_expert_bias_update(const int32_t* counts, int32_t E, float rate, float* sel_bias, hipStream_t stream) {
    if (E < 1 || E > kMaxE) return MOE_ERR_SHAPE;
    MOE_TRY(need(counts, (uint64_t)E * 4, 4));
    MOE_TRY(need(sel_bias, (uint64_t)E * 4, 4));
    return hip_status(moe::launch_expert_bias_update(counts, E, rate, sel_bias, stream));
}

int moe_combine_add(const moe_bf16* y_disp, const float* p_disp, const int32_t* inv_perm, const float* y_add,
                    int64_t S, int32_t D, int32_t K, moe_bf16* y, hipStream_t stream) {
    if (S < 0 || !dim_ok(D) || K < 1 || K > kMaxK || S * (int64_t)K >= kMaxRows) return MOE_ERR_SHAPE;
    const uint64_t R = (uint64_t)S * K;
    MOE_TRY(need(y_disp, R * D * 2, 16));
    MOE_TRY(opt(p_disp, 4));
    MOE_TRY(need(inv_perm, R * 4, 4));
    MOE_TRY(need(y_add, (uint64_t)S * D * 4, 16));
    MOE_TRY(need(y, (uint64_t)S * D * 2, 16));
    return hip_status(moe::launch_combine(y_disp, p_disp, inv_perm, S, D, K, y_add, y, stream));
}

static int check_shared(int64_t S, int32_t D, int32_t Fs) {
    if (S < 0 || S >= kMaxRows || !dim_ok(D) || !dim_ok(Fs)) return MOE_ERR_SHAPE;
    if (!weight_ok(D, Fs)) return MOE_ERR_UNSUPPORTED;
    return MOE_OK;
}

int moe_shared_expert_fwd(const moe_bf16* x, const moe_bf16* Ws1, const moe_bf16* Ws2, int64_t S, int32_t D,
                          int32_t Fs, moe_bf16* h_s, moe_bf16* u_s, float* y_s, hipStream_t stream) {
    MOE_TRY(check_shared(S, D, Fs));
    MOE_TRY(need(x, (uint64_t)S * D * 2, 16));
    MOE_TRY(need(Ws1, (uint64_t)D * Fs * 2, 16));
    MOE_TRY(need(Ws2, (uint64_t)Fs * D * 2, 16));
    MOE_TRY(need(h_s, (uint64_t)S * Fs * 2, 16));
    MOE_TRY(opt(u_s, 16));
    MOE_TRY(need(y_s, (uint64_t)S * D * 4, 16));
    if (S == 0) return MOE_OK;
    return shared_fwd(x, Ws1, Ws2, S, D, Fs, h_s, u_s, y_s, stream);
}

static size_t shared_bwd_ws(int64_t S, int32_t D, int32_t Fs) {
    const int nch = moe::wgrad_chunks(S, D > Fs ? D : Fs, D > Fs ? Fs : D);
    return align256((size_t)S * Fs * 2) + align256((size_t)nch * D * Fs * 4);
}

size_t moe_shared_expert_bwd_workspace_bytes(int64_t S, int32_t D, int32_t Fs) {
    if (check_shared(S, D, Fs) != MOE_OK) return 0;
    return shared_bwd_ws(S, D, Fs);
}

int moe_shared_expert_bwd(const moe_bf16* x, const moe_bf16* u_s, const moe_bf16* h_s, const moe_bf16* dy,
                          const moe_bf16* Ws1, const moe_bf16* Ws2, int64_t S, int32_t D, int32_t Fs, float* dx,
                          int32_t accumulate_dx, float* dWs1, float* dWs2, void* ws, size_t ws_bytes,
                          hipStream_t stream) {
    MOE_TRY(check_shared(S, D, Fs));
    if (!weight_ok(S, D > Fs ? D : Fs)) return MOE_ERR_UNSUPPORTED;  // wgrad operand rows
    MOE_TRY(need(x, (uint64_t)S * D * 2, 16));
    MOE_TRY(need(u_s, (uint64_t)S * Fs * 2, 16));
    MOE_TRY(need(h_s, (uint64_t)S * Fs * 2, 16));
    MOE_TRY(need(dy, (uint64_t)S * D * 2, 16));
    MOE_TRY(need(Ws1, (uint64_t)D * Fs * 2, 16));
    MOE_TRY(need(Ws2, (uint64_t)Fs * D * 2, 16));
    MOE_TRY(opt(dx, 16));
    MOE_TRY(need(dWs1, (uint64_t)D * Fs * 4, 4));
    MOE_TRY(need(dWs2, (uint64_t)Fs * D * 4, 4));
    if (ws == nullptr || ws_bytes < shared_bwd_ws(S, D, Fs)) return MOE_ERR_WORKSPACE;
    MOE_TRY(opt(ws, 256));
    moe_bf16* du = (moe_bf16*)ws;
    float* part = (float*)((char*)ws + align256((size_t)S * Fs * 2));
    if (S > 0) {
        // du = (dy Ws2^T) * 2 max(u, 0): Ws2 [Fs, D] read D-contiguous per output column
        MOE_HIP(moe::launch_grouped_rows(dy, D, Ws2, D, 0, true, du, Fs, moe::EPI_DRELU2, u_s, nullptr, nullptr, 1,
                                         S, Fs, D, stream));
        if (dx != nullptr) {
            // dx (+)= du Ws1^T: Ws1 [D, Fs] read Fs-contiguous per output column
            MOE_HIP(moe::launch_grouped_rows(du, Fs, Ws1, Fs, 0, true, dx, D, moe::EPI_F32, nullptr, nullptr,
                                             nullptr, 1, S, D, Fs, stream, accumulate_dx != 0));
        }
    }
    const int nch = moe::wgrad_chunks(S, D > Fs ? D : Fs, D > Fs ? Fs : D);
    const int64_t kchunk = S > 0 ? (S + nch - 1) / nch : 1;
    // dWs2 [Fs, D] = h_s^T dy;  dWs1 [D, Fs] = x^T du  (the partial buffer is reused in stream order)
    MOE_HIP(moe::launch_chunked_wgrad(h_s, Fs, dy, D, part, D, (int64_t)Fs * D, nch, kchunk, Fs, D, S, stream));
    MOE_HIP(moe::launch_sum_planes(part, nch, Fs, D, 1, D, dWs2, stream));
    MOE_HIP(moe::launch_chunked_wgrad(x, D, du, Fs, part, Fs, (int64_t)D * Fs, nch, kchunk, D, Fs, S, stream));
    MOE_HIP(moe::launch_sum_planes(part, nch, D, Fs, 1, Fs, dWs1, stream));
    return MOE_OK;
}

}  // extern "C"
