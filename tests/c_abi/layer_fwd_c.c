/* A plain C consumer of the library's C ABI (no Python, no torch): it
 * allocates device memory with the HIP runtime, runs one moe_layer_fwd and
 * writes the results back to files, so that a test can compare them with the
 * Python binding's call on the same inputs.
 *
 *   layer_fwd_c --abi          print the loaded library's ABI version and the
 *                              header's, exit 0 when they agree (no GPU call)
 *   layer_fwd_c DIR            read DIR/shape.txt ("S D E K F") and the raw
 *                              little-endian arrays DIR/x.bin (bf16 [S, D]),
 *                              Wr.bin (fp32 [D, E]), W1.bin (bf16 [E, D, F]),
 *                              W2.bin (bf16 [E, F, D]); write DIR/y.bin (bf16
 *                              [S, D]), logits.bin (fp32 [S, E]) and
 *                              topk_idx.bin (int32 [S, K])
 *
 * Before the layer call it checks that an invalid request (K > E) returns
 * MOE_ERR_SHAPE and that a workspace one byte short returns
 * MOE_ERR_WORKSPACE.  Exit status 0 on success, 1 on any failure (with a
 * message on stderr). */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "moe.h"

#define CHECK_HIP(call)                                                              \
    do {                                                                             \
        hipError_t e_ = (call);                                                      \
        if (e_ != hipSuccess) {                                                      \
            fprintf(stderr, "%s failed: %s\n", #call, hipGetErrorString(e_));       \
            exit(1);                                                                 \
        }                                                                            \
    } while (0)

static void* read_file(const char* dir, const char* name, size_t bytes) {
    char path[4096];
    snprintf(path, sizeof path, "%s/%s", dir, name);
    FILE* f = fopen(path, "rb");
    if (!f) {
        fprintf(stderr, "cannot open %s\n", path);
        exit(1);
    }
    void* p = malloc(bytes ? bytes : 1);
    if (!p || fread(p, 1, bytes, f) != bytes) {
        fprintf(stderr, "short read: %s\n", path);
        exit(1);
    }
    fclose(f);
    return p;
}

static void write_file(const char* dir, const char* name, const void* p, size_t bytes) {
    char path[4096];
    snprintf(path, sizeof path, "%s/%s", dir, name);
    FILE* f = fopen(path, "wb");
    if (!f || fwrite(p, 1, bytes, f) != bytes) {
        fprintf(stderr, "cannot write %s\n", path);
        exit(1);
    }
    fclose(f);
}

static void* to_device(const void* host, size_t bytes) {
    void* d = NULL;
    CHECK_HIP(hipMalloc(&d, bytes ? bytes : 1));
    if (bytes) CHECK_HIP(hipMemcpy(d, host, bytes, hipMemcpyHostToDevice));
    return d;
}

int main(int argc, char** argv) {
    if (argc != 2) {
        fprintf(stderr, "usage: %s --abi | DIR\n", argv[0]);
        return 1;
    }
    if (strcmp(argv[1], "--abi") == 0) {
        const int v = moe_abi_version();
        printf("%d %d\n", v, MOE_ABI_VERSION);
        return v == MOE_ABI_VERSION ? 0 : 1;
    }
    const char* dir = argv[1];
    long long S = 0;
    int D = 0, E = 0, K = 0, F = 0;
    {
        char path[4096];
        snprintf(path, sizeof path, "%s/shape.txt", dir);
        FILE* f = fopen(path, "r");
        if (!f || fscanf(f, "%lld %d %d %d %d", &S, &D, &E, &K, &F) != 5) {
            fprintf(stderr, "cannot read %s\n", path);
            return 1;
        }
        fclose(f);
    }
    const size_t nx = (size_t)S * D, nw = (size_t)E * D * F;
    void* hx = read_file(dir, "x.bin", nx * 2);
    void* hWr = read_file(dir, "Wr.bin", (size_t)D * E * 4);
    void* hW1 = read_file(dir, "W1.bin", nw * 2);
    void* hW2 = read_file(dir, "W2.bin", nw * 2);

    moe_layer_fwd_args a;
    memset(&a, 0, sizeof a);
    a.struct_size = sizeof a;
    a.S = S;
    a.D = D;
    a.E = E;
    a.K = K;
    a.F = F;
    a.x = (const moe_bf16*)to_device(hx, nx * 2);
    a.Wr = (const float*)to_device(hWr, (size_t)D * E * 4);
    a.W1 = (const moe_bf16*)to_device(hW1, nw * 2);
    a.W2 = (const moe_bf16*)to_device(hW2, nw * 2);
    CHECK_HIP(hipMalloc((void**)&a.y, nx * 2));
    CHECK_HIP(hipMalloc((void**)&a.logits, (size_t)S * E * 4));
    CHECK_HIP(hipMalloc((void**)&a.topk_idx, (size_t)S * K * 4));

    /* validation happens before anything is enqueued */
    moe_layer_fwd_args bad = a;
    bad.K = E + 1;
    if (moe_layer_fwd_workspace_bytes(&bad) != 0 || moe_layer_fwd(&bad, NULL) != MOE_ERR_SHAPE) {
        fprintf(stderr, "K > E was not rejected with MOE_ERR_SHAPE\n");
        return 1;
    }
    const size_t ws_bytes = moe_layer_fwd_workspace_bytes(&a);
    if (ws_bytes == 0) {
        fprintf(stderr, "moe_layer_fwd_workspace_bytes rejected a valid shape\n");
        return 1;
    }
    CHECK_HIP(hipMalloc(&a.ws, ws_bytes));
    a.ws_bytes = ws_bytes - 1;
    if (moe_layer_fwd(&a, NULL) != MOE_ERR_WORKSPACE) {
        fprintf(stderr, "a short workspace was not rejected with MOE_ERR_WORKSPACE\n");
        return 1;
    }
    a.ws_bytes = ws_bytes;

    hipStream_t st;
    CHECK_HIP(hipStreamCreate(&st));
    const int rc = moe_layer_fwd(&a, st);
    if (rc != MOE_OK) {
        fprintf(stderr, "moe_layer_fwd returned %d\n", rc);
        return 1;
    }
    CHECK_HIP(hipStreamSynchronize(st));

    void* hy = malloc(nx * 2);
    void* hl = malloc((size_t)S * E * 4);
    void* hi = malloc((size_t)S * K * 4);
    CHECK_HIP(hipMemcpy(hy, a.y, nx * 2, hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(hl, a.logits, (size_t)S * E * 4, hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(hi, a.topk_idx, (size_t)S * K * 4, hipMemcpyDeviceToHost));
    write_file(dir, "y.bin", hy, nx * 2);
    write_file(dir, "logits.bin", hl, (size_t)S * E * 4);
    write_file(dir, "topk_idx.bin", hi, (size_t)S * K * 4);

    CHECK_HIP(hipStreamDestroy(st));
    CHECK_HIP(hipFree((void*)a.x));
    CHECK_HIP(hipFree((void*)a.Wr));
    CHECK_HIP(hipFree((void*)a.W1));
    CHECK_HIP(hipFree((void*)a.W2));
    CHECK_HIP(hipFree(a.y));
    CHECK_HIP(hipFree(a.logits));
    CHECK_HIP(hipFree(a.topk_idx));
    CHECK_HIP(hipFree(a.ws));
    free(hx);
    free(hWr);
    free(hW1);
    free(hW2);
    free(hy);
    free(hl);
    free(hi);
    printf("ok\n");
    return 0;
}
