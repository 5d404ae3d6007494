"""CPU checks of the C ABI boundary: the library loads, exports every entry
point include/moe.h declares, and rejects bad arguments synchronously.

Only host-side paths run here: every call below fails validation (or is a
pure size query) before anything is enqueued, so no GPU is touched.
"""
import ctypes as C
import re
from pathlib import Path

import pytest

from paper_2608_28511_amd import _lib as L

ROOT = Path(__file__).resolve().parents[1]
FAKE = C.c_void_p(0x10000)        # 16-byte aligned, never dereferenced
ODD = C.c_void_p(0x10002)         # misaligned for 4- and 16-byte rules


def _declared():
    text = (ROOT / "include" / "moe.h").read_text()
    return sorted(set(re.findall(r"^\s*(?:int|size_t|uint64_t|const char\*)\s+(moe_\w+)\(",
                                 text, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    return L.load(build_if_missing=True)


def test_every_declared_symbol_is_exported(lib):
    names = _declared()
    assert len(names) >= 17
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(L.EXPORTED)


def test_version_status_payload(lib):
    assert L.moe_abi_version() == 5
    assert L.moe_status_string(0) == "ok"
    for code in range(-6, 0):
        assert L.moe_status_string(code) not in ("ok", "unknown status")
    assert L.moe_status_string(-99) == "unknown status"
    # Eq. 1: S*K*(D*b_x + b_p)
    assert L.moe_payload_bytes(8192, 6, 2048) == 8192 * 6 * (2048 * 2 + 4) == 201_523_200
    assert L.moe_payload_bytes(16384, 8, 2048) == 16384 * 8 * (2048 * 2 + 4)
    assert L.moe_payload_bytes(-1, 2, 8) == 0
    # MX-FP8 hidden payload: b_x = 1 + 1/32
    assert L.moe_mx_payload_bytes(8192, 6, 2048) == 8192 * 6 * (2048 + 64 + 4) == 104_005_632
    assert L.moe_mx_payload_bytes(8192, 6, 2040) == 0
    # scale allocation read by the MX up projection: whole 4-byte words
    assert L.moe_mx_scale_alloc_bytes(3, 96) == 12 and L.moe_mx_scale_alloc_bytes(111, 96) == 336
    assert L.moe_mx_scale_alloc_bytes(49152, 2048) == 49152 * 64
    assert L.moe_mx_scale_alloc_bytes(4, 48) == 0 and L.moe_mx_scale_alloc_bytes(-1, 64) == 0


def test_workspace_queries(lib):
    assert lib.moe_route_workspace_bytes(16384, 128, 8) >= 128 * (16384 // 32)   # one count byte per expert and block
    assert lib.moe_route_workspace_bytes(10, 4, 5) == 0          # K > E
    assert lib.moe_route_workspace_bytes(10, 2048, 2) == 0       # E > 1024
    assert lib.moe_route_workspace_bytes(10, 64, 33) == 0        # K > 32
    assert lib.moe_route_workspace_bytes(2 ** 28, 64, 8) == 0    # S*K >= 2^31
    assert lib.moe_router_logits_workspace_bytes(2048, 64) == 3 * 2048 * 64 * 2
    assert lib.moe_router_logits_workspace_bytes(1032, 37) == (3 * 1032 * 37 * 2 + 255) // 256 * 256
    assert lib.moe_router_logits_workspace_bytes(2044, 64) == 0   # D % 8
    assert lib.moe_router_logits_workspace_bytes(64, 0) == 0
    assert lib.moe_router_bwd_workspace_bytes(8192, 2048, 64) >= 8192 * 64 * 4 + 8192 * 192 * 2
    assert lib.moe_router_bwd_workspace_bytes(8192, 2044, 64) == 0
    assert lib.moe_latent_proj_bwd_workspace_bytes(16384, 4096, 1024) >= 4096 * 1024 * 4
    assert lib.moe_latent_proj_bwd_workspace_bytes(16384, 4096, 1020) == 0
    assert lib.moe_grouped_ffn_workspace_bytes(64, 49152, 2048, 1024) > 0
    assert lib.moe_grouped_ffn_workspace_bytes(64, 49152, 2044, 1024) == 0   # D % 8
    assert lib.moe_grouped_ffn_bwd_workspace_bytes(8, 100, 64, 64) >= 100 * 64 * 2
    # schedule: E+1 tile starts plus one 16-byte entry per possible 128-row tile
    assert lib.moe_grouped_schedule_bytes(64, 49152) >= 65 * 4 + (384 + 64) * 16
    assert lib.moe_grouped_schedule_bytes(0, 10) == 0
    # production router: balance-loss partials per 64-token chunk; the sigmoid
    # backward also holds the six-plane dx operands
    assert lib.moe_seq_aux_loss_workspace_bytes(16384, 192, 8192) >= 2 * 128 * 192 * 8
    assert lib.moe_seq_aux_loss_workspace_bytes(1000, 8, 300) == 0          # seq_len must divide S
    assert lib.moe_seq_aux_loss_workspace_bytes(1000, 8, 0) == 0
    assert (lib.moe_router_bwd_sigmoid_workspace_bytes(8192, 2048, 64)
            >= lib.moe_router_bwd_workspace_bytes(8192, 2048, 64) + 8192 * 384 * 2 + 2048 * 384 * 2)
    assert lib.moe_shared_expert_bwd_workspace_bytes(1024, 256, 512) >= 1024 * 512 * 2 + 256 * 512 * 4
    assert lib.moe_shared_expert_bwd_workspace_bytes(1024, 256, 500) == 0   # Fs % 8


def test_layer_struct_layout_matches(lib):
    a = L.LayerFwdArgs()
    a.struct_size = C.sizeof(L.LayerFwdArgs)
    a.S, a.H, a.D, a.E, a.K, a.F = 512, 0, 256, 8, 2, 512
    n = L.moe_layer_fwd_workspace_bytes(a)
    R = 512 * 2
    # y_disp + h at least; x_disp is not carved: with it unexported the dispatch
    # is fused into the up projection, which gathers from x
    assert R * 256 * 2 + R * 512 * 2 <= n < R * 256 * 2 * 2 + R * 512 * 2
    a.struct_size += 8
    assert L.moe_layer_fwd_workspace_bytes(a) == 0
    a.struct_size -= 8
    a.H = 12                                      # not a multiple of 8
    assert L.moe_layer_fwd_workspace_bytes(a) == 0


# The base layout of moe_layer_fwd_args, field for field, in the order the
# boundary of the layer forward lists them: sizes, weights, output, the
# optional exported intermediates, then the workspace.
BOUNDARY_LAYER_FIELDS = [
    "struct_size", "S", "H", "D", "E", "K", "F", "x", "Wr", "router_bias", "Wdown", "W1", "W2", "Wup", "y",
    "logits", "topk_idx", "topk_prob", "counts", "offsets", "perm", "inv_perm", "x_disp", "p_disp", "h",
    "u_save", "y_disp", "ws", "ws_bytes"]


def _c_offsets(tmp_path, fields):
    """offsetof of each field of moe_layer_fwd_args, sizeof and the base size,
    from a host C program compiled against include/moe.h."""
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    src = tmp_path / "off.c"
    lines = ["#include <stdio.h>", '#include "moe.h"', "int main(void) {"]
    for f in fields:
        lines.append(f'  printf("{f} %zu\\n", offsetof(moe_layer_fwd_args, {f}));')
    lines += ['  printf("sizeof %zu\\n", sizeof(moe_layer_fwd_args));',
              '  printf("base %zu\\n", (size_t)MOE_LAYER_FWD_ARGS_BASE_SIZE);', "  return 0;", "}"]
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "off"
    subprocess.run(["gcc", "-std=c99", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-I", str(ROOT / "include"),
                    str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    return {k: int(v) for k, v in (ln.split() for ln in out if ln)}


def test_layer_args_layout_follows_the_boundary(lib, tmp_path):
    full = [f for f, _ in L.LayerFwdArgs._fields_]
    assert full[:len(BOUNDARY_LAYER_FIELDS)] == BOUNDARY_LAYER_FIELDS
    c = _c_offsets(tmp_path, full)
    for f in full:
        assert getattr(L.LayerFwdArgs, f).offset == c[f], f
    assert C.sizeof(L.LayerFwdArgs) == c["sizeof"]
    # the base layout ends at ws_bytes; every extension follows it
    assert c["base"] == C.sizeof(L.LayerFwdBaseArgs) == L.LayerFwdArgs.x_lat.offset
    assert [f for f, _ in L.LayerFwdBaseArgs._fields_] == BOUNDARY_LAYER_FIELDS
    # a caller that fills only the base layout gets the plain softmax layer
    b = L.LayerFwdBaseArgs()
    b.struct_size = C.sizeof(L.LayerFwdBaseArgs)
    b.S, b.H, b.D, b.E, b.K, b.F = 512, 0, 256, 8, 2, 512
    a = L.LayerFwdArgs()
    a.struct_size = C.sizeof(L.LayerFwdArgs)
    a.S, a.H, a.D, a.E, a.K, a.F = 512, 0, 256, 8, 2, 512
    pb = C.cast(C.pointer(b), C.POINTER(L.LayerFwdArgs))
    n = lib.moe_layer_fwd_workspace_bytes(pb)
    assert n > 0 and n == lib.moe_layer_fwd_workspace_bytes(C.byref(a))
    b.struct_size += 8
    assert lib.moe_layer_fwd_workspace_bytes(pb) == 0
    assert lib.moe_layer_fwd(pb, None) == -2


def test_validation_errors_return_before_launch(lib):
    st = None
    # route: bad shapes, null and misaligned pointers, short workspace
    assert lib.moe_route_topk(FAKE, 4, 8, 9, *[FAKE] * 6, FAKE, 1 << 20, st) == -2
    assert lib.moe_route_topk(None, 4, 8, 2, *[FAKE] * 6, FAKE, 1 << 20, st) == -1
    assert lib.moe_route_topk(FAKE, 4, 8, 2, ODD, *[FAKE] * 5, FAKE, 1 << 20, st) == -3
    assert lib.moe_route_topk(FAKE, 4, 8, 2, *[FAKE] * 6, FAKE, 4, st) == -4
    assert lib.moe_route_topk(FAKE, 4, 8, 2, *[FAKE] * 6, None, 1 << 20, st) == -4
    assert lib.moe_route_topk(FAKE, -1, 8, 2, *[FAKE] * 6, FAKE, 1 << 20, st) == -2
    # dispatch: D % 8, prob / p_disp must be both given or both NULL, alignment
    assert lib.moe_dispatch(FAKE, FAKE, FAKE, 4, 12, 2, FAKE, FAKE, st) == -2
    assert lib.moe_dispatch(FAKE, None, FAKE, 4, 16, 2, FAKE, FAKE, st) == -1
    assert lib.moe_dispatch(C.c_void_p(0x10008), FAKE, FAKE, 4, 16, 2, FAKE, FAKE, st) == -3
    # combine / grouped ffn / latent / backward
    assert lib.moe_combine(FAKE, None, FAKE, 4, 16, 0, FAKE, st) == -2
    assert lib.moe_combine(FAKE, None, None, 4, 16, 2, FAKE, st) == -1
    assert lib.moe_grouped_ffn(FAKE, FAKE, 0, 4, 16, 16, FAKE, FAKE, FAKE, None, FAKE, FAKE, 4096, st) == -2
    assert lib.moe_grouped_ffn(FAKE, FAKE, 2, 4, 16, 16, FAKE, FAKE, FAKE, None, FAKE, FAKE, 0, st) == -4
    assert lib.moe_grouped_ffn(FAKE, FAKE, 2, 4, 16, 16, FAKE, FAKE, FAKE, ODD, FAKE, FAKE, 4096, st) == -3
    assert lib.moe_latent_proj(FAKE, FAKE, 4, 20, 16, FAKE, st) == -2
    # operands whose DMA descriptor range would reach 2^31 bytes
    assert lib.moe_latent_proj(FAKE, FAKE, 4, 65536, 16384, FAKE, st) == -6
    assert lib.moe_grouped_gemm(FAKE, FAKE, 2, 4, 65536, 16384, FAKE, 0, FAKE, None, st) == -6
    assert lib.moe_grouped_ffn(FAKE, FAKE, 2, 4, 65536, 16384, FAKE, FAKE, FAKE, None, FAKE, FAKE,
                               4096, st) == -6
    assert lib.moe_grouped_ffn_bwd(FAKE, FAKE, FAKE, FAKE, FAKE, 2, 1 << 20, 2048, 1024, FAKE, FAKE, FAKE,
                                   FAKE, FAKE, FAKE, 1 << 40, st) == -6
    assert lib.moe_grouped_schedule(FAKE, 4, 100, FAKE, 16, st) == -4
    # the entry point without a workspace: rows beyond its fixed array are refused on the host
    assert lib.moe_grouped_ffn_static(FAKE, FAKE, 4, 1 << 21, 16, 16, FAKE, FAKE, FAKE, None, FAKE, st) == -4
    assert lib.moe_grouped_ffn_static(FAKE, FAKE, 0, 4, 16, 16, FAKE, FAKE, FAKE, None, FAKE, st) == -2
    assert lib.moe_grouped_ffn_static(FAKE, FAKE, 4, 4, 16, 16, FAKE, FAKE, FAKE, ODD, FAKE, st) == -3
    assert lib.moe_grouped_gemm(FAKE, None, 2, 4, 16, 16, FAKE, 1, FAKE, None, st) == -1
    # the gathering up projection: R must be S * K; the router input must fit one descriptor
    assert lib.moe_grouped_gemm_gather(FAKE, FAKE, 4, 2, FAKE, 2, 9, 16, 16, FAKE, 1, FAKE, None, st) == -2
    assert lib.moe_grouped_gemm_gather(FAKE, FAKE, 1 << 20, 2, FAKE, 2, 1 << 21, 2048, 16, FAKE, 1, FAKE, None,
                                       st) == -6
    assert lib.moe_grouped_gemm_gather(FAKE, None, 4, 2, FAKE, 2, 8, 16, 16, FAKE, 1, FAKE, None, st) == -1
    assert lib.moe_grouped_gemm(FAKE, FAKE, 2, 4, 16, 16, FAKE, 2, FAKE, None, st) == -6
    assert lib.moe_router_logits(FAKE, FAKE, None, 4, 16, 0, FAKE, FAKE, 4096, st) == -2
    assert lib.moe_router_logits(FAKE, FAKE, ODD, 4, 16, 4, FAKE, FAKE, 4096, st) == -3
    assert lib.moe_router_logits(FAKE, FAKE, None, 4, 16, 4, FAKE, None, 4096, st) == -4
    assert lib.moe_router_logits(FAKE, FAKE, None, 4, 16, 4, FAKE, FAKE, 8, st) == -4
    assert lib.moe_combine_bwd(FAKE, FAKE, None, FAKE, 4, 16, 33, FAKE, None, st) == -2
    assert lib.moe_grouped_ffn_bwd(FAKE, None, FAKE, FAKE, FAKE, 2, 4, 16, 16, FAKE, FAKE, FAKE,
                                   FAKE, FAKE, FAKE, 1 << 20, st) == -1
    assert lib.moe_grouped_ffn_bwd(FAKE, FAKE, FAKE, FAKE, FAKE, 2, 4, 16, 16, FAKE, FAKE, FAKE,
                                   FAKE, FAKE, FAKE, 8, st) == -4
    assert lib.moe_dispatch_bwd(FAKE, FAKE, 4, 16, 40, FAKE, st) == -2
    assert lib.moe_dispatch_bwd(FAKE, None, 4, 16, 2, FAKE, st) == -1
    assert lib.moe_dispatch_bwd(FAKE, FAKE, 4, 16, 2, ODD, st) == -3
    assert lib.moe_dispatch_bwd_add(FAKE, FAKE, ODD, 4, 16, 2, FAKE, st) == -3
    assert lib.moe_dispatch_bwd_add(FAKE, FAKE, None, 4, 16, 2, FAKE, st) == -1
    # router / latent backward
    assert lib.moe_router_bwd(FAKE, FAKE, FAKE, FAKE, FAKE, 4, 16, 8, 9, None, FAKE, None, None, FAKE,
                              1 << 20, st) == -2                       # K > E
    assert lib.moe_router_bwd(FAKE, FAKE, FAKE, FAKE, FAKE, 4, 16, 8, 2, None, FAKE, None, None, FAKE,
                              8, st) == -4                             # workspace too small
    assert lib.moe_router_bwd(FAKE, FAKE, FAKE, FAKE, FAKE, 4, 16, 8, 2, None, FAKE, None, ODD, FAKE,
                              1 << 20, st) == -3                       # dx_r must be 16-byte aligned
    assert lib.moe_latent_proj_bwd(FAKE, FAKE, FAKE, 4, 16, 12, FAKE, None, None, 0, st) == -2
    assert lib.moe_latent_proj_bwd(FAKE, FAKE, FAKE, 4, 16, 16, None, FAKE, None, 0, st) == -4
    assert lib.moe_latent_proj_bwd(FAKE, FAKE, FAKE, 4, 65536, 16384, FAKE, None, None, 0, st) == -6
    # layer: null args, wrong struct size, latent weights without H
    assert lib.moe_layer_fwd(None, st) == -1
    a = L.LayerFwdArgs()
    a.struct_size = 4
    assert lib.moe_layer_fwd(C.byref(a), st) == -2
    a.struct_size = C.sizeof(L.LayerFwdArgs)
    a.S, a.H, a.D, a.E, a.K, a.F = 4, 0, 16, 4, 2, 16
    for f in ("x", "Wr", "W1", "W2", "y", "Wdown"):
        setattr(a, f, 0x10000)
    a.ws, a.ws_bytes = 0x10000, 1 << 30
    assert lib.moe_layer_fwd(C.byref(a), st) == -2       # Wdown given with H == 0
    a.Wdown = None
    a.ws_bytes = 16
    assert lib.moe_layer_fwd(C.byref(a), st) == -4       # workspace too small
    a.ws_bytes = 1 << 30
    a.sel_bias = 0x10000
    assert lib.moe_layer_fwd(C.byref(a), st) == -2       # selection bias with softmax scores
    a.score_fn = 1
    a.seq_len = 3
    assert lib.moe_layer_fwd(C.byref(a), st) == -2       # seq_len does not divide S
    a.seq_len = 2
    assert lib.moe_layer_fwd(C.byref(a), st) == -1       # balance loss without its output
    a.seq_len = 0
    a.Fs = 12
    assert lib.moe_layer_fwd(C.byref(a), st) == -2       # shared width not a multiple of 8
    a.Fs, a.H = 16, 16
    assert lib.moe_layer_fwd_workspace_bytes(C.byref(a)) == 0  # shared expert with a latent layer
    a.H = 0
    assert lib.moe_layer_fwd(C.byref(a), st) == -1       # shared expert without its weights
    a.score_fn = 7
    assert lib.moe_layer_fwd(C.byref(a), st) == -2
    a.score_fn, a.Fs = 0, 0
    a.payload = 2
    assert lib.moe_layer_fwd(C.byref(a), st) == -2       # unknown payload format
    a.payload = 1                                         # MX-FP8 needs D % 32 == 0 (D = 16 here)
    assert lib.moe_layer_fwd(C.byref(a), st) == -2


def test_production_validation_errors(lib):
    st = None
    # MX-FP8 payload: D a multiple of 32, x_q 8-byte aligned, both outputs required
    assert lib.moe_dispatch_mxfp8(FAKE, FAKE, FAKE, 4, 48, 2, FAKE, FAKE, FAKE, st) == -2
    assert lib.moe_dispatch_mxfp8(FAKE, FAKE, FAKE, 4, 64, 2, FAKE, None, FAKE, st) == -1
    assert lib.moe_dispatch_mxfp8(FAKE, FAKE, FAKE, 4, 64, 2, C.c_void_p(0x10004), FAKE, FAKE, st) == -3
    assert lib.moe_dispatch_mxfp8(FAKE, None, FAKE, 4, 64, 2, FAKE, FAKE, FAKE, st) == -1
    assert lib.moe_mxfp8_dequant(FAKE, FAKE, 4, 40, FAKE, st) == -2
    assert lib.moe_mxfp8_dequant(FAKE, None, 4, 64, FAKE, st) == -1
    # MX-FP8 up projection: Kd a multiple of 32, 16-byte aligned codes, scale
    # and schedule given, epilogue 0 or 1, weights within the descriptor range
    assert lib.moe_grouped_gemm_mxfp8(FAKE, FAKE, FAKE, 2, 4, 48, 16, FAKE, 1, FAKE, None, st) == -2
    assert lib.moe_grouped_gemm_mxfp8(C.c_void_p(0x10008), FAKE, FAKE, 2, 4, 64, 16, FAKE, 1, FAKE, None,
                                      st) == -3
    assert lib.moe_grouped_gemm_mxfp8(FAKE, None, FAKE, 2, 4, 64, 16, FAKE, 1, FAKE, None, st) == -1
    assert lib.moe_grouped_gemm_mxfp8(FAKE, FAKE, None, 2, 4, 64, 16, FAKE, 1, FAKE, None, st) == -1
    assert lib.moe_grouped_gemm_mxfp8(FAKE, FAKE, FAKE, 2, 4, 64, 16, FAKE, 2, FAKE, None, st) == -6
    assert lib.moe_grouped_gemm_mxfp8(FAKE, FAKE, FAKE, 2, 4, 64, 16, FAKE, 0, FAKE, FAKE, st) == -2
    assert lib.moe_grouped_gemm_mxfp8(FAKE, FAKE, FAKE, 2, 4, 65536, 16384, FAKE, 0, FAKE, None, st) == -6
    assert lib.moe_grouped_gemm_mxfp8(FAKE, FAKE, FAKE, 2, 0, 64, 16, FAKE, 1, FAKE, None, st) == 0
    assert lib.moe_route_sigmoid(FAKE, None, 4, 8, 9, *[FAKE] * 6, FAKE, 1 << 20, st) == -2
    assert lib.moe_route_sigmoid(FAKE, ODD, 4, 8, 2, *[FAKE] * 6, FAKE, 1 << 20, st) == -3
    assert lib.moe_route_sigmoid(FAKE, None, 4, 8, 2, *[FAKE] * 6, FAKE, 4, st) == -4
    assert lib.moe_seq_aux_loss(FAKE, FAKE, 10, 8, 2, 3, 1e-4, FAKE, None, FAKE, 1 << 20, st) == -2
    assert lib.moe_seq_aux_loss(FAKE, FAKE, 10, 8, 2, 5, 1e-4, None, None, FAKE, 1 << 20, st) == -1
    assert lib.moe_seq_aux_loss(FAKE, FAKE, 10, 8, 2, 5, 1e-4, FAKE, None, FAKE, 8, st) == -4
    args = [FAKE] * 7 + [5, 1e-4, 10, 16, 8, 2, None, FAKE, None, None, FAKE, 1 << 24, st]
    bad = list(args)
    bad[7] = 3                                              # seq_len does not divide S
    assert lib.moe_router_bwd_sigmoid(*bad) == -2
    bad = list(args)
    bad[-2] = 8                                             # workspace too small
    assert lib.moe_router_bwd_sigmoid(*bad) == -4
    bad = list(args)
    bad[12] = 9                                             # K > E
    assert lib.moe_router_bwd_sigmoid(*bad) == -2
    assert lib.moe_expert_bias_update(FAKE, 0, 1e-3, FAKE, st) == -2
    assert lib.moe_expert_bias_update(FAKE, 8, 1e-3, None, st) == -1
    assert lib.moe_combine_add(FAKE, None, FAKE, ODD, 4, 16, 2, FAKE, st) == -3
    assert lib.moe_combine_add(FAKE, None, FAKE, None, 4, 16, 2, FAKE, st) == -1
    assert lib.moe_shared_expert_fwd(FAKE, FAKE, FAKE, 4, 16, 12, FAKE, None, FAKE, st) == -2
    assert lib.moe_shared_expert_fwd(FAKE, FAKE, FAKE, 4, 65536, 16384, FAKE, None, FAKE, st) == -6
    assert lib.moe_shared_expert_fwd(FAKE, FAKE, FAKE, 4, 16, 16, FAKE, ODD, FAKE, st) == -3
    assert lib.moe_shared_expert_bwd(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 4, 16, 16, None, 0, FAKE, FAKE,
                                     FAKE, 8, st) == -4
    assert lib.moe_shared_expert_bwd(FAKE, None, FAKE, FAKE, FAKE, FAKE, 4, 16, 16, None, 0, FAKE, FAKE,
                                     FAKE, 1 << 20, st) == -1


def test_binding_refuses_host_tensors():
    import torch
    with pytest.raises(ValueError):
        L._ptr(torch.zeros(4), torch.float32, "x")
    with pytest.raises(TypeError):
        L._ptr([1, 2], torch.float32, "x")


def test_c_consumer_reports_the_header_abi_version(lib):
    """The plain C consumer (tests/c_abi/layer_fwd_c.c, gcc, no Python) links
    against libmoe.so and reads the same ABI version as its header (no GPU
    call on this path)."""
    import importlib.util
    import subprocess

    spec = importlib.util.spec_from_file_location("c_abi_build", ROOT / "tests" / "c_abi" / "build.py")
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    exe = mod.ensure_built()
    r = subprocess.run([str(exe), "--abi"], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stderr
    assert r.stdout.split() == [str(L.moe_abi_version())] * 2
