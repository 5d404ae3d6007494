"""ctypes binding of libmoe.so (the C ABI in include/moe.h).

Argument marshalling only: every function here has the name of the C entry
point it wraps, takes torch tensors (or None where the C argument may be
NULL), checks that each tensor is a contiguous device tensor of the dtype
the C side expects (so a host pointer can never reach a kernel), and passes
raw pointers plus the current HIP stream.  A negative status raises
``MoeError``.  All arithmetic happens in the HIP kernels; if the library is
missing this module raises instead of falling back to anything.
"""
from __future__ import annotations

import ctypes as C
from pathlib import Path
from typing import Optional

import torch

LIB_PATH = Path(__file__).resolve().parent / "libmoe.so"

_lib: Optional[C.CDLL] = None

vp = C.c_void_p
i32 = C.c_int32
i64 = C.c_int64
u32 = C.c_uint32
sz = C.c_size_t


class MoeError(RuntimeError):
    def __init__(self, code: int, text: str, where: str):
        super().__init__(f"{where}: {text} (status {code})")
        self.code = code


# Fields of moe_layer_fwd_args up to ws_bytes (the base layout).
LAYER_FWD_BASE_FIELDS = [
    ("struct_size", u32), ("S", i64), ("H", i32), ("D", i32), ("E", i32), ("K", i32),
    ("F", i32),
    ("x", vp), ("Wr", vp), ("router_bias", vp), ("Wdown", vp), ("W1", vp), ("W2", vp),
    ("Wup", vp), ("y", vp),
    ("logits", vp), ("topk_idx", vp), ("topk_prob", vp), ("counts", vp),
    ("offsets", vp), ("perm", vp), ("inv_perm", vp), ("x_disp", vp), ("p_disp", vp),
    ("h", vp), ("u_save", vp), ("y_disp", vp),
    ("ws", vp), ("ws_bytes", sz),
]


class LayerFwdBaseArgs(C.Structure):
    """Mirror of the base layout of moe_layer_fwd_args (struct_size =
    MOE_LAYER_FWD_ARGS_BASE_SIZE)."""
    _fields_ = LAYER_FWD_BASE_FIELDS


class LayerFwdArgs(C.Structure):
    """Mirror of moe_layer_fwd_args."""
    _fields_ = LAYER_FWD_BASE_FIELDS + [
        ("x_lat", vp), ("y_lat", vp),
        ("score_fn", i32), ("Fs", i32), ("sel_bias", vp), ("Ws1", vp), ("Ws2", vp),
        ("seq_len", i64), ("aux_coeff", C.c_float), ("aux_loss", vp), ("seq_counts", vp),
        ("h_s", vp), ("u_s", vp), ("y_s", vp),
        ("payload", i32), ("x_q", vp), ("x_scale", vp),
    ]


SCORE_SOFTMAX, SCORE_SIGMOID = 0, 1
PAYLOAD_BF16, PAYLOAD_MXFP8 = 0, 1
U8 = torch.uint8


_PROTOS = {
    "moe_abi_version": (C.c_int, []),
    "moe_status_string": (C.c_char_p, [C.c_int]),
    "moe_payload_bytes": (C.c_uint64, [i64, i32, i32]),
    "moe_router_logits_workspace_bytes": (sz, [i32, i32]),
    "moe_router_logits": (C.c_int, [vp, vp, vp, i64, i32, i32, vp, vp, sz, vp]),
    "moe_route_workspace_bytes": (sz, [i64, i32, i32]),
    "moe_route_topk": (C.c_int, [vp, i64, i32, i32, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
    "moe_dispatch": (C.c_int, [vp, vp, vp, i64, i32, i32, vp, vp, vp]),
    "moe_grouped_ffn_workspace_bytes": (sz, [i32, i64, i32, i32]),
    "moe_grouped_ffn": (C.c_int, [vp, vp, i32, i64, i32, i32, vp, vp, vp, vp, vp, vp, sz, vp]),
    "moe_grouped_ffn_static": (C.c_int, [vp, vp, i32, i64, i32, i32, vp, vp, vp, vp, vp, vp]),
    "moe_grouped_schedule_bytes": (sz, [i32, i64]),
    "moe_grouped_schedule": (C.c_int, [vp, i32, i64, vp, sz, vp]),
    "moe_grouped_gemm": (C.c_int, [vp, vp, i32, i64, i32, i32, vp, i32, vp, vp, vp]),
    "moe_grouped_gemm_gather": (C.c_int, [vp, vp, i64, i32, vp, i32, i64, i32, i32, vp, i32, vp, vp, vp]),
    "moe_combine": (C.c_int, [vp, vp, vp, i64, i32, i32, vp, vp]),
    "moe_latent_proj": (C.c_int, [vp, vp, i64, i32, i32, vp, vp]),
    "moe_layer_fwd_workspace_bytes": (sz, [C.POINTER(LayerFwdArgs)]),
    "moe_layer_fwd": (C.c_int, [C.POINTER(LayerFwdArgs), vp]),
    "moe_combine_bwd": (C.c_int, [vp, vp, vp, vp, i64, i32, i32, vp, vp, vp]),
    "moe_grouped_ffn_bwd_workspace_bytes": (sz, [i32, i64, i32, i32]),
    "moe_grouped_ffn_bwd": (C.c_int, [vp, vp, vp, vp, vp, i32, i64, i32, i32, vp, vp, vp, vp, vp,
                                      vp, sz, vp]),
    "moe_dispatch_bwd": (C.c_int, [vp, vp, i64, i32, i32, vp, vp]),
    "moe_dispatch_bwd_add": (C.c_int, [vp, vp, vp, i64, i32, i32, vp, vp]),
    "moe_router_bwd_workspace_bytes": (sz, [i64, i32, i32]),
    "moe_router_bwd": (C.c_int, [vp, vp, vp, vp, vp, i64, i32, i32, i32, vp, vp, vp, vp, vp, sz, vp]),
    "moe_latent_proj_bwd_workspace_bytes": (sz, [i64, i32, i32]),
    "moe_latent_proj_bwd": (C.c_int, [vp, vp, vp, i64, i32, i32, vp, vp, vp, sz, vp]),
    "moe_route_sigmoid": (C.c_int, [vp, vp, i64, i32, i32, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
    "moe_seq_aux_loss_workspace_bytes": (sz, [i64, i32, i64]),
    "moe_seq_aux_loss": (C.c_int, [vp, vp, i64, i32, i32, i64, C.c_float, vp, vp, vp, sz, vp]),
    "moe_router_bwd_sigmoid_workspace_bytes": (sz, [i64, i32, i32]),
    "moe_router_bwd_sigmoid": (C.c_int, [vp, vp, vp, vp, vp, vp, vp, i64, C.c_float, i64, i32, i32, i32,
                                         vp, vp, vp, vp, vp, sz, vp]),
    "moe_expert_bias_update": (C.c_int, [vp, i32, C.c_float, vp, vp]),
    "moe_combine_add": (C.c_int, [vp, vp, vp, vp, i64, i32, i32, vp, vp]),
    "moe_shared_expert_fwd": (C.c_int, [vp, vp, vp, i64, i32, i32, vp, vp, vp, vp]),
    "moe_shared_expert_bwd_workspace_bytes": (sz, [i64, i32, i32]),
    "moe_mx_payload_bytes": (C.c_uint64, [i64, i32, i32]),
    "moe_dispatch_mxfp8": (C.c_int, [vp, vp, vp, i64, i32, i32, vp, vp, vp, vp]),
    "moe_mxfp8_dequant": (C.c_int, [vp, vp, i64, i32, vp, vp]),
    "moe_mx_scale_alloc_bytes": (C.c_uint64, [i64, i32]),
    "moe_grouped_gemm_mxfp8": (C.c_int, [vp, vp, vp, i32, i64, i32, i32, vp, i32, vp, vp, vp]),
    "moe_shared_expert_bwd": (C.c_int, [vp, vp, vp, vp, vp, vp, i64, i32, i32, vp, i32, vp, vp, vp, sz, vp]),
}

EXPORTED = tuple(_PROTOS)


def load(build_if_missing: bool = False) -> C.CDLL:
    """Load libmoe.so from the package directory (building it first only if
    asked and absent).  Raises if it cannot be loaded."""
    global _lib
    if _lib is not None:
        return _lib
    if not LIB_PATH.exists():
        if not build_if_missing:
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        from . import build as _build
        _build.build()
    lib = C.CDLL(str(LIB_PATH))
    for name, (res, args) in _PROTOS.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def _check(status: int, where: str) -> None:
    if status != 0:
        raise MoeError(status, load().moe_status_string(status).decode(), where)


def _stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t: Optional[torch.Tensor], dtype=None, name: str = "tensor"):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.numel() and t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor, got {t.device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    return C.c_void_p(t.data_ptr()) if t.numel() else None


BF16, F32, I32 = torch.bfloat16, torch.float32, torch.int32


def moe_abi_version() -> int:
    return load().moe_abi_version()


def moe_status_string(status: int) -> str:
    return load().moe_status_string(status).decode()


def moe_payload_bytes(S: int, K: int, D: int) -> int:
    return load().moe_payload_bytes(S, K, D)


def moe_router_logits_workspace_bytes(D, E) -> int:
    return load().moe_router_logits_workspace_bytes(D, E)


def moe_router_logits(x_r, Wr, bias, S, D, E, logits, ws):
    _check(load().moe_router_logits(_ptr(x_r, BF16, "x_r"), _ptr(Wr, F32, "Wr"),
                                    _ptr(bias, F32, "bias"), S, D, E, _ptr(logits, F32, "logits"),
                                    _ptr(ws, None, "ws"),
                                    0 if ws is None else ws.numel() * ws.element_size(), _stream()),
           "moe_router_logits")


def moe_route_workspace_bytes(S, E, K) -> int:
    return load().moe_route_workspace_bytes(S, E, K)


def moe_route_topk(logits, S, E, K, topk_idx, topk_prob, counts, offsets, perm, inv_perm, ws):
    _check(load().moe_route_topk(
        _ptr(logits, F32, "logits"), S, E, K, _ptr(topk_idx, I32, "topk_idx"),
        _ptr(topk_prob, F32, "topk_prob"), _ptr(counts, I32, "counts"),
        _ptr(offsets, I32, "offsets"), _ptr(perm, I32, "perm"), _ptr(inv_perm, I32, "inv_perm"),
        _ptr(ws, None, "ws"), 0 if ws is None else ws.numel() * ws.element_size(), _stream()),
        "moe_route_topk")


def moe_dispatch(x, topk_prob, inv_perm, S, D, K, x_disp, p_disp):
    _check(load().moe_dispatch(_ptr(x, BF16, "x"), _ptr(topk_prob, F32, "topk_prob"),
                               _ptr(inv_perm, I32, "inv_perm"), S, D, K,
                               _ptr(x_disp, BF16, "x_disp"), _ptr(p_disp, F32, "p_disp"),
                               _stream()), "moe_dispatch")


def moe_grouped_ffn_workspace_bytes(E, R, D, F) -> int:
    return load().moe_grouped_ffn_workspace_bytes(E, R, D, F)


def moe_grouped_ffn(x_disp, offsets, E, R, D, F, W1, W2, h, u_save, y_disp, ws):
    _check(load().moe_grouped_ffn(
        _ptr(x_disp, BF16, "x_disp"), _ptr(offsets, I32, "offsets"), E, R, D, F,
        _ptr(W1, BF16, "W1"), _ptr(W2, BF16, "W2"), _ptr(h, BF16, "h"),
        _ptr(u_save, BF16, "u_save"), _ptr(y_disp, BF16, "y_disp"), _ptr(ws, None, "ws"),
        0 if ws is None else ws.numel() * ws.element_size(), _stream()), "moe_grouped_ffn")


def moe_grouped_ffn_static(x_disp, offsets, E, R, D, F, W1, W2, h, u_save, y_disp):
    _check(load().moe_grouped_ffn_static(
        _ptr(x_disp, BF16, "x_disp"), _ptr(offsets, I32, "offsets"), E, R, D, F,
        _ptr(W1, BF16, "W1"), _ptr(W2, BF16, "W2"), _ptr(h, BF16, "h"),
        _ptr(u_save, BF16, "u_save"), _ptr(y_disp, BF16, "y_disp"), _stream()), "moe_grouped_ffn_static")


def moe_grouped_schedule_bytes(E, R) -> int:
    return load().moe_grouped_schedule_bytes(E, R)


def moe_grouped_schedule(offsets, E, R, sched):
    _check(load().moe_grouped_schedule(_ptr(offsets, I32, "offsets"), E, R, _ptr(sched, None, "sched"),
                                       sched.numel() * sched.element_size(), _stream()),
           "moe_grouped_schedule")


def moe_grouped_gemm(A, sched, E, R, Kd, N, W, epilogue, Cout, u_save):
    _check(load().moe_grouped_gemm(_ptr(A, BF16, "A"), _ptr(sched, None, "sched"), E, R, Kd, N,
                                   _ptr(W, BF16, "W"), epilogue, _ptr(Cout, BF16, "C"),
                                   _ptr(u_save, BF16, "u_save"), _stream()), "moe_grouped_gemm")


def moe_grouped_gemm_gather(x, perm, S, K, sched, E, R, Kd, N, W, epilogue, Cout, u_save):
    _check(load().moe_grouped_gemm_gather(_ptr(x, BF16, "x"), _ptr(perm, I32, "perm"), S, K, _ptr(sched, None, "sched"),
                                          E, R, Kd, N, _ptr(W, BF16, "W"), epilogue, _ptr(Cout, BF16, "C"),
                                          _ptr(u_save, BF16, "u_save"), _stream()), "moe_grouped_gemm_gather")


def moe_combine(y_disp, p_disp, inv_perm, S, D, K, y):
    _check(load().moe_combine(_ptr(y_disp, BF16, "y_disp"), _ptr(p_disp, F32, "p_disp"),
                              _ptr(inv_perm, I32, "inv_perm"), S, D, K, _ptr(y, BF16, "y"),
                              _stream()), "moe_combine")


def moe_latent_proj(A, W, M, Kd, N, Cout):
    _check(load().moe_latent_proj(_ptr(A, BF16, "A"), _ptr(W, BF16, "W"), M, Kd, N,
                                  _ptr(Cout, BF16, "C"), _stream()), "moe_latent_proj")


_LAYER_TENSORS = {
    "x": BF16, "Wr": F32, "router_bias": F32, "Wdown": BF16, "W1": BF16, "W2": BF16, "Wup": BF16,
    "y": BF16, "x_lat": BF16, "logits": F32, "topk_idx": I32, "topk_prob": F32, "counts": I32,
    "offsets": I32, "perm": I32, "inv_perm": I32, "x_disp": BF16, "p_disp": F32, "h": BF16,
    "u_save": BF16, "y_disp": BF16, "y_lat": BF16, "sel_bias": F32, "Ws1": BF16, "Ws2": BF16,
    "aux_loss": F32, "seq_counts": I32, "h_s": BF16, "u_s": BF16, "y_s": F32,
    "x_q": torch.uint8, "x_scale": torch.uint8,
}


def layer_fwd_args(S, H, D, E, K, F, ws=None, score_fn=SCORE_SOFTMAX, Fs=0, seq_len=0, aux_coeff=0.0,
                   payload=PAYLOAD_BF16, **tensors) -> LayerFwdArgs:
    """Fill a moe_layer_fwd_args from sizes and named tensors (None = NULL)."""
    a = LayerFwdArgs()
    a.struct_size = C.sizeof(LayerFwdArgs)
    a.S, a.H, a.D, a.E, a.K, a.F = S, H, D, E, K, F
    a.score_fn, a.Fs, a.seq_len, a.aux_coeff = score_fn, Fs, seq_len, aux_coeff
    a.payload = payload
    for name, t in tensors.items():
        if name not in _LAYER_TENSORS:
            raise KeyError(name)
        p = _ptr(t, _LAYER_TENSORS[name], name)
        setattr(a, name, p.value if p is not None else None)
    if ws is not None:
        p = _ptr(ws, None, "ws")
        a.ws = p.value if p is not None else None
        a.ws_bytes = ws.numel() * ws.element_size()
    return a


def moe_layer_fwd_workspace_bytes(args: LayerFwdArgs) -> int:
    return load().moe_layer_fwd_workspace_bytes(C.byref(args))


def moe_layer_fwd(args: LayerFwdArgs):
    _check(load().moe_layer_fwd(C.byref(args), _stream()), "moe_layer_fwd")


def moe_combine_bwd(dy, y_disp, p_disp, inv_perm, S, D, K, dy_disp, dp):
    _check(load().moe_combine_bwd(_ptr(dy, BF16, "dy"), _ptr(y_disp, BF16, "y_disp"),
                                  _ptr(p_disp, F32, "p_disp"), _ptr(inv_perm, I32, "inv_perm"),
                                  S, D, K, _ptr(dy_disp, BF16, "dy_disp"), _ptr(dp, F32, "dp"),
                                  _stream()), "moe_combine_bwd")


def moe_grouped_ffn_bwd_workspace_bytes(E, R, D, F) -> int:
    return load().moe_grouped_ffn_bwd_workspace_bytes(E, R, D, F)


def moe_grouped_ffn_bwd(x_disp, u_save, h, dy_disp, offsets, E, R, D, F, W1, W2, dx_disp, dW1,
                        dW2, ws):
    _check(load().moe_grouped_ffn_bwd(
        _ptr(x_disp, BF16, "x_disp"), _ptr(u_save, BF16, "u_save"), _ptr(h, BF16, "h"),
        _ptr(dy_disp, BF16, "dy_disp"), _ptr(offsets, I32, "offsets"), E, R, D, F,
        _ptr(W1, BF16, "W1"), _ptr(W2, BF16, "W2"), _ptr(dx_disp, BF16, "dx_disp"),
        _ptr(dW1, F32, "dW1"), _ptr(dW2, F32, "dW2"), _ptr(ws, None, "ws"),
        0 if ws is None else ws.numel() * ws.element_size(), _stream()), "moe_grouped_ffn_bwd")


def moe_dispatch_bwd(dx_disp, inv_perm, S, D, K, dx):
    _check(load().moe_dispatch_bwd(_ptr(dx_disp, BF16, "dx_disp"), _ptr(inv_perm, I32, "inv_perm"), S, D, K,
                                   _ptr(dx, BF16, "dx"), _stream()), "moe_dispatch_bwd")


def moe_dispatch_bwd_add(dx_disp, inv_perm, dx_add, S, D, K, dx):
    _check(load().moe_dispatch_bwd_add(_ptr(dx_disp, BF16, "dx_disp"), _ptr(inv_perm, I32, "inv_perm"),
                                       _ptr(dx_add, F32, "dx_add"), S, D, K, _ptr(dx, BF16, "dx"), _stream()),
           "moe_dispatch_bwd_add")


def moe_router_bwd_workspace_bytes(S, D, E) -> int:
    return load().moe_router_bwd_workspace_bytes(S, D, E)


def moe_router_bwd(x_r, Wr, topk_idx, topk_prob, dp, S, D, E, K, dlogits, dWr, dbias, dx_r, ws):
    _check(load().moe_router_bwd(
        _ptr(x_r, BF16, "x_r"), _ptr(Wr, F32, "Wr"), _ptr(topk_idx, I32, "topk_idx"),
        _ptr(topk_prob, F32, "topk_prob"), _ptr(dp, F32, "dp"), S, D, E, K, _ptr(dlogits, F32, "dlogits"),
        _ptr(dWr, F32, "dWr"), _ptr(dbias, F32, "dbias"), _ptr(dx_r, F32, "dx_r"), _ptr(ws, None, "ws"),
        0 if ws is None else ws.numel() * ws.element_size(), _stream()), "moe_router_bwd")


def moe_latent_proj_bwd_workspace_bytes(M, Kd, N) -> int:
    return load().moe_latent_proj_bwd_workspace_bytes(M, Kd, N)


def moe_latent_proj_bwd(x_in, W, dout, M, Kd, N, dx_in, dW, ws):
    _check(load().moe_latent_proj_bwd(
        _ptr(x_in, BF16, "x_in"), _ptr(W, BF16, "W"), _ptr(dout, BF16, "dout"), M, Kd, N,
        _ptr(dx_in, BF16, "dx_in"), _ptr(dW, F32, "dW"), _ptr(ws, None, "ws"),
        0 if ws is None else ws.numel() * ws.element_size(), _stream()), "moe_latent_proj_bwd")


def _wsz(ws):
    return 0 if ws is None else ws.numel() * ws.element_size()


def moe_route_sigmoid(logits, sel_bias, S, E, K, topk_idx, topk_gate, counts, offsets, perm, inv_perm, ws):
    _check(load().moe_route_sigmoid(
        _ptr(logits, F32, "logits"), _ptr(sel_bias, F32, "sel_bias"), S, E, K, _ptr(topk_idx, I32, "topk_idx"),
        _ptr(topk_gate, F32, "topk_gate"), _ptr(counts, I32, "counts"), _ptr(offsets, I32, "offsets"),
        _ptr(perm, I32, "perm"), _ptr(inv_perm, I32, "inv_perm"), _ptr(ws, None, "ws"), _wsz(ws), _stream()),
        "moe_route_sigmoid")


def moe_seq_aux_loss_workspace_bytes(S, E, seq_len) -> int:
    return load().moe_seq_aux_loss_workspace_bytes(S, E, seq_len)


def moe_seq_aux_loss(logits, topk_idx, S, E, K, seq_len, coeff, loss, seq_counts, ws):
    _check(load().moe_seq_aux_loss(
        _ptr(logits, F32, "logits"), _ptr(topk_idx, I32, "topk_idx"), S, E, K, seq_len, coeff,
        _ptr(loss, F32, "loss"), _ptr(seq_counts, I32, "seq_counts"), _ptr(ws, None, "ws"), _wsz(ws), _stream()),
        "moe_seq_aux_loss")


def moe_router_bwd_sigmoid_workspace_bytes(S, D, E) -> int:
    return load().moe_router_bwd_sigmoid_workspace_bytes(S, D, E)


def moe_router_bwd_sigmoid(x_r, Wr, logits, topk_idx, topk_gate, dg, seq_counts, seq_len, coeff, S, D, E, K,
                           dlogits, dWr, dbias, dx_r, ws):
    _check(load().moe_router_bwd_sigmoid(
        _ptr(x_r, BF16, "x_r"), _ptr(Wr, F32, "Wr"), _ptr(logits, F32, "logits"), _ptr(topk_idx, I32, "topk_idx"),
        _ptr(topk_gate, F32, "topk_gate"), _ptr(dg, F32, "dg"), _ptr(seq_counts, I32, "seq_counts"), seq_len,
        coeff, S, D, E, K, _ptr(dlogits, F32, "dlogits"), _ptr(dWr, F32, "dWr"), _ptr(dbias, F32, "dbias"),
        _ptr(dx_r, F32, "dx_r"), _ptr(ws, None, "ws"), _wsz(ws), _stream()), "moe_router_bwd_sigmoid")


def moe_expert_bias_update(counts, E, rate, sel_bias):
    _check(load().moe_expert_bias_update(_ptr(counts, I32, "counts"), E, rate, _ptr(sel_bias, F32, "sel_bias"),
                                         _stream()), "moe_expert_bias_update")


def moe_combine_add(y_disp, p_disp, inv_perm, y_add, S, D, K, y):
    _check(load().moe_combine_add(_ptr(y_disp, BF16, "y_disp"), _ptr(p_disp, F32, "p_disp"),
                                  _ptr(inv_perm, I32, "inv_perm"), _ptr(y_add, F32, "y_add"), S, D, K,
                                  _ptr(y, BF16, "y"), _stream()), "moe_combine_add")


def moe_shared_expert_fwd(x, Ws1, Ws2, S, D, Fs, h_s, u_s, y_s):
    _check(load().moe_shared_expert_fwd(_ptr(x, BF16, "x"), _ptr(Ws1, BF16, "Ws1"), _ptr(Ws2, BF16, "Ws2"), S, D,
                                        Fs, _ptr(h_s, BF16, "h_s"), _ptr(u_s, BF16, "u_s"), _ptr(y_s, F32, "y_s"),
                                        _stream()), "moe_shared_expert_fwd")


def moe_shared_expert_bwd_workspace_bytes(S, D, Fs) -> int:
    return load().moe_shared_expert_bwd_workspace_bytes(S, D, Fs)


def moe_shared_expert_bwd(x, u_s, h_s, dy, Ws1, Ws2, S, D, Fs, dx, accumulate_dx, dWs1, dWs2, ws):
    _check(load().moe_shared_expert_bwd(
        _ptr(x, BF16, "x"), _ptr(u_s, BF16, "u_s"), _ptr(h_s, BF16, "h_s"), _ptr(dy, BF16, "dy"),
        _ptr(Ws1, BF16, "Ws1"), _ptr(Ws2, BF16, "Ws2"), S, D, Fs, _ptr(dx, F32, "dx"), int(bool(accumulate_dx)),
        _ptr(dWs1, F32, "dWs1"), _ptr(dWs2, F32, "dWs2"), _ptr(ws, None, "ws"), _wsz(ws), _stream()),
        "moe_shared_expert_bwd")


def moe_mx_payload_bytes(S, K, D) -> int:
    return load().moe_mx_payload_bytes(S, K, D)


def moe_dispatch_mxfp8(x, topk_prob, inv_perm, S, D, K, x_q, x_scale, p_disp):
    _check(load().moe_dispatch_mxfp8(_ptr(x, BF16, "x"), _ptr(topk_prob, F32, "topk_prob"),
                                     _ptr(inv_perm, I32, "inv_perm"), S, D, K, _ptr(x_q, U8, "x_q"),
                                     _ptr(x_scale, U8, "x_scale"), _ptr(p_disp, F32, "p_disp"), _stream()),
           "moe_dispatch_mxfp8")


def moe_mxfp8_dequant(x_q, x_scale, R, D, out):
    _check(load().moe_mxfp8_dequant(_ptr(x_q, U8, "x_q"), _ptr(x_scale, U8, "x_scale"), R, D,
                                    _ptr(out, BF16, "out"), _stream()), "moe_mxfp8_dequant")


def moe_mx_scale_alloc_bytes(R, D) -> int:
    return load().moe_mx_scale_alloc_bytes(R, D)


def moe_grouped_gemm_mxfp8(x_q, x_scale, sched, E, R, Kd, N, W, epilogue, Cout, u_save):
    if x_scale is not None and (x_scale.untyped_storage().nbytes() - x_scale.storage_offset()
                                < moe_mx_scale_alloc_bytes(R, Kd)):
        raise ValueError("x_scale's allocation must hold moe_mx_scale_alloc_bytes(R, Kd) bytes")
    _check(load().moe_grouped_gemm_mxfp8(_ptr(x_q, U8, "x_q"), _ptr(x_scale, U8, "x_scale"),
                                         _ptr(sched, None, "sched"), E, R, Kd, N, _ptr(W, BF16, "W"), epilogue,
                                         _ptr(Cout, BF16, "C"), _ptr(u_save, BF16, "u_save"), _stream()),
           "moe_grouped_gemm_mxfp8")
