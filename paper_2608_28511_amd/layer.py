"""Convenience wrappers that allocate outputs and workspace with torch and
call the C ABI through ``_lib``.  Plumbing only: no arithmetic of the layer
happens here."""
from __future__ import annotations

from typing import Dict, Optional

import torch

from . import _lib as L

BF16, F32, I32 = torch.bfloat16, torch.float32, torch.int32


def _empty(shape, dtype, device):
    return torch.empty(shape, dtype=dtype, device=device)


def _ws(nbytes: int, device) -> torch.Tensor:
    return torch.empty((max(int(nbytes), 1),), dtype=torch.uint8, device=device)


def router_logits(x_r: torch.Tensor, Wr: torch.Tensor, bias: Optional[torch.Tensor] = None):
    S, D = x_r.shape
    E = Wr.shape[1]
    out = _empty((S, E), F32, x_r.device)
    ws = _ws(L.moe_router_logits_workspace_bytes(D, E), x_r.device)
    L.moe_router_logits(x_r, Wr, bias, S, D, E, out, ws)
    return out


def route(logits: torch.Tensor, K: int) -> Dict[str, torch.Tensor]:
    S, E = logits.shape
    dev = logits.device
    R = S * K
    o = dict(topk_idx=_empty((S, K), I32, dev), topk_prob=_empty((S, K), F32, dev),
             counts=_empty((E,), I32, dev), offsets=_empty((E + 1,), I32, dev),
             perm=_empty((R,), I32, dev), inv_perm=_empty((R,), I32, dev))
    ws = _ws(L.moe_route_workspace_bytes(S, E, K), dev)
    L.moe_route_topk(logits, S, E, K, o["topk_idx"], o["topk_prob"], o["counts"], o["offsets"],
                     o["perm"], o["inv_perm"], ws)
    return o


def dispatch(x: torch.Tensor, topk_prob: Optional[torch.Tensor], inv_perm: torch.Tensor, K: int):
    S, D = x.shape
    x_disp = _empty((S * K, D), BF16, x.device)
    p_disp = _empty((S * K,), F32, x.device) if topk_prob is not None else None
    L.moe_dispatch(x, topk_prob, inv_perm, S, D, K, x_disp, p_disp)
    return x_disp, p_disp


def mx_scales(R: int, D: int, device) -> torch.Tensor:
    """uint8 [R, D/32] scale rows in an allocation padded as the MX grouped GEMM reads it."""
    nbytes = max(L.moe_mx_scale_alloc_bytes(R, D), 1)
    return _empty((nbytes,), torch.uint8, device)[: R * (D // 32)].view(R, D // 32)


def dispatch_mxfp8(x: torch.Tensor, topk_prob: Optional[torch.Tensor], inv_perm: torch.Tensor, K: int):
    """(x_q uint8 [S*K, D], x_scale uint8 [S*K, D/32], p_disp fp32 or None)."""
    S, D = x.shape
    dev = x.device
    x_q = _empty((S * K, D), torch.uint8, dev)
    x_scale = mx_scales(S * K, D, dev)
    p_disp = _empty((S * K,), F32, dev) if topk_prob is not None else None
    L.moe_dispatch_mxfp8(x, topk_prob, inv_perm, S, D, K, x_q, x_scale, p_disp)
    return x_q, x_scale, p_disp


def mxfp8_dequant(x_q: torch.Tensor, x_scale: torch.Tensor) -> torch.Tensor:
    R, D = x_q.shape
    out = _empty((R, D), BF16, x_q.device)
    L.moe_mxfp8_dequant(x_q, x_scale, R, D, out)
    return out


def grouped_ffn(x_disp: torch.Tensor, offsets: torch.Tensor, W1: torch.Tensor, W2: torch.Tensor,
                save_u: bool = False):
    R, D = x_disp.shape
    E, _, F = W1.shape
    dev = x_disp.device
    h = _empty((R, F), BF16, dev)
    u = _empty((R, F), BF16, dev) if save_u else None
    y_disp = _empty((R, D), BF16, dev)
    ws = _ws(L.moe_grouped_ffn_workspace_bytes(E, R, D, F), dev)
    L.moe_grouped_ffn(x_disp, offsets, E, R, D, F, W1, W2, h, u, y_disp, ws)
    return h, u, y_disp


def grouped_schedule(offsets: torch.Tensor, E: int, R: int) -> torch.Tensor:
    """Device tile schedule; its first E+1 int32 are the per-expert tile starts."""
    sched = _empty((L.moe_grouped_schedule_bytes(E, R) // 4,), I32, offsets.device)
    L.moe_grouped_schedule(offsets, E, R, sched)
    return sched


def grouped_gemm(A: torch.Tensor, sched: torch.Tensor, W: torch.Tensor, epilogue: int,
                 out: Optional[torch.Tensor] = None, u_save: Optional[torch.Tensor] = None):
    R, Kd = A.shape
    E, _, N = W.shape
    C = out if out is not None else _empty((R, N), BF16, A.device)
    L.moe_grouped_gemm(A, sched, E, R, Kd, N, W, epilogue, C, u_save)
    return C


def grouped_gemm_mxfp8(x_q: torch.Tensor, x_scale: torch.Tensor, sched: torch.Tensor, W: torch.Tensor,
                       epilogue: int, out: Optional[torch.Tensor] = None, u_save: Optional[torch.Tensor] = None):
    """grouped_gemm with the MX-FP8 payload (x_scale from mx_scales) as A."""
    R, Kd = x_q.shape
    E, _, N = W.shape
    C = out if out is not None else _empty((R, N), BF16, x_q.device)
    L.moe_grouped_gemm_mxfp8(x_q, x_scale, sched, E, R, Kd, N, W, epilogue, C, u_save)
    return C


def combine(y_disp: torch.Tensor, p_disp: Optional[torch.Tensor], inv_perm: torch.Tensor, S: int,
            K: int):
    D = y_disp.shape[1]
    y = _empty((S, D), BF16, y_disp.device)
    L.moe_combine(y_disp, p_disp, inv_perm, S, D, K, y)
    return y


def latent_proj(A: torch.Tensor, W: torch.Tensor):
    M, Kd = A.shape
    N = W.shape[1]
    C = _empty((M, N), BF16, A.device)
    L.moe_latent_proj(A, W, M, Kd, N, C)
    return C


def combine_bwd(dy, y_disp, p_disp, inv_perm, K: int, want_dp: bool = True):
    S, D = dy.shape
    dy_disp = _empty((S * K, D), BF16, dy.device)
    dp = _empty((S, K), F32, dy.device) if want_dp else None
    L.moe_combine_bwd(dy, y_disp, p_disp, inv_perm, S, D, K, dy_disp, dp)
    return dy_disp, dp


def grouped_ffn_bwd(x_disp, u_save, h, dy_disp, offsets, W1, W2):
    R, D = x_disp.shape
    E, _, F = W1.shape
    dev = x_disp.device
    dx_disp = _empty((R, D), BF16, dev)
    dW1 = _empty((E, D, F), F32, dev)
    dW2 = _empty((E, F, D), F32, dev)
    ws = _ws(L.moe_grouped_ffn_bwd_workspace_bytes(E, R, D, F), dev)
    L.moe_grouped_ffn_bwd(x_disp, u_save, h, dy_disp, offsets, E, R, D, F, W1, W2, dx_disp, dW1,
                          dW2, ws)
    return dx_disp, dW1, dW2


def dispatch_bwd(dx_disp, inv_perm, S: int, K: int, dx_add: Optional[torch.Tensor] = None):
    D = dx_disp.shape[1]
    dx = _empty((S, D), BF16, dx_disp.device)
    if dx_add is None:
        L.moe_dispatch_bwd(dx_disp, inv_perm, S, D, K, dx)
    else:
        L.moe_dispatch_bwd_add(dx_disp, inv_perm, dx_add, S, D, K, dx)
    return dx


def router_bwd(x_r, Wr, topk_idx, topk_prob, dp, want_dlogits: bool = True, want_dbias: bool = True,
               want_dx: bool = True) -> Dict[str, torch.Tensor]:
    """Router gradients with the selection held fixed: dlogits, dWr, dbias, dx_r (fp32)."""
    S, D = x_r.shape
    E = Wr.shape[1]
    K = topk_idx.shape[1]
    dev = x_r.device
    o = dict(dWr=_empty((D, E), F32, dev))
    o["dlogits"] = _empty((S, E), F32, dev) if want_dlogits else None
    o["dbias"] = _empty((E,), F32, dev) if want_dbias else None
    o["dx_r"] = _empty((S, D), F32, dev) if want_dx else None
    ws = _ws(L.moe_router_bwd_workspace_bytes(S, D, E), dev)
    L.moe_router_bwd(x_r, Wr, topk_idx, topk_prob, dp, S, D, E, K, o["dlogits"], o["dWr"], o["dbias"],
                     o["dx_r"], ws)
    return o


def latent_proj_bwd(x_in, W, dout, want_dx: bool = True, want_dW: bool = True):
    """Gradients of out = x_in @ W: (dx_in bf16 or None, dW fp32 or None)."""
    M, N = dout.shape
    Kd = W.shape[0]
    dev = dout.device
    dx = _empty((M, Kd), BF16, dev) if want_dx else None
    dW = _empty((Kd, N), F32, dev) if want_dW else None
    ws = _ws(L.moe_latent_proj_bwd_workspace_bytes(M, Kd, N), dev) if want_dW else None
    L.moe_latent_proj_bwd(x_in, W, dout, M, Kd, N, dx, dW, ws)
    return dx, dW


def route_sigmoid(logits: torch.Tensor, K: int, sel_bias: Optional[torch.Tensor] = None) -> Dict[str, torch.Tensor]:
    """Sigmoid routing with a selection-only bias; ``topk_prob`` holds the gates."""
    S, E = logits.shape
    dev = logits.device
    R = S * K
    o = dict(topk_idx=_empty((S, K), I32, dev), topk_prob=_empty((S, K), F32, dev),
             counts=_empty((E,), I32, dev), offsets=_empty((E + 1,), I32, dev),
             perm=_empty((R,), I32, dev), inv_perm=_empty((R,), I32, dev))
    ws = _ws(L.moe_route_workspace_bytes(S, E, K), dev)
    L.moe_route_sigmoid(logits, sel_bias, S, E, K, o["topk_idx"], o["topk_prob"], o["counts"], o["offsets"],
                        o["perm"], o["inv_perm"], ws)
    return o


def seq_aux_loss(logits: torch.Tensor, topk_idx: torch.Tensor, seq_len: int, coeff: float):
    """(loss [1] fp32, seq_counts [S/seq_len, E] int32)."""
    S, E = logits.shape
    K = topk_idx.shape[1]
    dev = logits.device
    loss = _empty((1,), F32, dev)
    counts = _empty((S // seq_len, E), I32, dev)
    ws = _ws(L.moe_seq_aux_loss_workspace_bytes(S, E, seq_len), dev)
    L.moe_seq_aux_loss(logits, topk_idx, S, E, K, seq_len, coeff, loss, counts, ws)
    return loss, counts


def router_bwd_sigmoid(x_r, Wr, logits, topk_idx, topk_gate, dg, seq_counts=None, seq_len: int = 0,
                       coeff: float = 0.0, want_dlogits: bool = True, want_dbias: bool = True,
                       want_dx: bool = True) -> Dict[str, torch.Tensor]:
    """Sigmoid-router gradients (selection fixed), plus the balance loss's when
    seq_counts is given: dlogits, dWr, dbias, dx_r (fp32)."""
    S, D = x_r.shape
    E = Wr.shape[1]
    K = topk_idx.shape[1]
    dev = x_r.device
    o = dict(dWr=_empty((D, E), F32, dev))
    o["dlogits"] = _empty((S, E), F32, dev) if want_dlogits else None
    o["dbias"] = _empty((E,), F32, dev) if want_dbias else None
    o["dx_r"] = _empty((S, D), F32, dev) if want_dx else None
    ws = _ws(L.moe_router_bwd_sigmoid_workspace_bytes(S, D, E), dev)
    L.moe_router_bwd_sigmoid(x_r, Wr, logits, topk_idx, topk_gate, dg, seq_counts, seq_len, coeff, S, D, E, K,
                             o["dlogits"], o["dWr"], o["dbias"], o["dx_r"], ws)
    return o


def expert_bias_update(counts: torch.Tensor, sel_bias: torch.Tensor, rate: float) -> torch.Tensor:
    """In place on sel_bias; returns it."""
    L.moe_expert_bias_update(counts, counts.shape[0], rate, sel_bias)
    return sel_bias


def combine_add(y_disp, p_disp, inv_perm, y_add, S: int, K: int):
    D = y_disp.shape[1]
    y = _empty((S, D), BF16, y_disp.device)
    L.moe_combine_add(y_disp, p_disp, inv_perm, y_add, S, D, K, y)
    return y


def shared_expert_fwd(x, Ws1, Ws2, save_u: bool = True):
    """(h_s bf16, u_s bf16 or None, y_s fp32)."""
    S, D = x.shape
    Fs = Ws1.shape[1]
    dev = x.device
    h = _empty((S, Fs), BF16, dev)
    u = _empty((S, Fs), BF16, dev) if save_u else None
    y = _empty((S, D), F32, dev)
    L.moe_shared_expert_fwd(x, Ws1, Ws2, S, D, Fs, h, u, y)
    return h, u, y


def shared_expert_bwd(x, u_s, h_s, dy, Ws1, Ws2, dx: Optional[torch.Tensor] = None, accumulate_dx: bool = False,
                      want_dx: bool = True):
    """(dx fp32 or None, dWs1, dWs2); with accumulate_dx the product is added to ``dx``."""
    S, D = x.shape
    Fs = Ws1.shape[1]
    dev = x.device
    if dx is None and want_dx:
        dx = _empty((S, D), F32, dev)
        accumulate_dx = False
    dW1 = _empty((D, Fs), F32, dev)
    dW2 = _empty((Fs, D), F32, dev)
    ws = _ws(L.moe_shared_expert_bwd_workspace_bytes(S, D, Fs), dev)
    L.moe_shared_expert_bwd(x, u_s, h_s, dy, Ws1, Ws2, S, D, Fs, dx, accumulate_dx, dW1, dW2, ws)
    return dx, dW1, dW2


class LayerFwd:
    """Preallocated buffers for repeated moe_layer_fwd calls on one shape.

    With export=True every intermediate is a torch tensor owned here (for
    parity checks); otherwise intermediates live in the workspace.

    With ``score="sigmoid"``, ``Fs`` and ``seq_len`` it runs the production
    variant (sigmoid routing with a selection-only bias, shared expert,
    sequence balance loss; exported as ``aux_loss``, ``seq_counts``, ``h_s``,
    ``u_s`` and ``y_s``).
    """

    def __init__(self, S, D, E, K, F, H=0, device="cuda", export=True, save_u=False, score="softmax",
                 Fs=0, seq_len=0, aux_coeff=0.0, payload="bf16"):
        self.S, self.D, self.E, self.K, self.F, self.H = S, D, E, K, F, H
        self.payload = {"bf16": L.PAYLOAD_BF16, "mxfp8": L.PAYLOAD_MXFP8}[payload]
        self.score_fn = {"softmax": L.SCORE_SOFTMAX, "sigmoid": L.SCORE_SIGMOID}[score]
        self.Fs, self.seq_len, self.aux_coeff = Fs, seq_len, aux_coeff
        dev = torch.device(device)
        R = S * K
        self.out: Dict[str, Optional[torch.Tensor]] = {}
        self.out["y"] = _empty((S, H if H else D), BF16, dev)
        if export:
            if H:
                self.out["x_lat"] = _empty((S, D), BF16, dev)
                self.out["y_lat"] = _empty((S, D), BF16, dev)
            self.out.update(
                logits=_empty((S, E), F32, dev), topk_idx=_empty((S, K), I32, dev),
                topk_prob=_empty((S, K), F32, dev), counts=_empty((E,), I32, dev),
                offsets=_empty((E + 1,), I32, dev), perm=_empty((R,), I32, dev),
                inv_perm=_empty((R,), I32, dev), x_disp=_empty((R, D), BF16, dev),
                p_disp=_empty((R,), F32, dev), h=_empty((R, F), BF16, dev),
                y_disp=_empty((R, D), BF16, dev))
        if save_u:
            self.out["u_save"] = _empty((R, F), BF16, dev)
        if seq_len:
            self.out["aux_loss"] = _empty((1,), F32, dev)
            if export:
                self.out["seq_counts"] = _empty((S // seq_len, E), I32, dev)
        if payload == "mxfp8" and export:
            self.out["x_q"] = _empty((R, D), torch.uint8, dev)
            self.out["x_scale"] = mx_scales(R, D, dev)
        if Fs:
            if export:
                self.out["h_s"] = _empty((S, Fs), BF16, dev)
                self.out["y_s"] = _empty((S, D), F32, dev)
            if save_u:
                self.out["u_s"] = _empty((S, Fs), BF16, dev)
        probe = L.layer_fwd_args(S, H, D, E, K, F, **self._modes(), **{k: v for k, v in self.out.items()})
        self.ws_bytes = L.moe_layer_fwd_workspace_bytes(probe)
        if self.ws_bytes == 0:
            raise ValueError("invalid layer shape")
        self.ws = _ws(self.ws_bytes, dev)

    def _modes(self):
        return dict(score_fn=self.score_fn, Fs=self.Fs, seq_len=self.seq_len, aux_coeff=self.aux_coeff,
                    payload=self.payload)

    def __call__(self, x, Wr, W1, W2, bias=None, Wdown=None, Wup=None, sel_bias=None, Ws1=None, Ws2=None):
        a = L.layer_fwd_args(self.S, self.H, self.D, self.E, self.K, self.F, ws=self.ws, x=x, Wr=Wr,
                             router_bias=bias, Wdown=Wdown, W1=W1, W2=W2, Wup=Wup, sel_bias=sel_bias,
                             Ws1=Ws1, Ws2=Ws2, **self._modes(), **self.out)
        L.moe_layer_fwd(a)
        return self.out
