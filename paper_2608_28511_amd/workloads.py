"""Seeded synthetic inputs for one routed MoE layer.

This module only draws random numbers and lays them out; it computes no step
of the layer.  Both the HIP path and the CPU oracle consume what it returns,
so it must stay free of routing, GEMM or combine arithmetic.

Notation follows the paper: S tokens per micro-batch, D dispatch (hidden)
dimension, E experts, top-K routing, F per-expert FFN width (f_expert in
Table 2), H model hidden when a LatentMoE-style projection precedes dispatch
(Section 1 "dispatch dimension" lever; Table 2 d_latent).

Draw order per workload is fixed (x, Wr, bias, Wdown, W1, W2, Wup, dy, then
for the production variant sel_bias, Ws1, Ws2) from
one ``torch.Generator`` seeded with the workload's seed, on the requested
device.  CPU and GPU generators produce different streams; a test always
feeds the same bytes to both sides, so cross-device stream parity is never
needed.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, replace
from typing import Dict, Optional

import torch


@dataclass(frozen=True)
class MoEShape:
    """One routed-MoE-layer workload.

    bias: how router logits are offset per expert before softmax.
      "none"      no bias
      "normal"    b_e ~ N(0, 0.5)  (variance 0.5: moderate load imbalance)
      "zipf"      b_e = -1.1 * ln(r_e), r a seeded rank permutation of 1..E,
                  and the 4 lowest-ranked experts masked to -inf so that some
                  experts receive no rows at all

    The production variant of Section 5.2 (score "sigmoid"): a selection-only
    expert bias ~ N(0, sel_bias_std^2) (the state a load-driven update leaves
    it in: small, of either sign), a shared expert of width Fs, and the
    sequence balance loss over sequences of seq_len tokens.
    """

    name: str
    S: int
    D: int
    E: int
    K: int
    F: int
    H: int = 0
    bias: str = "none"
    backward: bool = False
    seed: int = 0
    score: str = "softmax"
    sel_bias_std: float = 0.0
    Fs: int = 0
    seq_len: int = 0
    aux_coeff: float = 0.0

    @property
    def R(self) -> int:
        """Routed rows (token, slot) pairs: S*K."""
        return self.S * self.K

    @property
    def D_in(self) -> int:
        """Width of the layer input x: H when a latent projection is used."""
        return self.H if self.H else self.D

    def scaled(self, **kw) -> "MoEShape":
        return replace(self, **kw)


# The five workloads, named by what they are.
WORKLOADS: Dict[str, MoEShape] = {
    # tiny layer: small enough for the oracle to run in full in seconds
    "tiny_s512_d256_e8_k2": MoEShape("tiny_s512_d256_e8_k2", S=512, D=256, E=8, K=2, F=512, seed=1),
    # full-MoE-baseline-style layer: seq 4096 x micro-batch 2, 64 experts top-6
    "base_s8192_d2048_e64_k6": MoEShape("base_s8192_d2048_e64_k6", S=8192, D=2048, E=64, K=6,
                                        F=1024, seed=2),
    # CE-MoE-style fewer-but-wider layer with biased (imbalanced) routing
    "ce_s8192_d2048_e256_k8": MoEShape("ce_s8192_d2048_e256_k8", S=8192, D=2048, E=256, K=8,
                                       F=2688, bias="normal", seed=3),
    # LatentMoE-style: hidden 4096 projected to a 1024-wide dispatch dimension
    "latent_s16384_h4096_d1024_e128_k6": MoEShape("latent_s16384_h4096_d1024_e128_k6", S=16384,
                                                  D=1024, E=128, K=6, F=1536, H=4096, seed=4),
    # Zipf-skewed routing with the backward pass
    "skew_s16384_d2048_e128_k8_bwd": MoEShape("skew_s16384_d2048_e128_k8_bwd", S=16384, D=2048,
                                              E=128, K=8, F=1024, bias="zipf", backward=True,
                                              seed=5),
}

# The production layer of Section 5.2 (sigmoid scores with a selection-only
# bias, shared expert, sequence balance loss with coefficient 1e-4): a tiny
# one for full oracle parity, and the 31.5B CE-MoE layer shape of Table 2 and
# Section 4.3 (hidden 2688, 192 experts top-7, expert and shared width 3520)
# over two sequences of 8192 tokens, with the backward pass.
PRODUCTION: Dict[str, MoEShape] = {
    "prod_tiny_s512_d256_e8_k2": MoEShape("prod_tiny_s512_d256_e8_k2", S=512, D=256, E=8, K=2, F=512,
                                          backward=True, seed=6, score="sigmoid", sel_bias_std=0.05,
                                          Fs=256, seq_len=128, aux_coeff=1e-4),
    "prod_s16384_d2688_e192_k7": MoEShape("prod_s16384_d2688_e192_k7", S=16384, D=2688, E=192, K=7,
                                          F=3520, backward=True, seed=7, score="sigmoid",
                                          sel_bias_std=0.05, Fs=3520, seq_len=8192, aux_coeff=1e-4),
}
# The paper's own latent layers at the 31.5B scale (Table 2): hidden 2688
# projected to the dispatch width d_latent, with LatentMoE's 512 experts
# top-22 (expert width 1856) and CE-LatentMoE's 640 experts top-24 (expert
# width 3712), over two sequences of 8192 tokens; softmax routing as in the
# latent workload above.
PAPER_SHAPES: Dict[str, MoEShape] = {
    "latentmoe_s16384_h2688_d672_e512_k22": MoEShape("latentmoe_s16384_h2688_d672_e512_k22", S=16384, D=672,
                                                     E=512, K=22, F=1856, H=2688, seed=8),
    "celatent_s16384_h2688_d768_e640_k24": MoEShape("celatent_s16384_h2688_d768_e640_k24", S=16384, D=768,
                                                    E=640, K=24, F=3712, H=2688, seed=9),
}

PROD_TINY = PRODUCTION["prod_tiny_s512_d256_e8_k2"]
PROD = PRODUCTION["prod_s16384_d2688_e192_k7"]

TINY = WORKLOADS["tiny_s512_d256_e8_k2"]
BASE = WORKLOADS["base_s8192_d2048_e64_k6"]
CE = WORKLOADS["ce_s8192_d2048_e256_k8"]
LATENT = WORKLOADS["latent_s16384_h4096_d1024_e128_k6"]
SKEW = WORKLOADS["skew_s16384_d2048_e128_k8_bwd"]

ZIPF_S = 1.1
ZIPF_MASKED = 4


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def _normal(shape, std: float, g: torch.Generator, device, out_dtype, chunk_dim0: int = 0):
    """N(0, std^2) draws, rounded (RNE) to out_dtype.  Large tensors are
    drawn in chunks along dim 0 so the fp32 temporary stays small."""
    shape = tuple(shape)
    if chunk_dim0 <= 0 or shape[0] <= chunk_dim0:
        return (torch.randn(shape, generator=g, device=device, dtype=torch.float32) * std).to(out_dtype)
    out = torch.empty(shape, device=device, dtype=out_dtype)
    for i in range(0, shape[0], chunk_dim0):
        j = min(shape[0], i + chunk_dim0)
        out[i:j] = (torch.randn((j - i,) + shape[1:], generator=g, device=device,
                                dtype=torch.float32) * std).to(out_dtype)
    return out


def router_bias(shape: MoEShape, g: torch.Generator, device) -> Optional[torch.Tensor]:
    if shape.bias == "none":
        return None
    if shape.bias == "normal":
        return torch.randn((shape.E,), generator=g, device=device, dtype=torch.float32) * math.sqrt(0.5)
    if shape.bias == "zipf":
        rank = torch.randperm(shape.E, generator=g, device=device).to(torch.float64) + 1.0
        b = (-ZIPF_S * torch.log(rank)).to(torch.float32)
        b[rank > shape.E - ZIPF_MASKED] = float("-inf")
        return b
    raise ValueError(f"unknown bias kind {shape.bias!r}")


def make_inputs(shape: MoEShape, device="cpu", seed: Optional[int] = None,
                with_experts: bool = True) -> Dict[str, torch.Tensor]:
    """All inputs of one layer call, as torch tensors on ``device``.

    x      [S, D_in] bf16 ~ N(0,1)
    Wr     [D, E]    fp32 ~ N(0, 1/D)     (router reads the dispatch-width input)
    bias   [E]       fp32 or None
    Wdown  [H, D]    bf16 ~ N(0, 1/H)     (latent workloads only)
    W1     [E, D, F] bf16 ~ N(0, 1/D)
    W2     [E, F, D] bf16 ~ N(0, 1/F)
    Wup    [D, H]    bf16 ~ N(0, 1/D)     (latent workloads only)
    dy     [S, D_in] bf16 ~ N(0,1)        (backward workloads only)
    sel_bias [E]     fp32 ~ N(0, sel_bias_std^2)   (sigmoid-score workloads)
    Ws1    [D, Fs]   bf16 ~ N(0, 1/D)     (shared expert)
    Ws2    [Fs, D]   bf16 ~ N(0, 1/Fs)
    """
    s = shape
    g = _gen(device, s.seed if seed is None else seed)
    out: Dict[str, Optional[torch.Tensor]] = {}
    out["x"] = _normal((s.S, s.D_in), 1.0, g, device, torch.bfloat16, chunk_dim0=4096)
    out["Wr"] = _normal((s.D, s.E), 1.0 / math.sqrt(s.D), g, device, torch.float32)
    out["bias"] = router_bias(s, g, device)
    if s.H:
        out["Wdown"] = _normal((s.H, s.D), 1.0 / math.sqrt(s.H), g, device, torch.bfloat16)
    if with_experts:
        out["W1"] = _normal((s.E, s.D, s.F), 1.0 / math.sqrt(s.D), g, device, torch.bfloat16,
                            chunk_dim0=8)
        out["W2"] = _normal((s.E, s.F, s.D), 1.0 / math.sqrt(s.F), g, device, torch.bfloat16,
                            chunk_dim0=8)
    if s.H:
        out["Wup"] = _normal((s.D, s.H), 1.0 / math.sqrt(s.D), g, device, torch.bfloat16)
    if s.backward:
        out["dy"] = _normal((s.S, s.D_in), 1.0, g, device, torch.bfloat16, chunk_dim0=4096)
    if s.score == "sigmoid":
        out["sel_bias"] = _normal((s.E,), s.sel_bias_std, g, device, torch.float32)
    if s.Fs:
        out["Ws1"] = _normal((s.D_in, s.Fs), 1.0 / math.sqrt(s.D_in), g, device, torch.bfloat16)
        out["Ws2"] = _normal((s.Fs, s.D_in), 1.0 / math.sqrt(s.Fs), g, device, torch.bfloat16)
    return out


# ---------------------------------------------------------------------------
# Router-logit suites for exercising top-K selection corner cases directly.
# ---------------------------------------------------------------------------

def make_logits(kind: str, S: int, E: int, seed: int, device="cpu") -> torch.Tensor:
    """fp32 router logits [S, E] with a chosen structure.

    normal     N(0,1)
    quantised  integers in {-2..2}: many exact ties
    equal      every row constant: selection must be experts 0..K-1
    signed0    entries drawn from {-0.0, +0.0, -1, 1}
    masked     N(0,1) with ~half the entries set to -inf (entry t % E of row t
               always finite, so every row has a finite best score)
    nan        N(0,1) with a few NaN entries per row
    """
    g = _gen(device, seed)
    if kind == "normal":
        return torch.randn((S, E), generator=g, device=device)
    if kind == "quantised":
        return torch.randint(-2, 3, (S, E), generator=g, device=device).to(torch.float32)
    if kind == "equal":
        v = torch.randn((S, 1), generator=g, device=device)
        return v.expand(S, E).contiguous()
    if kind == "signed0":
        choice = torch.randint(0, 4, (S, E), generator=g, device=device)
        table = torch.tensor([-0.0, 0.0, -1.0, 1.0], device=device)
        return table[choice]
    if kind == "masked":
        v = torch.randn((S, E), generator=g, device=device)
        drop = torch.rand((S, E), generator=g, device=device) < 0.5
        rows = torch.arange(S, device=device)
        drop[rows, rows % E] = False
        v[drop] = float("-inf")
        return v
    if kind == "nan":
        v = torch.randn((S, E), generator=g, device=device)
        bad = torch.rand((S, E), generator=g, device=device) < (2.0 / max(E, 2))
        v[bad] = float("nan")
        return v
    raise ValueError(kind)


def make_topk_indices(S: int, E: int, K: int, seed: int, device="cpu",
                      weights: Optional[torch.Tensor] = None) -> torch.Tensor:
    """K distinct expert ids per token, drawn without replacement ([S,K] int32)."""
    g = _gen(device, seed)
    w = torch.ones((E,), device=device) if weights is None else weights.to(device)
    idx = torch.multinomial(w.expand(S, E), K, replacement=False, generator=g)
    return idx.to(torch.int32)


def make_segments(R: int, E: int, seed: int, empty: int = 0, skew: float = 0.0) -> torch.Tensor:
    """Random expert segment boundaries: int32 [E+1] with offsets[0] = 0,
    offsets[E] = R, non-decreasing.  ``empty`` experts (chosen at random)
    get no rows; ``skew`` > 0 makes segment lengths Zipf-like."""
    g = _gen("cpu", seed)
    w = torch.rand((E,), generator=g, dtype=torch.float64) + 0.05
    if skew > 0:
        order = torch.randperm(E, generator=g).to(torch.float64) + 1.0
        w = order ** (-skew)
    if empty:
        dead = torch.randperm(E, generator=g)[:empty]
        w[dead] = 0.0
    cut = torch.floor(torch.cumsum(w, 0) / w.sum() * R).to(torch.int64)
    cut[-1] = R
    off = torch.zeros((E + 1,), dtype=torch.int64)
    off[1:] = cut
    return off.to(torch.int32)


def make_sparse_sign_rows(R: int, D: int, nnz: int, seed: int) -> torch.Tensor:
    """[R, D] float32 rows holding exactly min(nnz, D) entries of +-1 at random
    columns and zeros elsewhere (exact-arithmetic GEMM inputs)."""
    g = _gen("cpu", seed)
    out = torch.zeros((R, D), dtype=torch.float32)
    n = min(nnz, D)
    cols = torch.argsort(torch.rand((R, D), generator=g), dim=1)[:, :n]
    signs = torch.randint(0, 2, (R, n), generator=g).to(torch.float32) * 2 - 1
    out.scatter_(1, cols, signs)
    return out
