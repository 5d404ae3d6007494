"""GPU parity: dispatch, combine and their transposes.

Dispatch is a bit-exact copy (the Eq. 1 payload); combine with identity
experts must return x bit-exactly; everything else within the bf16 bar.
Routing for these tests comes from generated logits on both sides (the GPU
route and the oracle route agree bit-exactly, checked in test_gpu_route).
"""
import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from paper_2608_28511_amd import _lib as L
from paper_2608_28511_amd import layer
from paper_2608_28511_amd.workloads import WORKLOADS, make_logits

from gpu_helpers import assert_bf16_close, np64, npi

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _setup(S, D, E, K, seed):
    g = torch.Generator().manual_seed(seed)
    x = torch.randn((S, D), generator=g).to(torch.bfloat16)
    logits = make_logits("normal", S, E, seed=seed)
    r = layer.route(logits.to(DEV), K)
    idx, prob = O.route(logits.numpy(), K)
    counts, offsets, perm, inv = O.expert_permutation(idx, E)
    return g, x, r, prob, inv


SHAPES = [(1, 8, 1, 1), (33, 264, 8, 2), (512, 256, 8, 2), (1000, 2048, 64, 6), (301, 1032, 37, 5),
          (130, 4096, 256, 8)]


@pytest.mark.parametrize("S,D,E,K", SHAPES)
def test_dispatch_bit_exact_and_eq1_bytes(S, D, E, K):
    g, x, r, prob, inv = _setup(S, D, E, K, seed=S + D)
    x_disp, p_disp = layer.dispatch(x.to(DEV), r["topk_prob"], r["inv_perm"], K)
    torch.cuda.synchronize()
    xd_ref, pd_ref = O.dispatch(np64(x), prob, inv, K)
    assert np.array_equal(np64(x_disp), xd_ref)
    # p_disp is a copy of the GPU's routed probabilities (checked against the
    # oracle within 1e-5 in the route tests); compare it to them exactly
    assert np.array_equal(np64(p_disp), np64(r["topk_prob"]).reshape(-1)[npi(r["perm"])])
    nbytes = x_disp.numel() * x_disp.element_size() + p_disp.numel() * p_disp.element_size()
    assert nbytes == L.moe_payload_bytes(S, K, D) == O.dispatch_payload_bytes(S, K, D)


@pytest.mark.parametrize("S,D,E,K", SHAPES)
def test_combine_identity_experts_bit_exact(S, D, E, K):
    g, x, r, prob, inv = _setup(S, D, E, K, seed=3 * S + D)
    xg = x.to(DEV)
    x_disp, p_disp = layer.dispatch(xg, r["topk_prob"], r["inv_perm"], K)
    y = layer.combine(x_disp, p_disp, r["inv_perm"], S, K)
    torch.cuda.synchronize()
    assert torch.equal(y, xg)


@pytest.mark.parametrize("S,D,E,K", SHAPES)
def test_combine_matches_oracle(S, D, E, K):
    g, x, r, prob, inv = _setup(S, D, E, K, seed=5 * S + D)
    yd = torch.randn((S * K, D), generator=g).to(torch.bfloat16)
    _, p_disp = layer.dispatch(x.to(DEV), r["topk_prob"], r["inv_perm"], K)
    y = layer.combine(yd.to(DEV), p_disp, r["inv_perm"], S, K)
    _, pd_ref = O.dispatch(np64(x), prob, inv, K)
    ref = O.combine(np64(yd), pd_ref, inv, S, K)
    assert_bf16_close(np64(y), ref, "combine")
    # unit weights: the dispatch transpose
    dx = layer.dispatch_bwd(yd.to(DEV), r["inv_perm"], S, K)
    assert_bf16_close(np64(dx), O.dispatch_bwd(np64(yd), inv, S, K), "dispatch_bwd")


@pytest.mark.parametrize("S,D,E,K", SHAPES)
def test_combine_bwd_matches_oracle(S, D, E, K):
    g, x, r, prob, inv = _setup(S, D, E, K, seed=7 * S + D)
    yd = torch.randn((S * K, D), generator=g).to(torch.bfloat16)
    dy = torch.randn((S, D), generator=g).to(torch.bfloat16)
    _, p_disp = layer.dispatch(x.to(DEV), r["topk_prob"], r["inv_perm"], K)
    dyd, dp = layer.combine_bwd(dy.to(DEV), yd.to(DEV), p_disp, r["inv_perm"], K)
    _, pd_ref = O.dispatch(np64(x), prob, inv, K)
    dyd_ref, dp_ref = O.combine_bwd(np64(dy), np64(yd), pd_ref, inv, K, round_payload=False)
    assert_bf16_close(np64(dyd), dyd_ref, "dy_disp")
    # dp is an fp32 dot product of length D: bound its error by the dot of magnitudes
    mag = O.combine_bwd(np.abs(np64(dy)), np.abs(np64(yd)), None, inv, K, round_payload=False)[1]
    assert np.all(np.abs(np64(dp) - dp_ref) <= 1e-5 * mag + 1e-6), "dp"


def test_full_size_dispatch_combine():
    """Largest dispatch in the workloads (16384 tokens, D = 2048, top-8)."""
    s = WORKLOADS["skew_s16384_d2048_e128_k8_bwd"]
    g = torch.Generator(device=DEV).manual_seed(9)
    x = torch.randn((s.S, s.D), generator=g, device=DEV).to(torch.bfloat16)
    logits = torch.randn((s.S, s.E), generator=g, device=DEV)
    r = layer.route(logits, s.K)
    x_disp, p_disp = layer.dispatch(x, r["topk_prob"], r["inv_perm"], s.K)
    y = layer.combine(x_disp, p_disp, r["inv_perm"], s.S, s.K)
    torch.cuda.synchronize()
    assert torch.equal(y, x)
    # spot rows of the dispatched buffer against the oracle's own route
    idx, prob = O.route(logits.cpu().numpy(), s.K)
    _, _, perm, inv = O.expert_permutation(idx, s.E)
    rows = np.random.default_rng(0).choice(s.R, 256, replace=False)
    xd = np64(x_disp[torch.as_tensor(rows, device=DEV)])
    xs = np64(x)
    assert np.array_equal(xd, xs[perm[rows] // s.K])


def test_out_of_range_inv_perm_is_ignored():
    """Malformed positions are skipped, never written or read out of bounds."""
    S, D, K = 16, 64, 2
    x = torch.randn((S, D), device=DEV).to(torch.bfloat16)
    inv = torch.arange(S * K, dtype=torch.int32, device=DEV)
    inv[3] = S * K + 5
    inv[4] = -2
    guard = torch.full((S * K + 64, D), 7.0, device=DEV).to(torch.bfloat16)
    x_disp = guard[: S * K]
    L.moe_dispatch(x, None, inv, S, D, K, x_disp, None)
    torch.cuda.synchronize()
    assert torch.all(guard[S * K:] == 7.0)
    y = layer.combine(x_disp, None, inv, S, K)
    torch.cuda.synchronize()
    assert torch.isfinite(y.float()).all()
