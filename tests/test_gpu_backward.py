"""GPU parity of the backward pass through combine, experts and dispatch.

Routing comes from generated logits on both sides (bit-identical routes), the
GPU runs its own forward (dispatch, grouped FFN with u saved) and backward
(combine^T, grouped dgrad + wgrad, dispatch^T); the oracle runs the same
chain in float64.  dx and du-derived bf16 outputs are held to the bf16 bar;
the fp32 weight gradients to the same two metrics per tensor with the
mean-absolute term taken relative to the tensor's rms.
"""
import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from paper_2608_28511_amd import layer
from paper_2608_28511_amd.workloads import WORKLOADS, make_inputs

from gpu_helpers import LazyExperts, assert_bf16_close, np64, npi

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def gpu_chain(x, logits, W1, W2, dy, K):
    S = x.shape[0]
    r = layer.route(logits, K)
    x_disp, p_disp = layer.dispatch(x, r["topk_prob"], r["inv_perm"], K)
    h, u, yd = layer.grouped_ffn(x_disp, r["offsets"], W1, W2, save_u=True)
    y = layer.combine(yd, p_disp, r["inv_perm"], S, K)
    dyd, dp = layer.combine_bwd(dy, yd, p_disp, r["inv_perm"], K)
    dxd, dW1, dW2 = layer.grouped_ffn_bwd(x_disp, u, h, dyd, r["offsets"], W1, W2)
    dx = layer.dispatch_bwd(dxd, r["inv_perm"], S, K)
    torch.cuda.synchronize()
    return dict(r=r, y=y, dp=dp, dx=dx, dW1=dW1, dW2=dW2, dxd=dxd)


def oracle_chain(x, logits, W1, W2, dy, K, E):
    S = x.shape[0]
    idx, p = O.route(logits, K)
    counts, off, perm, inv = O.expert_permutation(idx, E)
    xd, pd = O.dispatch(x, p, inv, K)
    u, h, yd = O.expert_ffn(xd, off, W1, W2, round_payload=False)
    y = O.combine(yd, pd, inv, S, K)
    dyd, dp = O.combine_bwd(dy, yd, pd, inv, K, round_payload=False)
    dxd, dW1, dW2, du = O.expert_ffn_bwd(xd, u, h, dyd, off, W1, W2, round_payload=False)
    dx = O.dispatch_bwd(dxd, inv, S, K)
    return dict(counts=counts, y=y, dp=dp, dx=dx, dW1=dW1, dW2=dW2, off=off, xd=xd, u=u, h=h,
                dyd=dyd, dxd=dxd, inv=inv, yd=yd, pd=pd)


def assert_grad_close(got, ref, what):
    assert_bf16_close(got, ref, what, mean_abs=1e-2, mean_rel_to_rms=True)


EPS_BF16 = 2.0 ** -8   # relative error of one round-to-nearest to bf16 (8 significant bits)
U32 = 2.0 ** -24       # unit roundoff of fp32


def u_bound(xd, W1e):
    """|u_gpu - u| of the up projection's fp32 accumulation over D products
    (before any bf16 rounding): (D + 8) U |x_disp| @ |W1_e|.  Where u cancels
    (|u| much smaller than its terms) this dominates the relative error of u
    and of h = max(u, 0)^2."""
    return (xd.shape[1] + 8) * U32 * (np.abs(xd) @ np.abs(W1e))


def h_u_bound(u, b_u):
    """|max(u_gpu, 0)^2 - max(u, 0)^2| from |u_gpu - u| <= b_u (a sign flip
    near zero included): 2 max(u, 0) b_u + b_u^2."""
    return 2 * np.maximum(u, 0) * b_u + b_u ** 2


def bwd_bounds(xd, u, h, dyd, dxd, W1e, W2e):
    """Elementwise error bounds for one expert segment of the backward.

    The GPU's forward carries u's fp32 accumulation error b_u (u_bound) into
    u_save and h; then it rounds dy_disp, u_save and du to bf16 (each <=
    EPS_BF16 relative) before they enter fp32-accumulated products.  With
    mag_dh = |dy_disp| @ |W2^T| bounding |dh| and its error,
        |du_gpu - du|       <= (4 EPS_BF16 2 max(u,0) + 2 (1 + EPS_BF16) b_u) mag_dh
                               (one rounding each in dy_disp, u, du, room for
                               fp32 accumulation; u_save off by b_u as well)
        |dW1_gpu - dW1|     <= |x_disp|^T @ b_du
        |dW2_gpu - dW2|     <= 4 EPS_BF16 |h|^T @ |dy_disp| + (1 + 4 EPS_BF16) h_u^T @ |dy_disp|
                               (h and dy_disp rounded; h_u = h_u_bound, h's
                               error from u's)
        |dx_disp_gpu - ref| <= b_du @ |W1^T| + EPS_BF16 * |dx_disp|  (final rounding)"""
    b_u = u_bound(xd, W1e)
    mag_dh = np.abs(dyd) @ np.abs(W2e).T
    b_du = (4 * EPS_BF16 * 2 * np.maximum(u, 0) + 2 * (1 + EPS_BF16) * b_u) * mag_dh
    b_dxd = b_du @ np.abs(W1e).T + EPS_BF16 * np.abs(dxd)
    b_dw2 = 4 * EPS_BF16 * (np.abs(h).T @ np.abs(dyd)) + (1 + 4 * EPS_BF16) * (h_u_bound(u, b_u).T @ np.abs(dyd))
    return np.abs(xd).T @ b_du, b_dw2, b_dxd


def y_bound(R, W1, W2, S, K, E):
    """Elementwise bound on |y_gpu - y| from the forward's fp32 accumulation
    of u (carried into h, h_u_bound) and its three bf16 roundings (h, the
    down projection's input; y_disp; y):
        |dy_disp| <= (EPS_BF16 |h| + h_u) @ |W2_e| + EPS_BF16 * |y_disp|
        |dy|      <= sum_k p_k |dy_disp| + EPS_BF16 * |y|
    with a factor 1.25 of room for fp32 accumulation.  A max-relative bar
    cannot stand in for it when the down projection sums few large terms
    that cancel."""
    b_yd = np.zeros_like(R["yd"])
    off = R["off"]
    for e in range(E):
        a, b = int(off[e]), int(off[e + 1])
        if a < b:
            h_u = h_u_bound(R["u"][a:b], u_bound(R["xd"][a:b], W1[e]))
            b_yd[a:b] = ((EPS_BF16 * np.abs(R["h"][a:b]) + h_u) @ np.abs(W2[e])
                         + EPS_BF16 * np.abs(R["yd"][a:b]))
    return 1.25 * (O.combine(b_yd, np.abs(R["pd"]), R["inv"], S, K) + EPS_BF16 * np.abs(R["y"]))


def assert_within(got, ref, bound, what):
    d = np.abs(got - ref)
    bad = d > bound
    worst = float(np.max(d / np.maximum(bound, 1e-300))) if d.size else 0.0
    assert not bad.any(), f"{what}: {int(bad.sum())} of {d.size} beyond the bound (worst {worst:.2f}x)"
    rms = float(np.sqrt(np.mean(ref ** 2))) if ref.size else 0.0
    assert float(np.mean(d)) <= 1e-2 * rms, f"{what}: mean error {np.mean(d):.3e} vs rms {rms:.3e}"


# the last expert is dead (-inf logits) in every case: (1, 8, 2, 1, 8) is one
# token on one live expert; (7, 72, 3, 2, 24) sends every token to every live
# expert; (64, 136, 1024, 32, 40) is the largest E and K the ABI takes
@pytest.mark.parametrize("S,D,E,K,F", [(64, 64, 4, 2, 64), (300, 136, 9, 3, 200), (512, 256, 8, 2, 512),
                                       (1024, 512, 32, 8, 256), (1, 8, 2, 1, 8), (7, 72, 3, 2, 24),
                                       (64, 136, 1024, 32, 40)])
def test_backward_small(S, D, E, K, F):
    check_backward_case(S, D, E, K, F, seed=S + D + E)


def test_backward_cancelling_u():
    """A seeded random case (two rows on expert 43) where one pre-activation
    nearly cancels (u = 4.8e-6 against sum |x||W1| = 7.4): u's fp32
    accumulation error is then over 1% of u, so h = max(u, 0)^2 and that
    row of dW2 miss a bound that budgets only the bf16 roundings; the
    bounds carry the forward accumulation term (u_bound)."""
    check_backward_case(91, 120, 53, 2, 336, seed=343)


def check_backward_case(S, D, E, K, F, seed):
    """Forward and backward chain of one seeded case (the last expert dead)
    against the oracle, with elementwise bounds on every gradient."""
    g = torch.Generator().manual_seed(seed)
    x = torch.randn((S, D), generator=g).to(torch.bfloat16)
    logits = torch.randn((S, E), generator=g)
    logits[:, E - 1] = float("-inf")          # one dead expert
    W1 = (torch.randn((E, D, F), generator=g) / np.sqrt(D)).to(torch.bfloat16)
    W2 = (torch.randn((E, F, D), generator=g) / np.sqrt(F)).to(torch.bfloat16)
    dy = torch.randn((S, D), generator=g).to(torch.bfloat16)
    G = gpu_chain(x.to(DEV), logits.to(DEV), W1.to(DEV), W2.to(DEV), dy.to(DEV), K)
    R = oracle_chain(np64(x), logits.numpy(), np64(W1), np64(W2), np64(dy), K, E)
    assert np.array_equal(npi(G["r"]["counts"]), R["counts"])
    assert_within(np64(G["y"]), R["y"], y_bound(R, np64(W1), np64(W2), S, K, E), "y")
    assert_grad_close(np64(G["dp"]), R["dp"], "dp")
    gW1, gW2 = np64(G["dW1"]), np64(G["dW2"])
    off = R["off"]
    b_dxd = np.zeros_like(R["dxd"])
    for e in range(E):
        a, b = int(off[e]), int(off[e + 1])
        if a == b:
            continue
        b1, b2, b_dxd[a:b] = bwd_bounds(R["xd"][a:b], R["u"][a:b], R["h"][a:b], R["dyd"][a:b],
                                        R["dxd"][a:b], np64(W1[e]), np64(W2[e]))
        assert_within(gW1[e], R["dW1"][e], b1, f"dW1[{e}]")
        assert_within(gW2[e], R["dW2"][e], b2, f"dW2[{e}]")
    # dx sums the K dx_disp rows of a token, then rounds once more
    b_dx = O.dispatch_bwd(b_dxd, R["inv"], S, K) + EPS_BF16 * np.abs(R["dx"])
    assert_within(np64(G["dx"]), R["dx"], b_dx, "dx")
    assert torch.all(G["dW1"][E - 1] == 0) and torch.all(G["dW2"][E - 1] == 0)


def test_backward_full_size():
    """Zipf-skewed 16384-token workload, every output against the oracle: dx
    and dp of every token, dW1 and dW2 of every live expert within their
    elementwise bounds, exactly zero dW for the dead experts.  The gradients
    are written into NaN-filled buffers with guard rows (guard experts for
    dW), so an unwritten element or a stray write shows, and the whole
    backward runs twice and must reproduce itself bit for bit."""
    from paper_2608_28511_amd import _lib as L
    from gpu_helpers import check_guarded, guarded

    s = WORKLOADS["skew_s16384_d2048_e128_k8_bwd"]
    S, D, E, K, F, R = s.S, s.D, s.E, s.K, s.F, s.R
    inp = make_inputs(s, device=DEV)
    logits = torch.randn((S, E), device=DEV,
                         generator=torch.Generator(device=DEV).manual_seed(2)) + inp["bias"][None, :]
    r = layer.route(logits, K)
    x_disp, p_disp = layer.dispatch(inp["x"], r["topk_prob"], r["inv_perm"], K)
    h, u, yd = layer.grouped_ffn(x_disp, r["offsets"], inp["W1"], inp["W2"], save_u=True)
    ws = torch.empty(L.moe_grouped_ffn_bwd_workspace_bytes(E, R, D, F), dtype=torch.uint8, device=DEV)
    G = 2

    def backward():
        b = {}
        b["dyd"], dyd = guarded((R, D), torch.bfloat16, DEV, G)
        b["dp"], dp = guarded((S, K), torch.float32, DEV, G)
        b["dxd"], dxd = guarded((R, D), torch.bfloat16, DEV, G)
        b["dW1"], dW1 = guarded((E, D, F), torch.float32, DEV, G)
        b["dW2"], dW2 = guarded((E, F, D), torch.float32, DEV, G)
        b["dx"], dx = guarded((S, D), torch.bfloat16, DEV, G)
        L.moe_combine_bwd(inp["dy"], yd, p_disp, r["inv_perm"], S, D, K, dyd, dp)
        L.moe_grouped_ffn_bwd(x_disp, u, h, dyd, r["offsets"], E, R, D, F, inp["W1"], inp["W2"], dxd, dW1, dW2, ws)
        L.moe_dispatch_bwd(dxd, r["inv_perm"], S, D, K, dx)
        torch.cuda.synchronize()
        for k, buf in b.items():
            check_guarded(buf, G, f"backward {k}")
        return {k: v[G:-G] for k, v in b.items()}

    got = backward()
    again = backward()
    for k in got:
        assert torch.equal(got[k], again[k]), f"{k} differs between two identical calls"
    del again

    lg = logits.cpu().numpy()
    W1, W2 = LazyExperts(inp["W1"], cache=True), LazyExperts(inp["W2"], cache=True)
    R_ = oracle_chain(np64(inp["x"]), lg, W1, W2, np64(inp["dy"]), K, E)
    counts = R_["counts"]
    assert np.array_equal(npi(r["counts"]), counts)
    assert np.array_equal(npi(r["inv_perm"]), R_["inv"])
    assert_grad_close(np64(got["dp"]), R_["dp"], "dp")
    off = R_["off"]
    b_dxd = np.zeros_like(R_["dxd"])
    live = 0
    for e in range(E):
        a, b = int(off[e]), int(off[e + 1])
        if a == b:
            assert torch.all(got["dW1"][e] == 0) and torch.all(got["dW2"][e] == 0), f"dead expert {e}"
            continue
        live += 1
        b1, b2, b_dxd[a:b] = bwd_bounds(R_["xd"][a:b], R_["u"][a:b], R_["h"][a:b], R_["dyd"][a:b],
                                        R_["dxd"][a:b], W1[e], W2[e])
        assert_within(np64(got["dW1"][e]), R_["dW1"][e], b1, f"dW1[{e}] ({b - a} rows)")
        assert_within(np64(got["dW2"][e]), R_["dW2"][e], b2, f"dW2[{e}] ({b - a} rows)")
    assert live == E - int((counts == 0).sum()) and (counts == 0).sum() >= 4
    b_dx = O.dispatch_bwd(b_dxd, R_["inv"], S, K) + EPS_BF16 * np.abs(R_["dx"])
    assert_within(np64(got["dx"]), R_["dx"], b_dx, "dx")
