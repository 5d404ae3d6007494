"""The paper's own latent layers at the 31.5B scale (Table 2) through
moe_layer_fwd: LatentMoE (hidden 2688 projected to d_latent 672, 512
experts top-22, expert width 1856) and CE-LatentMoE (d_latent 768, 640
experts top-24, expert width 3712), 16384 tokens each.

Checked as the full-size layers are, except that the expert outputs are
compared on sampled tokens: x_lat of every token within its fp32/bf16
bound, the logits of every token, the routing of every token (bit-exact
away from near ties, a valid selection within them), the permutation
properties, every dispatched row and probability bit for bit; then h and
y_disp of every routed row of 16 sampled unambiguous tokens and their y,
against the oracle's chain on that sub-batch in the paper's training
precision (valid because a token's output depends only on its own row and
routing), and the same for 16 sampled near-tie tokens on the GPU's own
selection."""
import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from paper_2608_28511_amd.workloads import PAPER_SHAPES, make_inputs

from gpu_helpers import (LOGIT_RTOL, PROB_RTOL, LazyExperts, ambiguous_tokens, assert_bf16_close,
                         check_permutation_props, check_tie_choice, np64, npi)
from test_gpu_layer import DEV, _rows, run_layer

pytestmark = pytest.mark.gpu
N_SAMPLES = 16


@pytest.mark.parametrize("name", list(PAPER_SHAPES))
def test_paper_latent_layer(name):
    s = PAPER_SHAPES[name]
    S, E, K = s.S, s.E, s.K
    inp = make_inputs(s, device=DEV)
    out = run_layer(s, inp)
    x, Wr, Wd, Wu = np64(inp["x"]), np64(inp["Wr"]), np64(inp["Wdown"]), np64(inp["Wup"])

    # router input: one bf16 rounding of an fp32 sum over H terms
    z = O.latent_down(x, Wd, round_payload=False)
    xr_ref = O.round_bf16(z)
    xr_gpu = np64(out["x_lat"])
    assert_bf16_close(xr_gpu, xr_ref, f"{name} x_lat")
    bound = 2.0 ** -8 * np.abs(z) + s.H * 2.0 ** -24 * (np.abs(x) @ np.abs(Wd))
    assert np.all(np.abs(xr_gpu - z) <= bound), "x_lat outside the fp32/bf16 error bound"
    dx = np.abs(xr_gpu - xr_ref)
    del z, xr_gpu

    # logits from each side's own router input
    logits32 = O.router_logits(xr_ref, Wr, None)
    logits_ref = logits32.astype(np.float64)
    tau = LOGIT_RTOL * np.maximum(np.abs(logits_ref), 1.0) + dx @ np.abs(Wr)
    assert np.all(np.abs(np64(out["logits"]) - logits_ref) <= tau), "logits"
    tau_t = tau.max(axis=1)
    del dx, tau

    # routing: exact away from near ties, a valid selection within them
    idx_ref, p_ref = O.route(logits32, K)
    idx_gpu, p_gpu = npi(out["topk_idx"]), np64(out["topk_prob"])
    amb = ambiguous_tokens(logits_ref, K, tau_t)
    ok = ~amb
    assert np.array_equal(idx_gpu[ok], idx_ref[ok]), "top-K of unambiguous tokens"
    rel = np.abs(p_gpu[ok] - p_ref[ok]) / np.maximum(p_ref[ok], 1e-30)
    assert np.all((rel <= PROB_RTOL + 2 * tau_t[ok, None]) | (p_ref[ok] == p_gpu[ok])), "probs"
    for t in np.nonzero(amb)[0]:
        check_tie_choice(logits_ref[t], idx_gpu[t], K, tau_t[t])
    # With E = 512 / 640 unit-scale logits the top K + 1 lie ~0.02 apart
    # (1 / (E phi(q)) at the (1 - K/E) quantile q), so each of the K gaps is
    # within 2 tau (~4e-5) with probability ~0.2%: about 5% of the tokens.
    assert amb.sum() <= S // 10
    inv_gpu = npi(out["inv_perm"])
    check_permutation_props(idx_gpu, npi(out["counts"]), npi(out["offsets"]), npi(out["perm"]), inv_gpu, E, K)

    # dispatch: every routed row is its token's router input row, bit for bit
    inv_t = torch.as_tensor(inv_gpu, device=DEV)
    xd = out["x_disp"].view(torch.int16)[inv_t]
    xr_bits = out["x_lat"].view(torch.int16)
    assert torch.equal(xd.view(S, K, -1), xr_bits[:, None, :].expand(S, K, xr_bits.shape[1])), "x_disp"
    del xd
    assert torch.equal(out["p_disp"][inv_t], out["topk_prob"].reshape(-1)), "p_disp"

    # sampled unambiguous tokens: their routed rows' h and y_disp, and y
    rng = np.random.default_rng(s.seed)
    tok = np.sort(rng.choice(np.nonzero(ok)[0], N_SAMPLES, replace=False))
    ref = O.layer_fwd(x[tok], Wr, LazyExperts(inp["W1"]), LazyExperts(inp["W2"]), K, Wdown=Wd, Wup=Wu,
                      round_payload=True, round_activations=True)
    assert np.array_equal(ref["topk_idx"], idx_ref[tok])
    pos_g = inv_gpu.reshape(S, K)[tok].reshape(-1)
    pos_r = np.asarray(ref["inv_perm"], np.int64)
    assert_bf16_close(_rows(out["h"], pos_g), ref["h"][pos_r], f"{name} h")
    assert_bf16_close(_rows(out["y_disp"], pos_g), ref["y_disp"][pos_r], f"{name} y_disp")
    assert_bf16_close(_rows(out["y"], tok), ref["y"], f"{name} y")
    del ref

    # sampled near-tie tokens: the GPU's own selection evaluated by the oracle
    tie = np.nonzero(amb)[0]
    if tie.size:
        tie = np.sort(rng.choice(tie, min(N_SAMPLES, tie.size), replace=False))
        sel = idx_gpu[tie]
        p_c = O.routing_probs(logits32[tie], sel)
        rel = np.abs(p_gpu[tie] - p_c) / np.maximum(p_c, 1e-30)
        assert np.all(rel <= PROB_RTOL + 2 * tau_t[tie, None]), "probs of near-tie tokens"
        _, off_c, _, inv_c = O.expert_permutation(sel, E)
        xd_c, pd_c = O.dispatch(xr_ref[tie], p_c, inv_c, K)
        _, h_c, yd_c = O.expert_ffn(xd_c, off_c, LazyExperts(inp["W1"]), LazyExperts(inp["W2"]),
                                    round_payload=True, round_hidden=True)
        y_c = O.latent_up(O.round_bf16(O.combine(yd_c, pd_c, inv_c, tie.size, K)), Wu)
        pos_g = inv_gpu.reshape(S, K)[tie].reshape(-1)
        assert_bf16_close(_rows(out["h"], pos_g), h_c[inv_c], f"{name} h (near ties)")
        assert_bf16_close(_rows(out["y_disp"], pos_g), yd_c[inv_c], f"{name} y_disp (near ties)")
        assert_bf16_close(_rows(out["y"], tie), y_c, f"{name} y (near ties)")
