"""Pins for the oracle's experts, latent projections, backward and Eq. 1."""
import json

import numpy as np
import pytest

from oracle import moe_oracle as O
from paper_2608_28511_amd.workloads import make_topk_indices


def _perm_matrix(pi):
    """P with P[d, pi[d]] = 1, so (x @ P)[:, pi[d]] = x[:, d]."""
    n = len(pi)
    P = np.zeros((n, n))
    P[np.arange(n), pi] = 1.0
    return P


def test_permutation_matrix_experts_closed_form():
    """W1[e] = P_e and W2[e] = c_e * Q_e give y_disp[r] = c_e * relu(x)^2
    scattered by pi_e then sigma_e: catches a transposed weight (which
    would apply the inverse permutation) and a wrong expert (wrong c_e)."""
    rng = np.random.default_rng(0)
    S, D, E, K = 24, 10, 4, 2
    pis = [rng.permutation(D) for _ in range(E)]
    sig = [rng.permutation(D) for _ in range(E)]
    c = [1.0, 2.0, -3.0, 0.5]
    W1 = np.stack([_perm_matrix(pis[e]) for e in range(E)])
    W2 = np.stack([c[e] * _perm_matrix(sig[e]) for e in range(E)])
    x = rng.standard_normal((S, D))
    idx = make_topk_indices(S, E, K, seed=1).numpy()
    _, offsets, perm, inv = O.expert_permutation(idx, E)
    xd, _ = O.dispatch(x, None, inv, K)
    u, h, yd = O.expert_ffn(xd, offsets, W1, W2, round_payload=False)
    for pos in range(S * K):
        t, k = divmod(int(perm[pos]), K)
        e = int(idx[t, k])
        ref_u = np.empty(D)
        ref_u[pis[e]] = x[t]
        ref_y = np.empty(D)
        ref_y[sig[e][pis[e]]] = c[e] * np.maximum(x[t], 0) ** 2
        assert np.array_equal(u[pos], ref_u)
        assert np.allclose(yd[pos], ref_y, rtol=0, atol=1e-14)


def test_expert_ffn_brute_force_integers():
    """Tiny integer inputs: every product and sum is exact, so a triple loop
    in plain Python must agree bit for bit."""
    rng = np.random.default_rng(2)
    S, D, F, E, K = 6, 4, 5, 3, 2
    x = rng.integers(-2, 3, (S, D)).astype(np.float64)
    W1 = rng.integers(-2, 3, (E, D, F)).astype(np.float64)
    W2 = rng.integers(-2, 3, (E, F, D)).astype(np.float64)
    idx = make_topk_indices(S, E, K, seed=3).numpy()
    _, offsets, perm, inv = O.expert_permutation(idx, E)
    xd, _ = O.dispatch(x, None, inv, K)
    u, h, yd = O.expert_ffn(xd, offsets, W1, W2, round_payload=False)
    for t in range(S):
        for k in range(K):
            e = int(idx[t, k])
            pos = int(inv[t * K + k])
            uu = [sum(x[t, d] * W1[e, d, f] for d in range(D)) for f in range(F)]
            hh = [max(v, 0.0) ** 2 for v in uu]
            yy = [sum(hh[f] * W2[e, f, d] for f in range(F)) for d in range(D)]
            assert u[pos].tolist() == uu and h[pos].tolist() == hh and yd[pos].tolist() == yy


def test_expert_ffn_rounds_only_the_payload():
    rng = np.random.default_rng(4)
    S, D, F, E, K = 16, 8, 12, 4, 2
    x = O.round_bf16(rng.standard_normal((S, D)))
    W1 = rng.standard_normal((E, D, F))
    W2 = rng.standard_normal((E, F, D))
    idx = make_topk_indices(S, E, K, seed=4).numpy()
    _, offsets, perm, inv = O.expert_permutation(idx, E)
    xd, _ = O.dispatch(x, None, inv, K)
    u0, h0, y0 = O.expert_ffn(xd, offsets, W1, W2, round_payload=False)
    u1, h1, y1 = O.expert_ffn(xd, offsets, W1, W2, round_payload=True)
    assert np.array_equal(u0, u1) and np.array_equal(h0, h1)
    assert np.array_equal(y1, O.round_bf16(y0)) and not np.array_equal(y0, y1)


def test_expert_ffn_rounds_the_hidden_activation_on_request():
    """Hand-worked: u = 1 + 2^-5 gives h = 1 + 2^-4 + 2^-10, which bf16 (7
    fraction bits) rounds to 1 + 2^-4; with W2 = 1 the expert output is
    exactly that rounded h with round_hidden, and the unrounded h without."""
    xd = np.array([[1.0, 2.0 ** -5]])
    W1 = np.array([[[1.0], [1.0]]])
    W2 = np.array([[[1.0, 0.0]]])
    off = np.array([0, 1])
    _, h, y = O.expert_ffn(xd, off, W1, W2, round_payload=False, round_hidden=True)
    assert h[0, 0] == 1 + 2.0 ** -4 and y[0, 0] == 1 + 2.0 ** -4
    _, h, y = O.expert_ffn(xd, off, W1, W2, round_payload=False)
    assert h[0, 0] == 1 + 2.0 ** -4 + 2.0 ** -10 and y[0, 0] == h[0, 0]


def test_layer_fwd_bf16_activations_round_the_latent_combine():
    """Hand-worked latent layer: two experts share a token with equal logits
    (p = 1/2 each), their outputs are 1 and 1 + 2^-7, so the combined latent
    value is 1 + 2^-8, exactly half a bf16 step above 1: with BF16
    activations it rounds to even (1) before the identity up projection;
    without, it passes through."""
    x = np.array([[1.0, 2.0 ** -7]])
    I2 = np.eye(2)
    Wr = np.zeros((2, 2))
    W1 = np.array([[[1.0], [0.0]], [[1.0], [0.0]]])
    W2 = np.array([[[1.0, 0.0]], [[1.0 + 2.0 ** -7, 0.0]]])
    kw = dict(Wdown=I2, Wup=I2)
    out = O.layer_fwd(x, Wr, W1, W2, 2, round_payload=True, round_activations=True, **kw)
    assert np.array_equal(out["topk_prob"], np.array([[0.5, 0.5]], np.float32))
    assert out["y_lat"][0, 0] == 1.0 and out["y"][0, 0] == 1.0
    out = O.layer_fwd(x, Wr, W1, W2, 2, round_payload=True, **kw)
    assert out["y"][0, 0] == 1.0 + 2.0 ** -8


def test_expert_ffn_empty_experts():
    idx = np.array([[1], [1], [3]])
    _, offsets, perm, inv = O.expert_permutation(idx, 5)
    x = np.arange(12.0).reshape(3, 4)
    W1 = np.stack([np.eye(4) * (e + 1) for e in range(5)])
    W2 = np.stack([np.eye(4) for _ in range(5)])
    xd, _ = O.dispatch(x, None, inv, 1)
    u, h, yd = O.expert_ffn(xd, offsets, W1, W2, round_payload=False)
    assert np.array_equal(yd[inv], np.array([(2 * x[0]) ** 2, (2 * x[1]) ** 2, (4 * x[2]) ** 2]))


def test_latent_projections():
    rng = np.random.default_rng(5)
    S, H, D = 9, 12, 4
    x = rng.standard_normal((S, H))
    sel = rng.permutation(H)[:D]
    Wdown = np.zeros((H, D))
    Wdown[sel, np.arange(D)] = 1.0               # picks columns sel of x
    assert np.array_equal(O.latent_down(x, Wdown, round_payload=False), x[:, sel])
    assert np.array_equal(O.latent_down(x, Wdown), O.round_bf16(x[:, sel]))
    Wup = rng.integers(-3, 4, (D, H)).astype(np.float64)
    yl = rng.integers(-3, 4, (S, D)).astype(np.float64)
    got = O.latent_up(yl, Wup)
    for s in range(S):
        for j in range(H):
            assert got[s, j] == sum(yl[s, d] * Wup[d, j] for d in range(D))


def test_layer_fwd_composes_and_reuses_given_logits():
    rng = np.random.default_rng(6)
    S, D, F, E, K = 20, 8, 6, 4, 2
    x = O.round_bf16(rng.standard_normal((S, D)))
    Wr = rng.standard_normal((D, E)) / np.sqrt(D)
    W1 = rng.standard_normal((E, D, F)) / np.sqrt(D)
    W2 = rng.standard_normal((E, F, D)) / np.sqrt(F)
    out = O.layer_fwd(x, Wr, W1, W2, K)
    assert np.array_equal(out["logits"], O.router_logits(x, Wr))
    # a token's output depends on its own row only: a sub-batch gives the same rows
    sub = [3, 11, 17]
    out_sub = O.layer_fwd(x[sub], Wr, W1, W2, K)
    assert np.allclose(out_sub["y"], out["y"][sub], rtol=0, atol=0)
    # routing from supplied logits
    fake = np.zeros((S, E), np.float32)
    fake[:, 3] = 1.0
    out2 = O.layer_fwd(x, Wr, W1, W2, K, logits=fake)
    assert np.all(out2["topk_idx"][:, 0] == 3) and np.all(out2["topk_idx"][:, 1] == 0)


# ---------------------------------------------------------------------------
# Backward: finite differences of the forward
# ---------------------------------------------------------------------------

def _loss(x, W1, W2, p, idx, dy, E, K):
    S = x.shape[0]
    _, offsets, perm, inv = O.expert_permutation(idx, E)
    xd, pd = O.dispatch(x, p.astype(np.float32), inv, K)
    pd = p.reshape(-1)[perm]  # keep float64 weights for differentiation
    _, _, yd = O.expert_ffn(xd, offsets, W1, W2, round_payload=False)
    return float(np.sum(O.combine(yd, pd, inv, S, K) * dy))


def test_backward_matches_central_differences():
    rng = np.random.default_rng(11)
    S, D, F, E, K = 6, 4, 5, 4, 2
    x = rng.standard_normal((S, D))
    W1 = rng.standard_normal((E, D, F))
    W2 = rng.standard_normal((E, F, D))
    p = rng.random((S, K))
    dy = rng.standard_normal((S, D))
    idx = np.array([[0, 2], [2, 0], [0, 1], [2, 3], [0, 2], [1, 2]])  # expert 3 used once
    _, offsets, perm, inv = O.expert_permutation(idx, E)
    xd, _ = O.dispatch(x, None, inv, K)
    pd = p.reshape(-1)[perm]
    u, h, yd = O.expert_ffn(xd, offsets, W1, W2, round_payload=False)
    dyd, dp = O.combine_bwd(dy, yd, pd, inv, K, round_payload=False)
    dxd, dW1, dW2, _ = O.expert_ffn_bwd(xd, u, h, dyd, offsets, W1, W2, round_payload=False)
    dx = O.dispatch_bwd(dxd, inv, S, K)

    eps = 1e-6

    def fd(arr, i):
        a0 = arr[i]
        arr[i] = a0 + eps
        lp = _loss(x, W1, W2, p, idx, dy, E, K)
        arr[i] = a0 - eps
        lm = _loss(x, W1, W2, p, idx, dy, E, K)
        arr[i] = a0
        return (lp - lm) / (2 * eps)

    for i in [(0, 0), (2, 3), (5, 1)]:
        assert abs(fd(x, i) - dx[i]) < 1e-6 * max(1, abs(dx[i]))
    for i in [(0, 1, 2), (3, 0, 4), (2, 3, 1)]:
        assert abs(fd(W1, i) - dW1[i]) < 1e-6 * max(1, abs(dW1[i]))
    for i in [(0, 4, 3), (3, 2, 0), (1, 0, 1)]:
        assert abs(fd(W2, i) - dW2[i]) < 1e-6 * max(1, abs(dW2[i]))
    for i in [(0, 0), (3, 1), (5, 0)]:
        assert abs(fd(p, i) - dp[i]) < 1e-6 * max(1, abs(dp[i]))


def test_backward_dead_expert_zero_and_adjoint():
    rng = np.random.default_rng(12)
    S, D, F, E, K = 10, 6, 7, 5, 2
    idx = np.array([[0, 1]] * 5 + [[1, 3]] * 5)       # experts 2 and 4 receive nothing
    _, offsets, perm, inv = O.expert_permutation(idx, E)
    x = rng.standard_normal((S, D))
    W1 = rng.standard_normal((E, D, F))
    W2 = rng.standard_normal((E, F, D))
    xd, _ = O.dispatch(x, None, inv, K)
    u, h, yd = O.expert_ffn(xd, offsets, W1, W2, round_payload=False)
    dyd = rng.standard_normal((S * K, D))
    dxd, dW1, dW2, du = O.expert_ffn_bwd(xd, u, h, dyd, offsets, W1, W2)
    for e in (2, 4):
        assert np.all(dW1[e] == 0.0) and np.all(dW2[e] == 0.0)
    # linear part adjoint: <du, x_disp W1> summed over experts equals <dW1, W1>
    lhs = sum(np.sum(du[offsets[e]:offsets[e + 1]] * (xd[offsets[e]:offsets[e + 1]] @ W1[e]))
              for e in range(E))
    assert abs(lhs - np.sum(dW1 * W1)) < 1e-9 * max(1, abs(lhs))


# ---------------------------------------------------------------------------
# Eq. 1
# ---------------------------------------------------------------------------

def test_eq1_closed_form_equals_route_decomposition():
    """Eq. 1's per-step volume equals forward dispatch (hidden + probability)
    plus forward combine, doubled for the inverse routes of the backward
    pass (the q = 6 footnote of Section 4.1)."""
    for (L, S, G, K, D) in [(23, 8192, 768, 6, 2688), (8, 8192, 768, 7, 2688), (1, 1, 1, 1, 1)]:
        assert O.ep_volume_per_step(L, S, G, K, D) == L * S * G * K * (4 * D * 2 + 2 * 4)


def test_eq1_printed_reductions(golden_dir):
    g = json.loads((golden_dir / "eq1_volume.json").read_text())
    S, G, D, K = 8192, 768, 2688, 6
    base = O.ep_volume_per_step(g["calls"]["L_E"]["baseline"], S, G, K, D)
    for v in ("switch", "ce"):
        L = g["calls"]["L_E"][v]
        red = 100 * (1 - O.ep_volume_per_step(L, S, G, K, D) / base)
        assert round(red, 1) == g["calls"]["printed_reduction_pct"][v]
        # same layers at 1.5x K_base: the probability term scales with K too
        Kx = g["volume_at_1p5K"]["K_factor"] * K
        red15 = 100 * (1 - L * Kx / (g["calls"]["L_E"]["baseline"] * K))
        vol15 = O.ep_volume_per_step(L, S, G, 9, D) / O.ep_volume_per_step(
            g["calls"]["L_E"]["baseline"], S, G, 6, D)
        assert round(100 * (1 - vol15), 1) == g["volume_at_1p5K"]["printed_reduction_pct"][v]
        assert round(red15, 1) == g["volume_at_1p5K"]["printed_reduction_pct"][v]
    lk = g["LE_K"]
    vb = O.ep_volume_per_step(lk["baseline"]["L_E"], S, G, lk["baseline"]["K"], D)
    vc = O.ep_volume_per_step(lk["ce"]["L_E"], S, G, lk["ce"]["K"], D)
    assert lk["baseline"]["L_E"] * lk["baseline"]["K"] == lk["baseline"]["printed_product"]
    assert lk["ce"]["L_E"] * lk["ce"]["K"] == lk["ce"]["printed_product"]
    assert round(100 * (1 - vc / vb), 1) == lk["printed_reduction_pct"]
