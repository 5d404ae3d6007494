"""Pins of the oracle's router and whole-layer backward (CPU only).

router_bwd is checked against central finite differences of the oracle's own
forward functions (routing_probs on perturbed scores, router_logits on
perturbed x / Wr / bias), with the expert selection held at the base point;
layer_bwd against directional finite differences of layer_fwd, which is
pinned separately.  A dropped term, a wrong sign or a transposed operand in
the backward changes these derivatives by O(1).
"""
import math

import numpy as np
import pytest

from oracle import moe_oracle as O


def _probs_loss(s, idx, dp):
    return float(np.sum(dp * O.routing_probs(s, idx).astype(np.float64)))


def test_router_bwd_ds_matches_finite_differences():
    rng = np.random.default_rng(11)
    S, E, K = 6, 7, 3
    s0 = rng.normal(size=(S, E)) * 2.0
    idx = O.topk_select(s0.astype(np.float32), K)
    p0 = O.routing_probs(s0, idx)
    dp = rng.normal(size=(S, K))
    ds, _, _, _ = O.router_bwd(np.zeros((S, 4)), np.zeros((4, E)), idx, p0, dp)
    eps = 1e-3
    fd = np.zeros((S, E))
    for t in range(S):
        for e in range(E):
            sp, sm = s0.copy(), s0.copy()
            sp[t, e] += eps
            sm[t, e] -= eps
            fd[t, e] = (_probs_loss(sp, idx, dp) - _probs_loss(sm, idx, dp)) / (2 * eps)
    # scores off the selection do not move the renormalised probabilities
    sel = np.zeros((S, E), bool)
    np.put_along_axis(sel, idx.astype(np.int64), True, axis=1)
    assert np.all(ds[~sel] == 0.0)
    assert np.max(np.abs(fd[~sel])) < 1e-4
    assert np.allclose(ds, fd, atol=2e-4), np.max(np.abs(ds - fd))


def test_router_bwd_weight_bias_input_match_finite_differences():
    rng = np.random.default_rng(12)
    S, D, E, K = 5, 6, 8, 3
    x = rng.normal(size=(S, D))
    Wr = rng.normal(size=(D, E)) * 0.7
    b = rng.normal(size=E)
    idx = O.topk_select(O.router_logits(x, Wr, b), K)
    p0 = O.routing_probs(O.router_logits(x, Wr, b), idx)
    dp = rng.normal(size=(S, K))
    _, dWr, dbias, dx = O.router_bwd(x, Wr, idx, p0, dp)

    def loss(x_, W_, b_):
        return _probs_loss(O.router_logits(x_, W_, b_).astype(np.float64), idx, dp)

    eps = 1e-2
    for grad, which in ((dWr, 1), (dbias, 2), (dx, 0)):
        for trial in range(3):
            v = rng.normal(size=grad.shape)
            args_p = [x.copy(), Wr.copy(), b.copy()]
            args_m = [x.copy(), Wr.copy(), b.copy()]
            args_p[which] = args_p[which] + eps * v
            args_m[which] = args_m[which] - eps * v
            for a in (args_p, args_m):  # selection unchanged at both points
                assert np.array_equal(O.topk_select(O.router_logits(*a), K), idx)
            fd = (loss(*args_p) - loss(*args_m)) / (2 * eps)
            an = float(np.sum(grad * v))
            assert abs(fd - an) <= 2e-3 * (1.0 + abs(an)), (which, fd, an)


def test_router_bwd_rows_sum_to_zero_and_k1_is_zero():
    rng = np.random.default_rng(13)
    S, D, E = 9, 4, 6
    x = rng.normal(size=(S, D))
    Wr = rng.normal(size=(D, E))
    logits = O.router_logits(x, Wr)
    for K in (1, 2, 4, 6):
        idx = O.topk_select(logits, K)
        p = O.routing_probs(logits, idx)
        dp = rng.normal(size=(S, K))
        ds, dWr, dbias, dx = O.router_bwd(x, Wr, idx, p, dp)
        # a common shift of all scores leaves softmax probabilities unchanged
        # (up to the fp32 rounding of p, whose rows sum to 1 within ~1e-7)
        assert np.allclose(ds.sum(axis=1), 0.0, atol=1e-6)
        assert np.allclose(dbias.sum(), 0.0, atol=1e-5)
        if K == 1:  # a single routed probability is identically 1
            assert np.all(ds == 0.0) and np.all(dWr == 0.0) and np.all(dx == 0.0)


def _layer(rng, latent):
    S, D, E, K, F, H = 6, 8, 5, 2, 12, 16
    din = H if latent else D
    P = dict(
        x=rng.normal(size=(S, din)),
        Wr=rng.normal(size=(D, E)) * 3.0 / math.sqrt(D),
        bias=rng.normal(size=E),
        W1=rng.normal(size=(E, D, F)) / math.sqrt(D),
        W2=rng.normal(size=(E, F, D)) / math.sqrt(F),
    )
    if latent:
        P["Wdown"] = rng.normal(size=(H, D)) / math.sqrt(H)
        P["Wup"] = rng.normal(size=(D, H)) / math.sqrt(D)
    return P, K, rng.normal(size=(S, din))


def _fwd(P, K):
    return O.layer_fwd(P["x"], P["Wr"], P["W1"], P["W2"], K, bias=P["bias"], Wdown=P.get("Wdown"),
                       Wup=P.get("Wup"), round_payload=False, round_latent=False)


@pytest.mark.parametrize("latent", [False, True])
def test_layer_bwd_matches_directional_finite_differences(latent):
    rng = np.random.default_rng(21 + latent)
    P, K, dy = _layer(rng, latent)
    fwd = _fwd(P, K)
    g = O.layer_bwd(fwd, P["x"], P["Wr"], P["W1"], P["W2"], K, dy, Wdown=P.get("Wdown"),
                    Wup=P.get("Wup"), round_payload=False)
    names = {"x": "dx", "Wr": "dWr", "bias": "dbias", "W1": "dW1", "W2": "dW2"}
    if latent:
        names.update(Wdown="dWdown", Wup="dWup")
    eps = 1e-4
    for pname, gname in names.items():
        for trial in range(2):
            v = rng.normal(size=P[pname].shape)
            Pp, Pm = dict(P), dict(P)
            Pp[pname] = P[pname] + eps * v
            Pm[pname] = P[pname] - eps * v
            fp, fm = _fwd(Pp, K), _fwd(Pm, K)
            assert np.array_equal(fp["topk_idx"], fwd["topk_idx"])
            assert np.array_equal(fm["topk_idx"], fwd["topk_idx"])
            fd = (np.sum(dy * fp["y"]) - np.sum(dy * fm["y"])) / (2 * eps)
            an = float(np.sum(g[gname] * v))
            assert abs(fd - an) <= 1e-3 * (1.0 + abs(an)), (pname, fd, an)
