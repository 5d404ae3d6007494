"""Pins of the oracle's production router (Section 5.2): sigmoid scores with
a selection-only expert bias, the sequence-level balance loss, the shared
expert, and their backward passes.  CPU only."""
import itertools
import json
import math
from pathlib import Path

import numpy as np
import pytest

from oracle import moe_oracle as O

GOLD = json.loads((Path(__file__).parent / "golden" / "sigmoid_route_handworked.json").read_text())


def _num(v):
    return {"ln3": math.log(3.0), "-ln3": -math.log(3.0), "ln7": math.log(7.0)}.get(v, v)


def _arr(rows):
    return np.array([[_num(v) for v in r] for r in rows], dtype=np.float64)


def _tie_free_logits(rng, S, E, scale=2.0):
    while True:
        z = (rng.normal(size=(S, E)) * scale).astype(np.float32)
        if len(np.unique(z)) == z.size:
            return z


@pytest.mark.parametrize("case", GOLD["route_cases"])
def test_sigmoid_route_handworked(case):
    logits = _arr(case["logits"]).astype(np.float32)
    idx, g = O.sigmoid_route(logits, case["K"], case["bias"])
    assert idx.tolist() == case["idx"], case["why"]
    np.testing.assert_allclose(g, np.array(case["gates"]), rtol=2e-7, err_msg=case["why"])


@pytest.mark.parametrize("case", GOLD["aux_cases"])
def test_seq_aux_loss_handworked(case):
    logits = _arr(case["logits"]).astype(np.float32)
    idx = O.sigmoid_topk_select(logits, case["K"])
    loss = O.seq_aux_loss(logits, idx, case["seq_len"], 1e-4)
    assert abs(loss - 1e-4 * case["loss_over_coeff"]) <= 1e-4 * 1e-6, case["why"]


def test_zero_bias_selection_equals_logit_topk():
    # sigmoid is strictly increasing, so without a bias the picks are the
    # top-K logits (the softmax router's selection, pinned separately)
    rng = np.random.default_rng(3)
    for K in (1, 2, 5, 8):
        z = _tie_free_logits(rng, 64, 8)
        assert np.array_equal(O.sigmoid_topk_select(z, K), O.topk_select(z, K))


def test_equal_logits_rank_by_bias():
    rng = np.random.default_rng(4)
    E, K = 9, 4
    bias = rng.normal(size=E)
    z = np.zeros((3, E), np.float32)
    want = np.argsort(-bias, kind="stable")[:K]
    assert np.all(O.sigmoid_topk_select(z, K, bias) == want[None, :])


def test_selection_brute_force():
    # every ordered K-tuple of distinct experts; the chosen one must be the
    # lexicographic best under (key descending, index ascending)
    rng = np.random.default_rng(5)
    E, K = 5, 3
    for _ in range(40):
        z = np.round(rng.normal(size=(1, E)) * 2) / 2          # quantised: ties happen
        z = z.astype(np.float32)
        bias = np.round(rng.normal(size=E) * 2) / 4
        key = [1.0 / (1.0 + math.exp(-float(z[0, e]))) + bias[e] for e in range(E)]
        best = max(itertools.permutations(range(E), K),
                   key=lambda tup: [(key[e], -e) for e in tup])
        assert O.sigmoid_topk_select(z, K, bias)[0].tolist() == list(best)


def test_gate_closed_forms():
    rng = np.random.default_rng(6)
    z = _tie_free_logits(rng, 32, 6)
    bias = rng.normal(size=6)
    # K = 1: a single routed weight is exactly 1
    _, g1 = O.sigmoid_route(z, 1, bias)
    assert np.all(g1 == 1.0)
    # K = 2 with opposite logits: s(-l) = 1 - s(l), so g0 = sigmoid(l0)
    l0 = rng.normal(size=16) * 3
    z2 = np.stack([l0, -l0, np.full(16, -30.0)], axis=1).astype(np.float32)
    idx = np.tile(np.array([[0, 1]]), (16, 1))
    g = O.sigmoid_gates(z2, idx)
    want = 1.0 / (1.0 + np.exp(-z2[:, 0].astype(np.float64)))
    np.testing.assert_allclose(g[:, 0], want, rtol=2e-7)
    # equal selected scores share the weight equally
    ze = np.zeros((4, 6), np.float32)
    _, ge = O.sigmoid_route(ze, 3, bias)
    np.testing.assert_allclose(ge, 1.0 / 3.0, rtol=1e-7)
    # rows sum to one; the bias does not enter the weights for a given pick
    idx, g = O.sigmoid_route(z, 4, bias)
    assert np.allclose(g.astype(np.float64).sum(axis=1), 1.0, atol=4 * 2.0 ** -24)
    np.testing.assert_array_equal(O.sigmoid_gates(z, idx), g)


def test_aux_loss_uniform_scores_give_coeff():
    # equal logits in a row: every normalised score is 1/E, so
    # sum_e f_e P_e = (1/E) sum_e f_e = 1 whatever the routing
    rng = np.random.default_rng(7)
    S, E, K, T = 48, 8, 3, 16
    z = np.repeat(rng.normal(size=(S, 1)), E, axis=1).astype(np.float32)
    bias = rng.normal(size=E)
    idx = O.sigmoid_topk_select(z, K, bias)
    assert abs(O.seq_aux_loss(z, idx, T, 1e-4) - 1e-4) <= 1e-16


def test_aux_loss_sequence_structure():
    rng = np.random.default_rng(8)
    S, E, K, T = 24, 6, 2, 12
    z = _tie_free_logits(rng, S, E)
    idx = O.sigmoid_topk_select(z, K)
    L = O.seq_aux_loss(z, idx, T, 1.0)
    # the mean of the two sequences' own losses
    L0 = O.seq_aux_loss(z[:T], idx[:T], T, 1.0)
    L1 = O.seq_aux_loss(z[T:], idx[T:], T, 1.0)
    assert abs(L - 0.5 * (L0 + L1)) <= 1e-14
    # token order inside a sequence does not matter
    p = np.concatenate([rng.permutation(T), T + rng.permutation(T)])
    assert abs(O.seq_aux_loss(z[p], idx[p], T, 1.0) - L) <= 1e-14
    # linear in the coefficient
    assert abs(O.seq_aux_loss(z, idx, T, 3e-4) - 3e-4 * L) <= 1e-16
    with pytest.raises(ValueError):
        O.seq_aux_loss(z, idx, 10, 1.0)


def _fd(f, x, v, eps=1e-6):
    return (f(x + eps * v) - f(x - eps * v)) / (2 * eps)


def test_aux_loss_bwd_finite_differences():
    rng = np.random.default_rng(9)
    S, E, K, T = 16, 7, 3, 8
    z = rng.normal(size=(S, E))
    idx = O.sigmoid_topk_select(z.astype(np.float32), K)
    g = O.seq_aux_loss_bwd(z, idx, T, 0.5)
    # sigmoid_scores reads fp32 logits; differentiate a float64 copy of the same formula path
    f = lambda zz: _aux64(zz, idx, T, 0.5)
    for _ in range(4):
        v = rng.normal(size=z.shape)
        assert abs(_fd(f, z, v) - np.sum(g * v)) <= 1e-7 * (1 + abs(np.sum(g * v)))


def _aux64(z, idx, T, coeff):
    # the loss with float64 logits (sigmoid_scores rounds its input to fp32,
    # which would swamp a finite difference); same steps as seq_aux_loss
    s = 1.0 / (1.0 + np.exp(-z))
    S, E = z.shape
    K = idx.shape[1]
    sn = s / s.sum(axis=1, keepdims=True)
    tot = 0.0
    for b in range(S // T):
        r = slice(b * T, (b + 1) * T)
        f = np.bincount(idx[r].ravel(), minlength=E) * (E / (K * T))
        tot += np.sum(f * sn[r].mean(axis=0))
    return coeff * tot / (S // T)


def test_sigmoid_gate_bwd_finite_differences():
    rng = np.random.default_rng(10)
    S, E = 12, 6
    for K in (1, 2, 4):
        z = rng.normal(size=(S, E))
        idx = O.sigmoid_topk_select(z.astype(np.float32), K)
        dg = rng.normal(size=(S, K))
        an = O.sigmoid_gate_bwd(z, idx, dg)

        def f(zz):
            s = 1.0 / (1.0 + np.exp(-zz))
            sel = np.take_along_axis(s, idx.astype(np.int64), axis=1)
            return np.sum(dg * sel / sel.sum(axis=1, keepdims=True))

        for _ in range(3):
            v = rng.normal(size=z.shape)
            assert abs(_fd(f, z, v) - np.sum(an * v)) <= 1e-7 * (1 + abs(np.sum(an * v)))
        if K == 1:
            assert np.all(an == 0.0)


def test_router_linear_bwd_finite_differences():
    rng = np.random.default_rng(11)
    x, W, b = rng.normal(size=(9, 5)), rng.normal(size=(5, 4)), rng.normal(size=4)
    dl = rng.normal(size=(9, 4))
    dW, db, dx = O.router_linear_bwd(x, W, dl)
    f = lambda xx, WW, bb: np.sum(dl * (xx @ WW + bb))
    for _ in range(2):
        vx, vW, vb = rng.normal(size=x.shape), rng.normal(size=W.shape), rng.normal(size=b.shape)
        assert abs(_fd(lambda t: f(x + t * vx, W, b), 0.0, 1.0) - np.sum(dx * vx)) < 1e-6
        assert abs(_fd(lambda t: f(x, W + t * vW, b), 0.0, 1.0) - np.sum(dW * vW)) < 1e-6
        assert abs(_fd(lambda t: f(x, W, b + t * vb), 0.0, 1.0) - np.sum(db * vb)) < 1e-6


def test_expert_bias_update_closed_form():
    b = np.array([0.5, -0.25, 0.0, 1.0])
    counts = np.array([30, 10, 20, 20])        # mean 20
    np.testing.assert_array_equal(O.expert_bias_update(b, counts, 1e-3),
                                  [0.5 - 1e-3, -0.25 + 1e-3, 0.0, 1.0])


def test_shared_expert_is_one_expert_over_all_rows():
    rng = np.random.default_rng(12)
    S, D, F = 10, 6, 14
    x = rng.normal(size=(S, D))
    W1, W2 = rng.normal(size=(1, D, F)), rng.normal(size=(1, F, D))
    u, h, y = O.shared_expert(x, W1[0], W2[0])
    u1, h1, y1 = O.expert_ffn(x, np.array([0, S]), W1, W2, round_payload=False)
    np.testing.assert_allclose(y, y1, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(h, h1, rtol=1e-13, atol=1e-13)
    # identity weights: relu(x)^2, elementwise
    I = np.eye(D)
    np.testing.assert_array_equal(O.shared_expert(x, I, I)[2], np.maximum(x, 0) ** 2)


def test_shared_expert_bwd_finite_differences():
    rng = np.random.default_rng(13)
    S, D, F = 7, 5, 9
    x, W1, W2 = rng.normal(size=(S, D)), rng.normal(size=(D, F)), rng.normal(size=(F, D))
    dy = rng.normal(size=(S, D))
    u, h, _ = O.shared_expert(x, W1, W2)
    dx, dW1, dW2 = O.shared_expert_bwd(x, u, h, dy, W1, W2)
    f = lambda xx, A, B: np.sum(dy * O.shared_expert(xx, A, B)[2])
    for _ in range(2):
        vx, v1, v2 = rng.normal(size=x.shape), rng.normal(size=W1.shape), rng.normal(size=W2.shape)
        for an, g in ((dx, lambda t: f(x + t * vx, W1, W2)), (dW1, lambda t: f(x, W1 + t * v1, W2)),
                      (dW2, lambda t: f(x, W1, W2 + t * v2))):
            v = vx if an is dx else (v1 if an is dW1 else v2)
            assert abs(_fd(g, 0.0, 1.0, 1e-5) - np.sum(an * v)) <= 1e-6 * (1 + abs(np.sum(an * v)))


def _prod_layer(rng, latent):
    S, D, E, K, F, H, Fs, T = 8, 8, 5, 2, 12, 16, 10, 4
    din = H if latent else D
    P = dict(x=rng.normal(size=(S, din)), Wr=rng.normal(size=(D, E)) * 3.0 / math.sqrt(D),
             bias=rng.normal(size=E), W1=rng.normal(size=(E, D, F)) / math.sqrt(D),
             W2=rng.normal(size=(E, F, D)) / math.sqrt(F), Ws1=rng.normal(size=(din, Fs)) / math.sqrt(din),
             Ws2=rng.normal(size=(Fs, din)) / math.sqrt(Fs))
    if latent:
        P["Wdown"] = rng.normal(size=(H, D)) / math.sqrt(H)
        P["Wup"] = rng.normal(size=(D, H)) / math.sqrt(D)
    sel_bias = rng.normal(size=E) * 0.3
    return P, K, T, sel_bias, rng.normal(size=(S, din))


def _prod_fwd(P, K, T, sel_bias, coeff):
    return O.layer_fwd(P["x"], P["Wr"], P["W1"], P["W2"], K, bias=P["bias"], Wdown=P.get("Wdown"),
                       Wup=P.get("Wup"), round_payload=False, round_latent=False, score="sigmoid",
                       sel_bias=sel_bias, Ws1=P["Ws1"], Ws2=P["Ws2"], seq_len=T, aux_coeff=coeff)


@pytest.mark.parametrize("latent", [False, True])
def test_production_layer_bwd_directional_finite_differences(latent):
    # loss = <dy, y> + aux_loss; a large coefficient so its gradient shows.
    # The forward rounds logits to fp32 (~1e-7 absolute), so the step is 1e-3
    # to keep that noise below the tolerance; the seeds leave a selection gap
    # (K-th vs (K+1)-th key) of 0.077 and 0.14, far above the step's effect.
    # The loss depends on the selected set only, so slot order may swap.
    rng = np.random.default_rng(37 + latent)
    P, K, T, sb, dy = _prod_layer(rng, latent)
    coeff = 0.5
    fwd = _prod_fwd(P, K, T, sb, coeff)
    g = O.layer_bwd(fwd, P["x"], P["Wr"], P["W1"], P["W2"], K, dy, Wdown=P.get("Wdown"),
                    Wup=P.get("Wup"), round_payload=False, score="sigmoid", Ws1=P["Ws1"],
                    Ws2=P["Ws2"], seq_len=T, aux_coeff=coeff)
    names = {"x": "dx", "Wr": "dWr", "bias": "dbias", "W1": "dW1", "W2": "dW2",
             "Ws1": "dWs1", "Ws2": "dWs2"}
    if latent:
        names.update(Wdown="dWdown", Wup="dWup")
    eps = 1e-3
    loss = lambda f: np.sum(dy * f["y"]) + f["aux_loss"]
    same_set = lambda a, b: np.array_equal(np.sort(a, axis=1), np.sort(b, axis=1))
    for pname, gname in names.items():
        v = rng.normal(size=P[pname].shape)
        Pp, Pm = dict(P), dict(P)
        Pp[pname] = P[pname] + eps * v
        Pm[pname] = P[pname] - eps * v
        fp, fm = _prod_fwd(Pp, K, T, sb, coeff), _prod_fwd(Pm, K, T, sb, coeff)
        assert same_set(fp["topk_idx"], fwd["topk_idx"]) and same_set(fm["topk_idx"], fwd["topk_idx"])
        fd = (loss(fp) - loss(fm)) / (2 * eps)
        an = float(np.sum(g[gname] * v))
        assert abs(fd - an) <= 1e-3 * (1.0 + abs(an)), (pname, fd, an)


def test_production_layer_output_composition():
    rng = np.random.default_rng(33)
    P, K, T, sb, _ = _prod_layer(rng, False)
    f = _prod_fwd(P, K, T, sb, 1e-4)
    routed = O.combine(f["y_disp"], f["p_disp"], f["inv_perm"], P["x"].shape[0], K)
    np.testing.assert_allclose(f["y"], routed + O.shared_expert(P["x"], P["Ws1"], P["Ws2"])[2], rtol=1e-13,
                               atol=1e-13)
    idx, g = O.sigmoid_route(f["logits"], K, sb)
    np.testing.assert_array_equal(f["topk_idx"], idx)
    np.testing.assert_array_equal(f["topk_prob"], g)
    with pytest.raises(ValueError):
        O.layer_fwd(P["x"], P["Wr"], P["W1"], P["W2"], K, sel_bias=sb)       # softmax + bias
