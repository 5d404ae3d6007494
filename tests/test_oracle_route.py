"""Pins for the oracle's router: logits, top-K selection, probabilities.

Every expected value here comes from a method other than the oracle's own:
a full sort per row (brute force), closed forms, exact small-integer
arithmetic, or hand-worked fixtures.
"""
import json
import math

import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from paper_2608_28511_amd.workloads import make_logits


def _brute_topk(row, K):
    """Full sort of expert ids by (NaN last, score descending, id ascending)."""
    vals = [float(v) for v in row]
    order = sorted(range(len(vals)),
                   key=lambda e: (math.isnan(vals[e]), 0.0 if math.isnan(vals[e]) else -vals[e], e))
    return order[:K]


@pytest.mark.parametrize("kind", ["normal", "quantised", "equal", "signed0", "masked", "nan"])
@pytest.mark.parametrize("E,K", [(8, 2), (8, 8), (64, 6), (37, 5), (256, 8), (1, 1)])
def test_topk_matches_full_sort(kind, E, K):
    logits = make_logits(kind, 40, E, seed=E * 31 + K).numpy()
    got = O.topk_select(logits, K)
    for t in range(logits.shape[0]):
        assert list(got[t]) == _brute_topk(logits[t], K), (kind, t, logits[t])


def test_topk_rejects_bad_k():
    with pytest.raises(ValueError):
        O.topk_select(np.zeros((2, 4), np.float32), 5)
    with pytest.raises(ValueError):
        O.topk_select(np.zeros((2, 4), np.float32), 0)


def test_handworked_routes(golden_dir):
    cases = json.loads((golden_dir / "route_handworked.json").read_text())["cases"]
    for c in cases:
        logits = np.array([[float(v) for v in r] for r in c["logits"]], dtype=np.float32)
        idx = O.topk_select(logits, c["K"])
        assert idx.tolist() == c["idx"], c["why"]
        if c["prob"] is None:
            with pytest.raises(ValueError):
                O.routing_probs(logits, idx)
        else:
            p = O.routing_probs(logits, idx)
            np.testing.assert_allclose(p, np.array(c["prob"]), rtol=1e-6, atol=1e-7, err_msg=c["why"])


def test_probs_k1_is_one():
    logits = make_logits("normal", 64, 16, seed=3).numpy()
    idx, p = O.route(logits, 1)
    assert np.all(p == np.float32(1.0))


@pytest.mark.parametrize("K", [2, 3, 5, 7])
def test_probs_equal_scores_are_uniform(K):
    logits = make_logits("equal", 16, 9, seed=K).numpy()
    idx, p = O.route(logits, K)
    assert idx.tolist() == [list(range(K))] * 16
    assert np.all(p == np.float32(1.0 / K))


def test_probs_k2_logistic():
    """For K = 2 the renormalised weight of the best expert is the logistic
    function of the score gap, whatever the other experts hold."""
    logits = make_logits("normal", 200, 12, seed=9).numpy()
    idx, p = O.route(logits, 2)
    s0 = logits[np.arange(200), idx[:, 0]].astype(np.float64)
    s1 = logits[np.arange(200), idx[:, 1]].astype(np.float64)
    ref = 1.0 / (1.0 + np.exp(-(s0 - s1)))
    np.testing.assert_allclose(p[:, 0], ref, rtol=2 ** -23)
    np.testing.assert_allclose(p[:, 1], 1.0 - ref, rtol=2 ** -22, atol=2 ** -26)


@pytest.mark.parametrize("E,K", [(8, 2), (64, 6), (256, 8), (128, 8)])
def test_probs_sum_to_one_and_match_k_only_softmax(E, K):
    """Softmax over E then renormalising over the K picked equals a softmax
    over the K picked scores alone (the normaliser cancels)."""
    logits = make_logits("masked", 100, E, seed=E + K).numpy()
    idx, p = O.route(logits, K)
    assert np.all(np.abs(p.astype(np.float64).sum(axis=1) - 1.0) <= K * 2 ** -23)
    sel = np.take_along_axis(logits.astype(np.float64), idx.astype(np.int64), axis=1)
    z = np.exp(sel - sel[:, :1])
    ref = (z / z.sum(axis=1, keepdims=True)).astype(np.float32)
    assert np.max(np.abs(p.astype(np.float64) - ref) / np.maximum(ref, 1e-30)) <= 2 ** -23 + 1e-12


def test_probs_nan_or_all_masked_rejected():
    with pytest.raises(ValueError):
        O.routing_probs(np.array([[1.0, np.nan]], np.float32), np.array([[0]]))
    with pytest.raises(ValueError):
        O.routing_probs(np.array([[-np.inf, -np.inf]], np.float32), np.array([[0]]))


def test_router_logits_exact_integers_and_bias():
    rng = np.random.default_rng(0)
    x = rng.integers(-3, 4, size=(7, 5)).astype(np.float64)
    Wr = rng.integers(-2, 3, size=(5, 4)).astype(np.float64)
    bias = np.array([0.5, -1.0, 0.0, -np.inf])
    got = O.router_logits(x, Wr, bias)
    assert got.dtype == np.float32
    for t in range(7):
        for e in range(4):
            ref = sum(x[t, d] * Wr[d, e] for d in range(5)) + bias[e]
            assert got[t, e] == np.float32(ref)
    assert np.all(np.isneginf(got[:, 3]))


def test_router_logits_round_once_to_fp32():
    """The float64 sum is rounded once: 1 + 2^-30 is not representable in
    fp32 and must come out as 1.0, and 1 + 2^-23 must survive."""
    x = np.array([[1.0, 1.0]])
    Wr = np.array([[1.0, 1.0], [2.0 ** -30, 2.0 ** -23]])
    got = O.router_logits(x, Wr)
    assert got[0, 0] == np.float32(1.0)
    assert got[0, 1] == np.float32(1.0 + 2.0 ** -23)


def test_round_bf16_matches_library_on_fp32_values():
    rng = np.random.default_rng(1)
    v = np.concatenate([rng.standard_normal(20000).astype(np.float32),
                        (rng.standard_normal(2000) * 1e-38).astype(np.float32),
                        (rng.standard_normal(2000) * 1e37).astype(np.float32)])
    ref = torch.from_numpy(v).to(torch.bfloat16).to(torch.float64).numpy()
    got = O.round_bf16(v.astype(np.float64))
    np.testing.assert_array_equal(got, ref)


def test_round_bf16_ties_overflow_subnormal():
    ulp1 = 2.0 ** -7
    got = O.round_bf16(np.array([1 + ulp1 / 2, 1 + 1.5 * ulp1, -(1 + 1.5 * ulp1), 3.4e38,
                                 1.5 * 2.0 ** -133, 2.0 ** -133, np.inf, -np.inf]))
    assert got[0] == 1.0
    assert got[1] == 1 + 2 * ulp1
    assert got[2] == -(1 + 2 * ulp1)
    assert got[3] == np.inf
    assert got[4] == 2.0 ** -132
    assert got[5] == 2.0 ** -133
    assert got[6] == np.inf and got[7] == -np.inf
    assert np.isnan(O.round_bf16(np.array([np.nan]))[0])
