"""Pins for the oracle's expert permutation, dispatch and combine."""
import json

import numpy as np
import pytest

from oracle import moe_oracle as O
from paper_2608_28511_amd.workloads import make_topk_indices


def _brute_perm(idx, E):
    S, K = idx.shape
    triples = sorted((int(idx[t, k]), t, k) for t in range(S) for k in range(K))
    perm = [t * K + k for (_, t, k) in triples]
    counts = [sum(1 for tr in triples if tr[0] == e) for e in range(E)]
    return counts, perm


def test_handworked_permutation(golden_dir):
    g = json.loads((golden_dir / "perm_handworked.json").read_text())
    counts, offsets, perm, inv = O.expert_permutation(np.array(g["idx"]), g["E"])
    assert counts.tolist() == g["counts"]
    assert offsets.tolist() == g["offsets"]
    assert perm.tolist() == g["perm"]
    assert inv.tolist() == g["inv_perm"]


@pytest.mark.parametrize("S,E,K", [(1, 1, 1), (7, 4, 4), (50, 8, 2), (333, 64, 6), (200, 256, 8)])
def test_permutation_matches_sorted_pairs_and_invariants(S, E, K):
    idx = make_topk_indices(S, E, K, seed=S + E).numpy()
    counts, offsets, perm, inv = O.expert_permutation(idx, E)
    bc, bp = _brute_perm(idx, E)
    assert counts.tolist() == bc
    assert perm.tolist() == bp
    R = S * K
    assert counts.sum() == R and offsets[0] == 0 and offsets[-1] == R
    assert np.all(np.diff(offsets) >= 0)
    assert sorted(perm.tolist()) == list(range(R))          # bijection
    assert np.all(inv[perm] == np.arange(R))                 # inverse
    for e in range(E):
        seg = perm[offsets[e]:offsets[e + 1]]
        assert np.all(idx.reshape(-1)[seg] == e)
        assert np.all(np.diff(seg // K) > 0)                 # ascending tokens


def test_permutation_empty_experts_and_rejects_duplicates():
    idx = np.array([[3, 1], [1, 3]])
    counts, offsets, perm, inv = O.expert_permutation(idx, 6)
    assert counts.tolist() == [0, 2, 0, 2, 0, 0]
    assert offsets.tolist() == [0, 0, 2, 2, 4, 4, 4]
    with pytest.raises(ValueError):
        O.expert_permutation(np.array([[1, 1]]), 4)
    with pytest.raises(ValueError):
        O.expert_permutation(np.array([[0, 4]]), 4)


def test_per_expert_load_section_5_3(golden_dir):
    """Uniform routing: CE-MoE experts (192/7) receive 22% fewer routed rows
    than baseline experts (128/6), as printed in Section 5.3."""
    g = json.loads((golden_dir / "eq1_volume.json").read_text())["per_expert_load"]
    S = 128 * 192
    means = {}
    for key in ("baseline", "ce"):
        E, K = g[key]["E"], g[key]["K"]
        idx = ((np.arange(S)[:, None] * K + np.arange(K)[None, :]) % E).astype(np.int32)
        counts, *_ = O.expert_permutation(idx, E)
        assert counts.min() == counts.max()                  # perfectly uniform
        means[key] = counts.mean()
    assert round(100 * (1 - means["ce"] / means["baseline"])) == g["printed_reduction_pct"]


def _setup(S, D, E, K, seed):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((S, D))
    idx = make_topk_indices(S, E, K, seed=seed).numpy()
    p = rng.random((S, K)).astype(np.float32)
    _, offsets, perm, inv = O.expert_permutation(idx, E)
    return rng, x, idx, p, offsets, perm, inv


def test_dispatch_copies_rows_and_eq1_bytes():
    S, D, E, K = 64, 24, 8, 3
    rng, x, idx, p, offsets, perm, inv = _setup(S, D, E, K, 5)
    xd, pd = O.dispatch(x, p, inv, K)
    for pos in range(S * K):
        t, k = divmod(int(perm[pos]), K)
        assert np.array_equal(xd[pos], x[t]) and pd[pos] == p[t, k]
    nbytes = xd.shape[0] * xd.shape[1] * O.B_X + pd.size * O.B_P
    assert nbytes == O.dispatch_payload_bytes(S, K, D) == S * K * (D * 2 + 4)
    # the 8192-token, D=2048, top-6 layer moves 201,523,200 bytes per forward dispatch
    assert O.dispatch_payload_bytes(8192, 6, 2048) == 201_523_200


def test_dispatch_combine_adjoint():
    S, D, E, K = 40, 16, 8, 4
    rng, x, idx, p, offsets, perm, inv = _setup(S, D, E, K, 6)
    g = rng.standard_normal((S * K, D))
    xd, _ = O.dispatch(x, None, inv, K)
    lhs = np.sum(xd * g)
    rhs = np.sum(x * O.dispatch_bwd(g, inv, S, K))
    assert abs(lhs - rhs) <= 1e-10 * max(1.0, abs(lhs))
    yd = rng.standard_normal((S * K, D))
    dy = rng.standard_normal((S, D))
    _, pd = O.dispatch(x, p, inv, K)
    y = O.combine(yd, pd, inv, S, K)
    dyd, dp = O.combine_bwd(dy, yd, pd, inv, K, round_payload=False)
    assert abs(np.sum(y * dy) - np.sum(yd * dyd)) <= 1e-10 * max(1.0, abs(np.sum(y * dy)))
    # dp[t,k] is the derivative of <y, dy> with respect to p[t,k]
    for t in (0, 7, S - 1):
        for k in range(K):
            pos = inv[t * K + k]
            assert abs(dp[t, k] - np.dot(dy[t], yd[pos])) < 1e-12


def test_identity_experts_return_input_exactly():
    """With y_disp = x_disp the combine returns sum_k p_k * x = x; the fp64
    error of that sum is far below half a bf16 ulp, so rounding gives x back."""
    S, D, E, K = 128, 32, 16, 6
    rng = np.random.default_rng(7)
    x = O.round_bf16(rng.standard_normal((S, D)))
    logits = rng.standard_normal((S, E)).astype(np.float32)
    idx, p = O.route(logits, K)
    _, offsets, perm, inv = O.expert_permutation(idx, E)
    xd, pd = O.dispatch(x, p, inv, K)
    y = O.combine(xd, pd, inv, S, K)
    assert np.array_equal(O.round_bf16(y), x)


def test_combine_k1_is_the_permuted_row():
    S, D, E, K = 30, 8, 5, 1
    rng, x, idx, p, offsets, perm, inv = _setup(S, D, E, K, 8)
    yd = rng.standard_normal((S, D))
    y = O.combine(yd, None, inv, S, K)
    assert np.array_equal(y, yd[inv])
