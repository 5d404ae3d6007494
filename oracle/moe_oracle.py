"""Plain float64 statement of one routed MoE layer (forward, and backward
through the experts and the permutation).

TEST INFRASTRUCTURE ONLY (see the package docstring): slow on purpose, no
blocking, fusion or reordering beyond what each definition states.

Notation (paper, Section 1 and Table 2): S tokens, D dispatch dimension,
E experts, top-K, F per-expert FFN width, H model hidden for a latent
projection, b_x / b_p bytes per dispatched hidden element / routed
probability.  R = S*K routed (token, slot) rows.

Precision.  Arithmetic is float64.  Values are rounded only where the paper
fixes a precision:
  * router logits and routed probabilities are fp32 (b_p = 4 bytes, Eq. 1);
  * every hidden-state payload that crosses the dispatch/combine boundary is
    bf16 (b_x = 2 bytes, Eq. 1): the dispatched activations, the expert
    outputs sent back for the combine, and in the backward pass the gradients
    travelling the inverse routes (footnote on q = 6 in Section 4.1).
Expert-internal values (u, h) and final outputs stay float64.

Pins (each in tests/test_oracle_*.py):
  round_bf16            library conversion on fp32-exact inputs, hand ties
  router_logits         exact small-integer products, bias offsets
  topk_select           brute-force full sort per row; tie / +-0 / -inf / NaN suites
  routing_probs         closed forms (K=1, equal scores, K=2 logistic), sum = 1,
                        K-only softmax agreement, hand-worked fixture
  expert_permutation    brute-force sort of (expert, token) pairs; bijection and
                        segment invariants; hand-worked fixture; Section 5.3 load
  dispatch / combine    Eq. 1 byte count, adjoint identity, identity experts, K=1
  expert_ffn            permutation-matrix experts (closed form), brute-force
                        triple loop on tiny integer inputs, per-expert scaling
  latent_down/up        permutation-matrix projections, brute-force loops
  *_bwd                 float64 central finite differences of the forward;
                        adjoint identities; dead experts give exactly zero dW
  router_bwd            central finite differences of routing_probs and
                        router_logits; rows of ds sum to zero; K = 1 gives 0
  layer_bwd             directional finite differences of the whole layer_fwd
                        (plain and latent, with bias) for every input
  sigmoid_topk_select   zero bias equals topk_select on the logits; equal
                        logits rank by bias; brute-force sort; hand fixture
  sigmoid_gates         K = 1 -> 1; equal scores -> 1/K; K = 2 with opposite
                        logits -> sigmoid(l0); sum = 1; bias-independent;
                        hand fixture (exact fractions)
  seq_aux_loss          uniform scores -> coeff exactly; hand fixture;
                        per-sequence mean (not batch-level); token-order
                        invariance; linear in coeff
  *_bwd (sigmoid, aux)  float64 central finite differences, selection fixed
  expert_bias_update    closed form on a hand example
  shared_expert         one expert over all rows of expert_ffn; identity
                        weights give relu(x)^2; finite differences of the bwd
  e4m3_encode/decode    the library fp8 (E4M3) conversion on every in-range
                        value, codes and midpoints; hand codes of the OCP
                        format; saturation; round trip of all 254 codes
  mx_shared_exponent    closed forms (powers of two, zero, clamping)
  mxfp8_(de)quantize    error bound per element, power-of-two equivariance,
                        block independence, exact round trip of encoded values
  dispatch_mxfp8        rows equal the token's encoding; Eq. 1 byte count
  ep_volume_per_step    the paper's printed reductions (Section 4.1, 4.3)
"""
from __future__ import annotations

import math
from typing import Optional, Sequence

import numpy as np

B_X = 2  # bytes per dispatched hidden element, bf16 (Eq. 1)
B_P = 4  # bytes per routed probability, fp32 (Eq. 1)

__all__ = [
    "B_X", "B_P", "round_bf16", "router_logits", "topk_select", "routing_probs",
    "route", "expert_permutation", "dispatch", "expert_ffn", "combine",
    "latent_down", "latent_up", "layer_fwd", "combine_bwd", "expert_ffn_bwd",
    "dispatch_bwd", "router_bwd", "latent_bwd", "layer_bwd", "sigmoid_scores",
    "sigmoid_topk_select", "sigmoid_gates", "sigmoid_route", "seq_aux_loss",
    "seq_aux_loss_bwd", "sigmoid_gate_bwd", "router_linear_bwd", "expert_bias_update",
    "shared_expert", "shared_expert_bwd", "MX_BLOCK", "E4M3_MAX", "e4m3_encode", "e4m3_decode",
    "mx_shared_exponent", "mxfp8_quantize", "mxfp8_dequantize", "dispatch_mxfp8", "mx_payload_bytes",
    "dispatch_payload_bytes",
    "combine_payload_bytes", "ep_volume_per_step",
]


# ---------------------------------------------------------------------------
# Rounding to the payload precision
# ---------------------------------------------------------------------------

def round_bf16(a) -> np.ndarray:
    """Round to the nearest bfloat16 value (ties to even), returned as float64.

    bf16 keeps 8 significant bits, so a finite value a = m * 2**e with
    0.5 <= |m| < 1 lies on a grid of spacing 2**(e-8); below the smallest
    normal (2**-126) the spacing stays at 2**-133.  Rounding is done directly
    from float64 (no intermediate fp32 step, which could round twice).
    """
    a = np.asarray(a, dtype=np.float64)
    out = a.copy()
    fin = np.isfinite(a)
    v = a[fin]
    _, e = np.frexp(v)
    e = np.maximum(e, -125)
    ulp = np.ldexp(np.ones_like(v), e - 8)
    r = np.rint(v / ulp) * ulp  # np.rint rounds halves to even
    r = np.where(np.abs(r) >= 2.0 ** 128, np.copysign(np.inf, v), r)
    out[fin] = r
    return out


# ---------------------------------------------------------------------------
# Router: logits, top-K selection, routed probabilities
# ---------------------------------------------------------------------------

def router_logits(x_r, Wr, bias=None) -> np.ndarray:
    """logits[t, e] = sum_d x_r[t, d] * Wr[d, e] (+ bias[e]), as fp32.

    The router scores every token against every expert (Section 5.2: MoE
    layers route with a learned router; this workload uses fp32 router
    logits).  Computed in float64 and rounded once to fp32.  An optional
    per-expert bias is added to the logits before the softmax, so it changes
    both which experts are picked and their weights.
    """
    z = np.asarray(x_r, np.float64) @ np.asarray(Wr, np.float64)
    if bias is not None:
        with np.errstate(invalid="ignore"):
            z = z + np.asarray(bias, np.float64)[None, :]
    return z.astype(np.float32)


def topk_select(logits, K: int) -> np.ndarray:
    """Indices of the K highest-scoring experts per token, best first.

    Dropless top-K routing (Section 1): every token keeps exactly K distinct
    experts.  Selection compares the fp32 scores under one total order:
    higher score first, equal scores broken towards the lower expert index,
    -0 equal to +0, NaN below every number including -inf.  The K picks are
    made one after another, each taking the best expert not yet taken.
    Returns int32 [S, K].
    """
    s = np.asarray(logits, dtype=np.float32)
    S, E = s.shape
    if not 1 <= K <= E:
        raise ValueError("need 1 <= K <= E")
    vals = s.astype(np.float64) + 0.0          # -0.0 + 0.0 == +0.0
    nan = np.isnan(vals)
    taken = np.zeros((S, E), dtype=bool)
    idx = np.empty((S, K), dtype=np.int32)
    rows = np.arange(S)
    for k in range(K):
        avail = ~taken
        num = avail & ~nan
        v = np.where(num, vals, -np.inf)
        best = v.max(axis=1) if E else None
        cand = num & (v == best[:, None])
        only_nan = ~num.any(axis=1)
        cand[only_nan] = (avail & nan)[only_nan]
        choice = np.argmax(cand, axis=1)       # first True: the lowest index
        idx[:, k] = choice
        taken[rows, choice] = True
    return idx


def routing_probs(logits, idx) -> np.ndarray:
    """Routed probabilities p[t, k] for the selected experts, as fp32 (b_p).

    Softmax over all E experts, keep the K selected, renormalise them to sum
    to one: p_k = q_{T_k} / sum_{j<K} q_{T_j} with q = softmax(s).  Each row
    must hold no NaN and at least one finite score; -inf entries get q = 0.
    """
    s = np.asarray(logits, dtype=np.float32).astype(np.float64)
    idx = np.asarray(idx)
    if np.isnan(s).any():
        raise ValueError("routing probabilities are undefined for NaN logits")
    m = s.max(axis=1, keepdims=True)
    if not np.isfinite(m).all():
        raise ValueError("each token needs a finite maximum score")
    ex = np.exp(s - m)
    q = ex / ex.sum(axis=1, keepdims=True)
    sel = np.take_along_axis(q, idx.astype(np.int64), axis=1)
    p = sel / sel.sum(axis=1, keepdims=True)
    return p.astype(np.float32)


def route(logits, K: int):
    """topk_select followed by routing_probs: (idx int32 [S,K], p fp32 [S,K])."""
    idx = topk_select(logits, K)
    return idx, routing_probs(logits, idx)


# ---------------------------------------------------------------------------
# Permutation into expert-contiguous order
# ---------------------------------------------------------------------------

def expert_permutation(idx, E: int):
    """Counting sort of the S*K routed rows by expert.

    Dropless, unpadded (Section 1): the expert-contiguous buffer has exactly
    S*K rows.  counts[e] is the number of rows routed to e, offsets the
    exclusive prefix sum (offsets[E] = S*K).  Rows are placed by walking
    tokens in ascending order and, within a token, slots in ascending order,
    each taking the next free position of its expert; so inside every expert
    segment rows appear in ascending token order.
      perm[pos]        = t*K + k  (which routed row sits at position pos)
      inv_perm[t*K+k]  = pos
    """
    idx = np.asarray(idx)
    S, K = idx.shape
    if idx.size and (idx.min() < 0 or idx.max() >= E):
        raise ValueError("expert index out of range")
    for t in range(S):
        if len(set(int(e) for e in idx[t])) != K:
            raise ValueError("a token's K experts must be distinct")
    counts = np.bincount(idx.ravel().astype(np.int64), minlength=E).astype(np.int64)
    offsets = np.zeros(E + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    cursor = offsets[:-1].copy()
    perm = np.empty(S * K, dtype=np.int64)
    inv_perm = np.empty(S * K, dtype=np.int64)
    for t in range(S):
        for k in range(K):
            e = int(idx[t, k])
            pos = int(cursor[e])
            cursor[e] += 1
            perm[pos] = t * K + k
            inv_perm[t * K + k] = pos
    return counts, offsets, perm, inv_perm


# ---------------------------------------------------------------------------
# Dispatch, experts, combine
# ---------------------------------------------------------------------------

def dispatch(x, prob, inv_perm, K: int):
    """The forward dispatch payload (Eq. 1: D*b_x + b_p bytes per routed row).

    Row t*K+k of the token-major expansion goes to position inv_perm[t*K+k]:
    x_disp[pos] = x[t] (bf16 hidden state, copied unchanged) and
    p_disp[pos] = prob[t, k] (fp32 routed probability).
    """
    x = np.asarray(x, np.float64)
    S, D = x.shape
    inv_perm = np.asarray(inv_perm, np.int64)
    x_disp = np.empty((S * K, D), dtype=np.float64)
    x_disp[inv_perm] = np.repeat(x, K, axis=0)
    p_disp = None
    if prob is not None:
        p_disp = np.empty(S * K, dtype=np.float32)
        p_disp[inv_perm] = np.asarray(prob, np.float32).reshape(-1)
    return x_disp, p_disp


def _expert(W, e) -> np.ndarray:
    return np.asarray(W[e], dtype=np.float64)


def expert_ffn(x_disp, offsets, W1, W2, round_payload: bool = True, round_hidden: bool = False):
    """Ungated per-expert FFN over each expert's contiguous segment
    (Section 5.2: grouped GEMM over expert segments; the activation is
    squared-ReLU for this workload since the paper does not state one).

    For expert e and rows r in [offsets[e], offsets[e+1]):
        u[r] = x_disp[r] @ W1[e]          W1[e]: [D, F]
        h[r] = max(u[r], 0)**2
        y_disp[r] = h[r] @ W2[e]          W2[e]: [F, D]
    y_disp is the combine payload and is rounded to bf16 (b_x) unless
    round_payload is False.  With round_hidden the hidden activation h is
    rounded to bf16 before the down projection reads it (the paper trains in
    BF16, Section 5.2: h is a stored bf16 activation tensor); the returned h
    is then the rounded one.  W1/W2 may be any object indexable by expert.
    Returns (u, h, y_disp) as float64.
    """
    x_disp = np.asarray(x_disp, np.float64)
    offsets = np.asarray(offsets, np.int64)
    R, D = x_disp.shape
    E = len(offsets) - 1
    F = None
    u = h = y = None
    for e in range(E):
        a, b = int(offsets[e]), int(offsets[e + 1])
        if a == b:
            continue
        w1 = _expert(W1, e)
        w2 = _expert(W2, e)
        if F is None:
            F = w1.shape[1]
            u = np.zeros((R, F))
            h = np.zeros((R, F))
            y = np.zeros((R, w2.shape[1]))
        u[a:b] = x_disp[a:b] @ w1
        h[a:b] = np.maximum(u[a:b], 0.0) ** 2
        if round_hidden:
            h[a:b] = round_bf16(h[a:b])
        y[a:b] = h[a:b] @ w2
    if F is None:  # no routed rows at all
        F = _expert(W1, 0).shape[1] if E else 0
        u = np.zeros((R, F))
        h = np.zeros((R, F))
        y = np.zeros((R, D))
    if round_payload:
        y = round_bf16(y)
    return u, h, y


def combine(y_disp, p_disp, inv_perm, S: int, K: int) -> np.ndarray:
    """Probability-weighted combine back to token order:
    y[t] = sum_{k<K} p_disp[pos] * y_disp[pos], pos = inv_perm[t*K+k],
    summed in ascending k.  p_disp None means unit weights.  float64 result.
    """
    y_disp = np.asarray(y_disp, np.float64)
    inv = np.asarray(inv_perm, np.int64).reshape(S, K)
    y = np.zeros((S, y_disp.shape[1]))
    for k in range(K):
        pos = inv[:, k]
        w = 1.0 if p_disp is None else np.asarray(p_disp, np.float64)[pos][:, None]
        y = y + w * y_disp[pos]
    return y


def latent_down(x, Wdown, round_payload: bool = True) -> np.ndarray:
    """LatentMoE-style projection to the dispatch dimension (Section 1, the
    dispatch-dimension lever; Table 2 d_latent): x_lat = x @ Wdown.  x_lat is
    what gets dispatched, so it is rounded to bf16 (b_x)."""
    z = np.asarray(x, np.float64) @ np.asarray(Wdown, np.float64)
    return round_bf16(z) if round_payload else z


def latent_up(y_lat, Wup) -> np.ndarray:
    """Projection of the combined latent output back to the model hidden:
    y = y_lat @ Wup (float64)."""
    return np.asarray(y_lat, np.float64) @ np.asarray(Wup, np.float64)


def layer_fwd(x, Wr, W1, W2, K: int, bias=None, Wdown=None, Wup=None,
              logits=None, round_payload: bool = True, round_latent: bool = True,
              round_activations: bool = False,
              score: str = "softmax", sel_bias=None, Ws1=None, Ws2=None,
              seq_len: Optional[int] = None, aux_coeff: float = 0.0, payload: str = "bf16") -> dict:
    """One routed MoE layer forward, in the paper's order (Section 4.1
    footnote: hidden dispatch, probability dispatch, hidden combine):
    [latent down] -> router logits -> top-K + probabilities -> permutation ->
    dispatch -> experts -> combine -> [latent up].

    If ``logits`` is given, routing uses those fp32 scores instead of the
    ones computed here.  ``round_latent`` rounds the projected activations
    (the dispatched, routed input) to bf16; ``round_payload`` rounds the
    expert outputs sent back for the combine.  ``round_activations`` also
    rounds to bf16 the activation tensors a BF16-trained layer stores between
    its products (the paper trains with BF16 precision, Section 5.2): each
    expert's hidden activation h before its down projection, and with a
    latent projection the combined latent output y_lat before the up
    projection.

    The production variant of Section 5.2: ``score="sigmoid"`` routes with
    sigmoid_route (``sel_bias`` steering selection only); ``Ws1``/``Ws2`` add
    the shared expert on the layer input to the layer output; ``aux_coeff``
    (sigmoid scores, batch of whole ``seq_len``-token sequences) adds the
    balance loss as ``aux_loss``.  ``payload="mxfp8"`` sends the dispatched
    hidden states as MX-FP8 (dispatch_mxfp8) and the experts read their
    decoded values.  Returns every intermediate.
    """
    x = np.asarray(x, np.float64)
    S = x.shape[0]
    out = {}
    x_r = x
    if Wdown is not None:
        x_r = latent_down(x, Wdown, round_latent)
        out["x_lat"] = x_r
    if logits is None:
        logits = router_logits(x_r, Wr, bias)
    out["logits"] = np.asarray(logits, np.float32)
    E = out["logits"].shape[1]
    if score == "sigmoid":
        idx, prob = sigmoid_route(out["logits"], K, sel_bias)
    elif score == "softmax" and sel_bias is None:
        idx, prob = route(out["logits"], K)
    else:
        raise ValueError("score is 'softmax' (no selection bias) or 'sigmoid'")
    counts, offsets, perm, inv_perm = expert_permutation(idx, E)
    if payload == "mxfp8":
        xq, xs, p_disp = dispatch_mxfp8(x_r, prob, inv_perm, K)
        x_disp = mxfp8_dequantize(xq, xs)
        out.update(x_q=xq, x_scale=xs)
    elif payload == "bf16":
        x_disp, p_disp = dispatch(x_r, prob, inv_perm, K)
    else:
        raise ValueError("payload is 'bf16' or 'mxfp8'")
    u, h, y_disp = expert_ffn(x_disp, offsets, W1, W2, round_payload, round_hidden=round_activations)
    y = combine(y_disp, p_disp, inv_perm, S, K)
    out.update(topk_idx=idx, topk_prob=prob, counts=counts, offsets=offsets, perm=perm,
               inv_perm=inv_perm, x_disp=x_disp, p_disp=p_disp, u=u, h=h, y_disp=y_disp)
    if Wup is not None:
        if round_activations:
            y = round_bf16(y)
        out["y_lat"] = y
        y = latent_up(y, Wup)
    if Ws1 is not None:
        out["u_s"], out["h_s"], out["y_shared"] = shared_expert(x, Ws1, Ws2)
        y = y + out["y_shared"]
    if aux_coeff:
        if score != "sigmoid":
            raise ValueError("the sequence balance loss is defined on sigmoid scores")
        out["aux_loss"] = seq_aux_loss(out["logits"], idx, seq_len, aux_coeff)
    out["y"] = y
    return out


# ---------------------------------------------------------------------------
# Backward through the combine, the experts and the dispatch
# ---------------------------------------------------------------------------

def combine_bwd(dy, y_disp, p_disp, inv_perm, K: int, round_payload: bool = True):
    """Transpose of the weighted combine (the first inverse route of the
    backward pass, Section 4.1 footnote):
        dy_disp[pos] = p_disp[pos] * dy[t]         (bf16 payload)
        dp[t, k]     = <dy[t], y_disp[pos]>        (gradient of the weight)
    with pos = inv_perm[t*K+k].  Returns (dy_disp, dp) as float64.
    """
    dy = np.asarray(dy, np.float64)
    y_disp = np.asarray(y_disp, np.float64)
    S, D = dy.shape
    inv = np.asarray(inv_perm, np.int64).reshape(S, K)
    dy_disp = np.zeros((S * K, D))
    dp = np.zeros((S, K))
    for k in range(K):
        pos = inv[:, k]
        w = 1.0 if p_disp is None else np.asarray(p_disp, np.float64)[pos][:, None]
        dy_disp[pos] = w * dy
        dp[:, k] = np.sum(dy * y_disp[pos], axis=1)
    if round_payload:
        dy_disp = round_bf16(dy_disp)
    return dy_disp, dp


def expert_ffn_bwd(x_disp, u, h, dy_disp, offsets, W1, W2, round_payload: bool = True):
    """Gradients of expert_ffn along the same expert segments.

    For expert e, rows r in its segment (chain rule of u = x W1,
    h = max(u,0)^2, y = h W2):
        dh = dy_disp @ W2[e]^T
        du = dh * 2*max(u, 0)
        dx_disp = du @ W1[e]^T                (bf16 payload of the inverse dispatch)
        dW2[e] = h^T @ dy_disp,  dW1[e] = x_disp^T @ du
    Experts with no rows get dW = 0 exactly.  Returns (dx_disp, dW1, dW2, du).
    """
    x_disp = np.asarray(x_disp, np.float64)
    u = np.asarray(u, np.float64)
    h = np.asarray(h, np.float64)
    dy_disp = np.asarray(dy_disp, np.float64)
    offsets = np.asarray(offsets, np.int64)
    R, D = x_disp.shape
    E = len(offsets) - 1
    w1_0 = _expert(W1, 0)
    F = w1_0.shape[1]
    dx_disp = np.zeros((R, D))
    du = np.zeros((R, F))
    dW1 = np.zeros((E, D, F))
    dW2 = np.zeros((E, F, D))
    for e in range(E):
        a, b = int(offsets[e]), int(offsets[e + 1])
        if a == b:
            continue
        w1 = _expert(W1, e)
        w2 = _expert(W2, e)
        dh = dy_disp[a:b] @ w2.T
        du[a:b] = dh * (2.0 * np.maximum(u[a:b], 0.0))
        dx_disp[a:b] = du[a:b] @ w1.T
        dW2[e] = h[a:b].T @ dy_disp[a:b]
        dW1[e] = x_disp[a:b].T @ du[a:b]
    if round_payload:
        dx_disp = round_bf16(dx_disp)
    return dx_disp, dW1, dW2, du


def dispatch_bwd(dx_disp, inv_perm, S: int, K: int) -> np.ndarray:
    """Transpose of the dispatch copy (the last inverse route of the backward
    pass): dx[t] = sum_{k<K} dx_disp[inv_perm[t*K+k]], ascending k."""
    dx_disp = np.asarray(dx_disp, np.float64)
    inv = np.asarray(inv_perm, np.int64).reshape(S, K)
    dx = np.zeros((S, dx_disp.shape[1]))
    for k in range(K):
        dx = dx + dx_disp[inv[:, k]]
    return dx


# ---------------------------------------------------------------------------
# Backward through the router and the latent projections
# ---------------------------------------------------------------------------

def router_bwd(x_r, Wr, topk_idx, topk_prob, dp):
    """Gradient of the routed probabilities with respect to the router
    (the learned router of Section 5.2), with the expert selection held
    fixed: top-K is piecewise constant in the scores, so no gradient flows
    through which experts are picked.

    The routed probability p_k is the softmax of the K selected scores (the
    full-E denominator cancels in routing_probs' renormalisation), so per
    token, with dp the gradient of the routed probabilities,
        ds[T_k] = p_k * (dp_k - sum_{j<K} p_j dp_j),    ds = 0 elsewhere,
    and through logits = x_r @ Wr + bias:
        dWr = x_r^T ds,   dbias = sum_t ds[t],   dx_r = ds @ Wr^T.
    Returns (ds [S,E], dWr [D,E], dbias [E], dx_r [S,D]) as float64.
    """
    x_r = np.asarray(x_r, np.float64)
    Wr = np.asarray(Wr, np.float64)
    idx = np.asarray(topk_idx, np.int64)
    p = np.asarray(topk_prob, np.float64)
    dp = np.asarray(dp, np.float64)
    S, K = idx.shape
    E = Wr.shape[1]
    ds = np.zeros((S, E))
    mean = np.sum(p * dp, axis=1)
    for t in range(S):
        for k in range(K):
            ds[t, idx[t, k]] = p[t, k] * (dp[t, k] - mean[t])
    return ds, x_r.T @ ds, ds.sum(axis=0), ds @ Wr.T


def latent_bwd(x_in, W, dout):
    """Gradients of a latent projection out = x_in @ W (latent_down with
    x_in = x, W = Wdown; latent_up with x_in = y_lat, W = Wup):
        dx_in = dout @ W^T,   dW = x_in^T @ dout      (float64)."""
    x_in = np.asarray(x_in, np.float64)
    W = np.asarray(W, np.float64)
    dout = np.asarray(dout, np.float64)
    return dout @ W.T, x_in.T @ dout


def layer_bwd(fwd: dict, x, Wr, W1, W2, K: int, dy, Wdown=None, Wup=None,
              round_payload: bool = True, score: str = "softmax", Ws1=None, Ws2=None,
              seq_len: Optional[int] = None, aux_coeff: float = 0.0) -> dict:
    """Backward of layer_fwd for the loss gradient dy = dL/dy, from the
    intermediates ``fwd`` that layer_fwd returned, in reverse order:
    [latent up] -> combine^T -> experts -> dispatch^T, plus the router path
    (router_bwd on the combine's probability gradient) -> [latent down].
    The input's gradient is the sum of the dispatch^T and router paths.
    ``round_payload`` rounds the gradients that travel the inverse routes
    (dy_disp, dx_disp) to bf16, as the forward payloads are.
    With the production variant (same arguments as layer_fwd) the loss is
    <dy, y> + aux_loss: the router path differentiates the sigmoid weights
    (and the balance loss), and the shared expert adds its input gradient.
    Returns dx, dWr, dbias, dW1, dW2 (and dWdown, dWup, dx_lat, dy_lat for a
    latent layer; dWs1, dWs2 with a shared expert), plus dp and ds (the
    gradient of the logits), as float64.
    """
    x = np.asarray(x, np.float64)
    S = x.shape[0]
    out = {}
    g = np.asarray(dy, np.float64)
    if Ws1 is not None:
        dx_shared, out["dWs1"], out["dWs2"] = shared_expert_bwd(x, fwd["u_s"], fwd["h_s"], g, Ws1, Ws2)
    if Wup is not None:
        g, out["dWup"] = latent_bwd(fwd["y_lat"], Wup, g)
        out["dy_lat"] = g
    dy_disp, dp = combine_bwd(g, fwd["y_disp"], fwd["p_disp"], fwd["inv_perm"], K, round_payload)
    dx_disp, dW1, dW2, _ = expert_ffn_bwd(fwd["x_disp"], fwd["u"], fwd["h"], dy_disp, fwd["offsets"],
                                          W1, W2, round_payload)
    x_r = fwd["x_lat"] if Wdown is not None else x
    if score == "sigmoid":
        ds = sigmoid_gate_bwd(fwd["logits"], fwd["topk_idx"], dp)
        if aux_coeff:
            ds = ds + seq_aux_loss_bwd(fwd["logits"], fwd["topk_idx"], seq_len, aux_coeff)
        dWr, dbias, dx_router = router_linear_bwd(x_r, Wr, ds)
    else:
        ds, dWr, dbias, dx_router = router_bwd(x_r, Wr, fwd["topk_idx"], fwd["topk_prob"], dp)
    dx_r = dispatch_bwd(dx_disp, fwd["inv_perm"], S, K) + dx_router
    if Wdown is not None:
        out["dx_lat"] = dx_r
        dx_r, out["dWdown"] = latent_bwd(x, Wdown, dx_r)
    if Ws1 is not None:
        dx_r = dx_r + dx_shared
    out.update(dx=dx_r, dWr=dWr, dbias=dbias, dW1=dW1, dW2=dW2, dp=dp, ds=ds,
               dy_disp=dy_disp, dx_disp=dx_disp)
    return out


# ---------------------------------------------------------------------------
# The paper's production router (Section 5.2): sigmoid scores with a
# selection-only expert bias, sequence-level balance loss, shared expert
# ---------------------------------------------------------------------------
#
# The paper names these parts but does not write them out.  They are read as
# the published forms they come from (sigmoid gating with a bias that only
# steers selection and a complementary per-sequence balance loss, as in
# DeepSeek-V3, arXiv:2412.19437, Section 2.1):
#   s[t, e]   = sigmoid(logit[t, e])
#   T_t       = top-K experts of s[t, e] + b[e]   (b: selection bias only)
#   g[t, k]   = s[t, T_k] / sum_{j<K} s[t, T_j]   (the routed weight, b_p)
#   loss      = coeff * mean over sequences of sum_e f_e * P_e, per sequence
#               f_e = E / (K * T) * #{tokens of the sequence routed to e},
#               P_e = (1 / T) * sum_t s[t, e] / sum_e' s[t, e'].
# The shared expert is one ungated squared-ReLU MLP on every token, its
# output added to the combined routed output.

def sigmoid_scores(logits) -> np.ndarray:
    """s = 1 / (1 + exp(-logit)) in float64 from the fp32 logits (-inf -> 0)."""
    z = np.asarray(logits, dtype=np.float32).astype(np.float64)
    if np.isnan(z).any():
        raise ValueError("sigmoid routing is undefined for NaN logits")
    with np.errstate(over="ignore"):
        return 1.0 / (1.0 + np.exp(-z))


def sigmoid_topk_select(logits, K: int, sel_bias=None) -> np.ndarray:
    """Top-K experts per token by the selection score s + b (float64), best
    first; equal selection scores go to the lower expert index.  The bias
    steers which experts are picked and nothing else."""
    s = sigmoid_scores(logits)
    S, E = s.shape
    if not 1 <= K <= E:
        raise ValueError("need 1 <= K <= E")
    key = s if sel_bias is None else s + np.asarray(sel_bias, np.float64)[None, :]
    idx = np.empty((S, K), dtype=np.int32)
    experts = np.arange(E)
    for t in range(S):
        order = np.lexsort((experts, -key[t]))   # score descending, then index ascending
        idx[t] = order[:K]
    return idx


def sigmoid_gates(logits, idx) -> np.ndarray:
    """Routed weights g[t, k] = s[t, T_k] / sum_j s[t, T_j], as fp32 (b_p).
    The selection bias does not enter.  A row whose selected scores are all
    zero (every selected logit -inf) has no defined weights."""
    s = sigmoid_scores(logits)
    sel = np.take_along_axis(s, np.asarray(idx, np.int64), axis=1)
    tot = sel.sum(axis=1, keepdims=True)
    if np.any(tot <= 0.0):
        raise ValueError("every token needs a selected expert with a non-zero score")
    return (sel / tot).astype(np.float32)


def sigmoid_route(logits, K: int, sel_bias=None):
    """sigmoid_topk_select then sigmoid_gates: (idx int32 [S,K], g fp32 [S,K])."""
    idx = sigmoid_topk_select(logits, K, sel_bias)
    return idx, sigmoid_gates(logits, idx)


def _sequences(S: int, seq_len: int) -> int:
    if seq_len <= 0 or S % seq_len:
        raise ValueError("the batch must hold whole sequences (S % seq_len == 0)")
    return S // seq_len


def seq_aux_loss(logits, topk_idx, seq_len: int, coeff: float) -> float:
    """Sequence-level balance loss (Section 5.2, coefficient 1e-4 there):
    per sequence of seq_len tokens, sum_e f_e * P_e with f_e the expert's
    share of the sequence's routed slots scaled by E / K (1 when balanced)
    and P_e its mean normalised sigmoid score; averaged over the sequences
    of the batch and scaled by coeff.  The selection is the routed one."""
    s = sigmoid_scores(logits)
    idx = np.asarray(topk_idx, np.int64)
    S, E = s.shape
    K = idx.shape[1]
    B = _sequences(S, seq_len)
    sn = s / s.sum(axis=1, keepdims=True)
    total = 0.0
    for b in range(B):
        rows = slice(b * seq_len, (b + 1) * seq_len)
        f = np.bincount(idx[rows].ravel(), minlength=E) * (E / (K * seq_len))
        P = sn[rows].sum(axis=0) / seq_len
        total += float(np.sum(f * P))
    return coeff * total / B


def seq_aux_loss_bwd(logits, topk_idx, seq_len: int, coeff: float) -> np.ndarray:
    """d(seq_aux_loss)/d(logits) [S,E] with the selection (f) held fixed.
    Through sn = s / sum(s) and s = sigmoid(logit), per token with
    a_e = coeff * f_e / (B * T) of its sequence:
        d sn_e      = a_e
        d s_e       = (a_e - sum_e' a_e' sn_e') / sum_e' s_e'
        d logit_e   = d s_e * s_e * (1 - s_e)."""
    s = sigmoid_scores(logits)
    idx = np.asarray(topk_idx, np.int64)
    S, E = s.shape
    K = idx.shape[1]
    B = _sequences(S, seq_len)
    tot = s.sum(axis=1, keepdims=True)
    sn = s / tot
    a = np.zeros((S, E))
    for b in range(B):
        rows = slice(b * seq_len, (b + 1) * seq_len)
        f = np.bincount(idx[rows].ravel(), minlength=E) * (E / (K * seq_len))
        a[rows] = coeff * f / (B * seq_len)
    ds = (a - np.sum(a * sn, axis=1, keepdims=True)) / tot
    return ds * s * (1.0 - s)


def sigmoid_gate_bwd(logits, topk_idx, dg) -> np.ndarray:
    """d(loss)/d(logits) [S,E] from dg = d(loss)/d(g) [S,K], selection held
    fixed: with sel_k = s[T_k] and Z = sum_j sel_j,
        d sel_k = (dg_k - sum_j dg_j g_j) / Z,   d logit = d s * s (1 - s)
    on the selected experts, 0 elsewhere."""
    s = sigmoid_scores(logits)
    idx = np.asarray(topk_idx, np.int64)
    dg = np.asarray(dg, np.float64)
    S, E = s.shape
    K = idx.shape[1]
    sel = np.take_along_axis(s, idx, axis=1)
    Z = sel.sum(axis=1, keepdims=True)
    g = sel / Z
    dsel = (dg - np.sum(dg * g, axis=1, keepdims=True)) / Z
    out = np.zeros((S, E))
    for t in range(S):
        for k in range(K):
            e = idx[t, k]
            out[t, e] = dsel[t, k] * s[t, e] * (1.0 - s[t, e])
    return out


def router_linear_bwd(x_r, Wr, dlogits):
    """Through logits = x_r @ Wr + bias: (dWr = x_r^T dl, dbias = sum_t dl,
    dx_r = dl @ Wr^T), float64."""
    x_r = np.asarray(x_r, np.float64)
    Wr = np.asarray(Wr, np.float64)
    dl = np.asarray(dlogits, np.float64)
    return x_r.T @ dl, dl.sum(axis=0), dl @ Wr.T


def expert_bias_update(sel_bias, counts, rate: float) -> np.ndarray:
    """Load-driven update of the selection bias (the bias is not trained by
    gradient): b_e += rate * sign(mean_e' counts - counts_e), i.e. an
    overloaded expert is made less attractive, an underloaded one more."""
    c = np.asarray(counts, np.float64)
    return np.asarray(sel_bias, np.float64) + rate * np.sign(c.mean() - c)


def shared_expert(x, Ws1, Ws2):
    """The ungated shared expert on every token (Section 5.2):
    u = x @ Ws1, h = max(u, 0)**2, y_s = h @ Ws2.  Returns (u, h, y_s)."""
    x = np.asarray(x, np.float64)
    u = x @ np.asarray(Ws1, np.float64)
    h = np.maximum(u, 0.0) ** 2
    return u, h, h @ np.asarray(Ws2, np.float64)


def shared_expert_bwd(x, u, h, dy, Ws1, Ws2):
    """Gradients of shared_expert: dh = dy Ws2^T, du = dh * 2 max(u, 0),
    dx = du Ws1^T, dWs1 = x^T du, dWs2 = h^T dy.  Returns (dx, dWs1, dWs2)."""
    x = np.asarray(x, np.float64)
    dy = np.asarray(dy, np.float64)
    Ws1 = np.asarray(Ws1, np.float64)
    Ws2 = np.asarray(Ws2, np.float64)
    du = (dy @ Ws2.T) * (2.0 * np.maximum(np.asarray(u, np.float64), 0.0))
    return du @ Ws1.T, x.T @ du, np.asarray(h, np.float64).T @ dy


# ---------------------------------------------------------------------------
# Lower-precision dispatch payload (Section 1, the precision lever on b_x)
# ---------------------------------------------------------------------------
#
# The payload format is OCP Microscaling (MX v1.0) with FP8 E4M3 elements:
# every block of 32 consecutive elements of a row shares one power-of-two
# scale X = 2^s stored as an E8M0 byte (s + 127), and each element is the
# E4M3 value nearest to x / X.  E4M3 (OCP 8-bit floating point): 1 sign,
# 4 exponent (bias 7) and 3 mantissa bits, no infinities, S.1111.111 = NaN,
# largest finite 448, smallest normal 2^-6, subnormals m * 2^-9.
# The shared exponent is floor(log2(max |x|)) - 8 (8 = the exponent of
# E4M3's largest power of two), so x / X of the block maximum lies in
# [256, 512); element values beyond 448 saturate to +-448.  Readings where
# the specification leaves a choice: an all-zero block (or one whose maximum
# is below 2^-119) takes the smallest scale 2^-127; NaN and infinite inputs
# are not defined here.

MX_BLOCK = 32
E4M3_MAX = 448.0
E4M3_EMAX = 8        # exponent of the largest power of two below E4M3_MAX
E8M0_BIAS = 127


def e4m3_encode(v) -> np.ndarray:
    """Round each value to the nearest E4M3 number (ties to even mantissa),
    saturating finite values beyond 448 to +-448; uint8 codes.  -0.0 keeps
    its sign bit."""
    v = np.asarray(v, np.float64)
    if not np.all(np.isfinite(v)):
        raise ValueError("E4M3 encoding is defined here for finite values only")
    sign = np.signbit(v).astype(np.uint8) << 7
    a = np.minimum(np.abs(v), E4M3_MAX)
    code = np.zeros(a.shape, np.int64)
    sub = a < 2.0 ** -6
    # subnormals (and zero): multiples of 2^-9; 8 * 2^-9 is the smallest normal
    code[sub] = np.rint(a[sub] / 2.0 ** -9).astype(np.int64)
    n = ~sub
    if np.any(n):
        _, ex = np.frexp(a[n])               # a = f * 2^ex, f in [0.5, 1)
        e = ex - 1                           # floor(log2 a), in [-6, 8]
        ulp = np.ldexp(1.0, e - 3)
        r = np.rint(a[n] / ulp) * ulp        # may carry into the next binade
        _, ex2 = np.frexp(r)
        e2 = ex2 - 1
        mant = np.rint((r / np.ldexp(1.0, e2) - 1.0) * 8).astype(np.int64)
        code[n] = ((e2 + 7) << 3) | mant
    return (sign | code.astype(np.uint8)).astype(np.uint8)


def e4m3_decode(codes) -> np.ndarray:
    """Value of each E4M3 code (float64); NaN codes raise."""
    c = np.asarray(codes, np.uint8).astype(np.int64)
    mag = c & 0x7F
    if np.any(mag == 0x7F):
        raise ValueError("NaN code")
    e = mag >> 3
    m = mag & 7
    val = np.where(e == 0, m * 2.0 ** -9, (1.0 + m / 8.0) * np.ldexp(1.0, e - 7))
    return np.where(c & 0x80, -val, val)


def mx_shared_exponent(amax) -> np.ndarray:
    """Block exponent s = floor(log2(amax)) - 8, clamped to E8M0's [-127, 127]
    (amax 0 -> -127)."""
    amax = np.asarray(amax, np.float64)
    _, ex = np.frexp(amax)
    s = np.where(amax > 0, ex - 1 - E4M3_EMAX, -E8M0_BIAS)
    return np.clip(s, -E8M0_BIAS, E8M0_BIAS).astype(np.int64)


def mxfp8_quantize(x):
    """MX-FP8 (E4M3) encoding of the rows of x [R, D], D a multiple of 32:
    (codes uint8 [R, D], scales uint8 [R, D/32] holding s + 127)."""
    x = np.asarray(x, np.float64)
    R, D = x.shape
    if D % MX_BLOCK:
        raise ValueError("row length must be a multiple of the MX block (32)")
    blocks = x.reshape(R, D // MX_BLOCK, MX_BLOCK)
    s = mx_shared_exponent(np.max(np.abs(blocks), axis=2))
    codes = e4m3_encode(blocks / np.ldexp(1.0, s)[:, :, None])
    return codes.reshape(R, D), (s + E8M0_BIAS).astype(np.uint8)


def mxfp8_dequantize(codes, scales) -> np.ndarray:
    """Values of an MX-FP8 payload, float64 [R, D]."""
    codes = np.asarray(codes, np.uint8)
    R, D = codes.shape
    s = np.asarray(scales, np.uint8).astype(np.int64) - E8M0_BIAS
    v = e4m3_decode(codes).reshape(R, D // MX_BLOCK, MX_BLOCK)
    return (v * np.ldexp(1.0, s)[:, :, None]).reshape(R, D)


def dispatch_mxfp8(x, prob, inv_perm, K: int):
    """Dispatch with an MX-FP8 hidden payload: each token row is encoded once
    and its codes and scales are copied to the token's K routed rows (the
    sender encodes, the payload travels); the probability stays fp32 (b_p).
    Returns (codes [S*K, D], scales [S*K, D/32], p_disp [S*K] or None)."""
    codes, scales = mxfp8_quantize(x)
    S = codes.shape[0]
    inv = np.asarray(inv_perm, np.int64).reshape(S, K)
    R = S * K
    cd = np.zeros((R, codes.shape[1]), np.uint8)
    sc = np.zeros((R, scales.shape[1]), np.uint8)
    pd = None if prob is None else np.zeros(R, np.float32)
    for k in range(K):
        cd[inv[:, k]] = codes
        sc[inv[:, k]] = scales
        if prob is not None:
            pd[inv[:, k]] = np.asarray(prob, np.float32)[:, k]
    return cd, sc, pd


def mx_payload_bytes(S: int, K: int, D: int, b_p: int = B_P) -> int:
    """Forward dispatch payload with MX-FP8 hidden elements: per routed row D
    one-byte elements, D/32 one-byte scales and the routed probability
    (Eq. 1 with b_x = 1 + 1/32)."""
    return S * K * (D + D // MX_BLOCK + b_p)


# ---------------------------------------------------------------------------
# Eq. 1: expert-parallel communication volume
# ---------------------------------------------------------------------------

def dispatch_payload_bytes(S: int, K: int, D: int, b_x: int = B_X, b_p: int = B_P) -> int:
    """Forward dispatch payload: every routed row carries its hidden state
    and its routed probability, S*K*(D*b_x + b_p) bytes (Eq. 1)."""
    return S * K * (D * b_x + b_p)


def combine_payload_bytes(S: int, K: int, D: int, b_x: int = B_X) -> int:
    """Forward combine payload: one hidden state per routed row, S*K*D*b_x."""
    return S * K * D * b_x


def ep_volume_per_step(L_E: int, S: int, GBS: int, K: int, D: int,
                       b_x: int = B_X, b_p: int = B_P) -> int:
    """Expert-parallel volume over one training step (Eq. 1): forward
    dispatch + combine and their backward inverses, summed over L_E MoE
    layers and GBS sequences of S tokens: L_E*S*GBS*K*(4*D*b_x + 2*b_p)."""
    per_layer_tokens = S * GBS
    fwd = dispatch_payload_bytes(per_layer_tokens, K, D, b_x, b_p) + \
        combine_payload_bytes(per_layer_tokens, K, D, b_x)
    return L_E * 2 * fwd
