"""Shared helpers for the GPU parity tests (comparison metrics, lazy weight
views for the oracle, routing-ambiguity detection).  Holds no arithmetic of
the layer itself."""
from __future__ import annotations

import numpy as np
import torch

# Tolerances of the parity bar (floating-point outputs).
PROB_RTOL = 1e-5          # fp32 routed probabilities, relative
LOGIT_RTOL = 1e-5         # fp32 router logits, relative to max(|ref|, 1)
BF16_MAX_REL = 2e-2       # bf16 outputs: max |d| / max(|ref|, rms(ref))
BF16_MEAN_ABS = 1e-2      # bf16 outputs: mean |d| (outputs have rms ~0.4-1.2)


def np64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu").to(torch.float64).numpy()


def npi(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu").numpy().astype(np.int64)


class LazyExperts:
    """Indexable view of a device weight stack [E, a, b] that the oracle can
    read one expert at a time (float64 on the host, cached)."""

    def __init__(self, W: torch.Tensor, cache: bool = False):
        self.W = W
        self.cache = {} if cache else None

    def __getitem__(self, e):
        e = int(e)
        if self.cache is None:
            return np64(self.W[e])
        if e not in self.cache:
            self.cache[e] = np64(self.W[e])
        return self.cache[e]

    def __len__(self):
        return self.W.shape[0]


def close_metrics(got: np.ndarray, ref: np.ndarray):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    d = np.abs(got - ref)
    rms = float(np.sqrt(np.mean(ref ** 2))) if ref.size else 0.0
    floor = np.maximum(np.abs(ref), max(rms, 1e-30))
    max_rel = float(np.max(d / floor)) if ref.size else 0.0
    mean_abs = float(np.mean(d)) if ref.size else 0.0
    return max_rel, mean_abs, rms


def assert_bf16_close(got, ref, what="", max_rel=BF16_MAX_REL, mean_abs=BF16_MEAN_ABS,
                      mean_rel_to_rms=False):
    mr, ma, rms = close_metrics(got, ref)
    lim = mean_abs * (rms if mean_rel_to_rms else 1.0)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    assert mr <= max_rel and ma <= lim, (
        f"{what}: max_rel {mr:.3e} (<= {max_rel}), mean_abs {ma:.3e} (<= {lim:.3e}), rms {rms:.3e}")
    return mr, ma


def assert_probs_close(got, ref, what="probs"):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    bad = np.abs(got - ref) > PROB_RTOL * np.abs(ref)
    assert not bad.any(), f"{what}: {bad.sum()} entries off, e.g. got {got[bad][:4]} ref {ref[bad][:4]}"


def ambiguous_tokens(logits_ref: np.ndarray, K: int, tau: np.ndarray) -> np.ndarray:
    """Tokens whose top-(K+1) scores hold an adjacent gap <= 2*tau, i.e. whose
    selection or slot order could legitimately flip under a perturbation of
    the scores by tau.  Returns a boolean mask [S]."""
    s = np.asarray(logits_ref, np.float64)
    E = s.shape[1]
    m = min(K + 1, E)
    top = -np.sort(-np.where(np.isnan(s), -np.inf, s), axis=1)[:, :m]
    with np.errstate(invalid="ignore"):
        gaps = np.diff(top, axis=1)  # <= 0
    tau = np.broadcast_to(np.asarray(tau, np.float64).reshape(-1, 1), (s.shape[0], 1))
    amb = np.any(np.abs(gaps) <= 2 * tau, axis=1) if m > 1 else np.zeros(s.shape[0], bool)
    return amb


def check_permutation_props(idx, counts, offsets, perm, inv_perm, E, K):
    """Properties that determine counts/offsets/perm/inv_perm uniquely from idx."""
    idx = np.asarray(idx, np.int64)
    S = idx.shape[0]
    R = S * K
    assert np.array_equal(counts, np.bincount(idx.ravel(), minlength=E))
    assert offsets[0] == 0 and offsets[-1] == R
    assert np.array_equal(np.diff(offsets), counts)
    assert np.array_equal(np.sort(perm), np.arange(R))
    assert np.array_equal(inv_perm[perm], np.arange(R))
    flat = idx.ravel()
    e_of_pos = flat[perm]
    assert np.all(np.diff(e_of_pos) >= 0)
    tok = perm // K
    same = np.diff(e_of_pos) == 0
    assert np.all(np.diff(tok)[same] > 0)


def takes_tall_tiles(counts, N, cus):
    """The rows kernel's tile-height rule, restated: the busiest XCD's rounds
    of 128-row and of 256-row tiles; tall tiles when 2 * rounds_tall * 0.91 <
    rounds_small.  The grid is one workgroup per CU (a multiple of 8), capped
    by the static bound on the number of output tiles."""
    def cdiv(a, b):
        return -(-a // b)
    R, E = int(sum(counts)), len(counts)
    m_small = int(sum(cdiv(int(c), 128) for c in counts))
    m_tall = int(sum(cdiv(int(c), 256) for c in counts))
    nt = cdiv(N, 256)
    bound = (cdiv(R, 128) + min(R, E)) * nt          # static bound on the output tiles
    G = min(cus // 8 * 8, cdiv(bound, 8) * 8)
    r_small = cdiv(cdiv(m_small, 8) * nt, G // 8)
    r_tall = cdiv(cdiv(m_tall, 8) * nt, G // 8)
    return 2 * r_tall * 91 < 100 * r_small


def tie_candidates(scores: np.ndarray, K: int, tau: float, cap: int = 5040):
    """Every slot-ordered top-K selection that reordering experts whose sorted
    scores lie within 2*tau of their neighbours can give, from the oracle's
    scores of one token: the experts sorted by (score desc, index asc) are cut
    into runs of adjacent gaps <= 2*tau; each run covering the first K
    positions is permuted freely and the first K experts kept.  A superset of
    the selections a perturbation of every score by tau could produce (each
    is then held to the pairwise 2*tau rule as well).  None if there are more
    than ``cap`` orderings."""
    import itertools
    import math
    s = np.where(np.isnan(scores), -np.inf, np.asarray(scores, np.float64))
    order = np.lexsort((np.arange(s.size), -s))
    runs, cur = [], [int(order[0])]
    for a, b in zip(order[:-1], order[1:]):
        close = s[a] == s[b] or abs(s[a] - s[b]) <= 2 * tau
        if close:
            cur.append(int(b))
        else:
            runs.append(cur)
            cur = [int(b)]
    runs.append(cur)
    need, n = [], 0
    for r in runs:
        need.append(r)
        n += len(r)
        if n >= K:
            break
    if math.prod(math.factorial(len(r)) for r in need) > cap:
        return None
    out = set()
    for combo in itertools.product(*[itertools.permutations(r) for r in need]):
        out.add(tuple(e for r in combo for e in r)[:K])
    return out


def check_tie_choice(scores: np.ndarray, chosen, K: int, tau: float):
    """The GPU's slot-ordered choice for a near-tie token is one of the
    oracle's candidate selections and obeys the 2*tau rule pairwise: every
    slot's score is at least every later slot's minus 2*tau, and every chosen
    score at least every unchosen one's minus 2*tau."""
    chosen = [int(e) for e in chosen]
    assert len(set(chosen)) == K
    s = np.asarray(scores, np.float64)
    cands = tie_candidates(s, K, tau)
    if cands is not None:
        assert tuple(chosen) in cands, (chosen, sorted(cands)[:4])
    cs = s[chosen]
    for i in range(K):
        for j in range(i + 1, K):
            assert cs[i] >= cs[j] - 2 * tau, ("slot order", chosen)
    rest = np.delete(s, chosen)
    if rest.size:
        assert cs.min() >= rest.max() - 2 * tau, ("selection", chosen)


def guarded(shape, dtype, device, guard: int = 2):
    """A NaN-filled buffer with `guard` extra rows (leading-dimension slices)
    before and after; returns (buffer, interior view).  A kernel that writes
    every element of the interior and nothing outside it leaves the guards
    all NaN and the interior free of NaN."""
    shape = tuple(shape)
    buf = torch.full((shape[0] + 2 * guard,) + shape[1:], float("nan"), dtype=dtype, device=device)
    return buf, buf[guard:guard + shape[0]]


def check_guarded(buf: torch.Tensor, guard: int, what: str):
    n = buf.shape[0] - 2 * guard
    assert bool(torch.isnan(buf[:guard]).all()) and bool(torch.isnan(buf[guard + n:]).all()), \
        f"{what}: a guard row was written"
    inner = buf[guard:guard + n]
    bad = int(torch.isnan(inner).sum())
    assert bad == 0, f"{what}: {bad} elements left unwritten (still NaN)"
