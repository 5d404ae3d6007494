"""GPU parity: grouped expert FFN (MFMA grouped GEMM + fused squared-ReLU)
and the dense latent projection.

Exact-arithmetic inputs (+-1 entries, at most 16 non-zeros per row, so every
product, sum and u^2 is exact) require bit-exact outputs; these pin the MFMA
lane layouts, the in-register transposes, the expert-segment mapping and the
ragged row / k / n tails.  Random inputs are held to the bf16 bar.
"""
import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from paper_2608_28511_amd import layer
from paper_2608_28511_amd.workloads import (WORKLOADS, make_inputs, make_logits, make_segments,
                                            make_sparse_sign_rows)

from gpu_helpers import LazyExperts, assert_bf16_close, np64, npi, takes_tall_tiles

pytestmark = pytest.mark.gpu
DEV = "cuda:0"

# (R, D, F, E, empty experts, skew)
SHAPES = [(1, 8, 8, 1, 0, 0.0), (100, 16, 24, 3, 0, 0.0), (1000, 264, 200, 5, 1, 0.0),
          (777, 136, 392, 9, 2, 1.5), (4096, 256, 512, 8, 0, 0.0), (300, 512, 128, 64, 20, 0.0),
          (2500, 192, 64, 2, 0, 2.0),
          # widths that 384-column tiles cover with less padding (up: F; down: D)
          (1500, 392, 1096, 7, 1, 1.0), (900, 2688, 360, 5, 1, 0.0), (640, 200, 360, 6, 1, 0.5)]


def _sign_weights(E, a, b, seed, density):
    g = torch.Generator().manual_seed(seed)
    v = torch.randint(-1, 2, (E, a, b), generator=g).to(torch.float32)
    keep = torch.rand((E, a, b), generator=g) < density
    return (v * keep).to(torch.bfloat16)


@pytest.mark.parametrize("R,D,F,E,empty,skew", SHAPES)
def test_grouped_ffn_exact(R, D, F, E, empty, skew):
    off = make_segments(R, E, seed=R + E, empty=empty, skew=skew)
    x = make_sparse_sign_rows(R, D, 16, seed=R).to(torch.bfloat16)
    W1 = _sign_weights(E, D, F, seed=D, density=1.0)
    # y = sum_f h_f W2[f, d] is an exact integer in fp32, so both sides round it identically
    W2 = _sign_weights(E, F, D, seed=F, density=min(1.0, 4.0 / F))
    h, u, yd = layer.grouped_ffn(x.to(DEV), off.to(DEV), W1.to(DEV), W2.to(DEV), save_u=True)
    torch.cuda.synchronize()
    u_ref, h_ref, y_ref = O.expert_ffn(np64(x), npi(off), np64(W1), np64(W2))
    assert np.array_equal(np64(u), u_ref)
    assert np.array_equal(np64(h), h_ref)
    assert np.array_equal(np64(yd), y_ref)


@pytest.mark.parametrize("R,D,F,E,empty,skew", SHAPES)
def test_grouped_ffn_random(R, D, F, E, empty, skew):
    g = torch.Generator().manual_seed(R * 3 + D)
    off = make_segments(R, E, seed=R + 2 * E, empty=empty, skew=skew)
    x = torch.randn((R, D), generator=g).to(torch.bfloat16)
    W1 = (torch.randn((E, D, F), generator=g) / np.sqrt(D)).to(torch.bfloat16)
    W2 = (torch.randn((E, F, D), generator=g) / np.sqrt(F)).to(torch.bfloat16)
    h, u, yd = layer.grouped_ffn(x.to(DEV), off.to(DEV), W1.to(DEV), W2.to(DEV), save_u=True)
    u_ref, h_ref, y_ref = O.expert_ffn(np64(x), npi(off), np64(W1), np64(W2), round_payload=False)
    assert_bf16_close(np64(u), u_ref, "u")
    assert_bf16_close(np64(h), h_ref, "h")
    assert_bf16_close(np64(yd), y_ref, "y_disp")


@pytest.mark.parametrize("M,Kd,N", [(1, 8, 8), (300, 264, 136), (4096, 4096, 1024), (1000, 1024, 4096)])
def test_latent_proj(M, Kd, N):
    g = torch.Generator().manual_seed(M + Kd + N)
    A = torch.randn((M, Kd), generator=g).to(torch.bfloat16)
    W = (torch.randn((Kd, N), generator=g) / np.sqrt(Kd)).to(torch.bfloat16)
    C = layer.latent_proj(A.to(DEV), W.to(DEV))
    assert_bf16_close(np64(C), O.latent_down(np64(A), np64(W), round_payload=False), "latent")
    # exact arithmetic: +-1 rows with 16 non-zeros times a +-1/0 weight
    Ae = make_sparse_sign_rows(M, Kd, 16, seed=M).to(torch.bfloat16)
    We = _sign_weights(1, Kd, N, seed=Kd, density=1.0)[0]
    Ce = layer.latent_proj(Ae.to(DEV), We.to(DEV))
    torch.cuda.synchronize()
    assert np.array_equal(np64(Ce), O.latent_down(np64(Ae), np64(We)))


@pytest.mark.parametrize("name", [n for n in WORKLOADS if not n.startswith("tiny")])
def test_grouped_ffn_full_size(name):
    """Full-size experts and routing (the same fp32 logits routed on both
    sides, so the routes are identical): u, h and y_disp of every routed row
    against the oracle."""
    s = WORKLOADS[name]
    inp = make_inputs(s.scaled(H=0), device=DEV)
    x = inp["x"][:, : s.D].contiguous()
    logits = torch.randn((s.S, s.E), device=DEV, generator=torch.Generator(device=DEV).manual_seed(1))
    if inp["bias"] is not None:
        logits = logits + inp["bias"][None, :]
    r = layer.route(logits, s.K)
    x_disp, p_disp = layer.dispatch(x, r["topk_prob"], r["inv_perm"], s.K)
    h, u, yd = layer.grouped_ffn(x_disp, r["offsets"], inp["W1"], inp["W2"], save_u=True)
    torch.cuda.synchronize()
    idx, _ = O.route(logits.cpu().numpy(), s.K)
    _, off, _, inv = O.expert_permutation(idx, s.E)
    assert np.array_equal(npi(r["offsets"]), off) and np.array_equal(npi(r["inv_perm"]), inv)
    xd, _ = O.dispatch(np64(x), None, inv, s.K)
    u_ref, h_ref, y_ref = O.expert_ffn(xd, off, LazyExperts(inp["W1"]), LazyExperts(inp["W2"]),
                                       round_payload=False)
    del xd
    assert_bf16_close(np64(u), u_ref, f"{name} u")
    del u_ref
    assert_bf16_close(np64(h), h_ref, f"{name} h")
    del h_ref
    assert_bf16_close(np64(yd), y_ref, f"{name} y_disp")


def test_grouped_ffn_exact_tall_tiles():
    """Both projections on 256-row tiles (long launch, few large experts with
    ragged last tiles): bit-exact like the 128-row shapes above."""
    R, D, F, E = 24576, 512, 1024, 4
    off = make_segments(R, E, seed=R + E)
    counts = np.diff(npi(off))
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    if not (takes_tall_tiles(counts, F, cus) and takes_tall_tiles(counts, D, cus)):
        pytest.skip(f"this device ({cus} CUs) keeps 128-row tiles for the shape")
    assert all(c % 256 for c in counts)   # every expert ends in a partly filled tall tile
    x = make_sparse_sign_rows(R, D, 16, seed=R).to(torch.bfloat16)
    W1 = _sign_weights(E, D, F, seed=D, density=1.0)
    W2 = _sign_weights(E, F, D, seed=F, density=min(1.0, 4.0 / F))
    h, u, yd = layer.grouped_ffn(x.to(DEV), off.to(DEV), W1.to(DEV), W2.to(DEV), save_u=True)
    torch.cuda.synchronize()
    u_ref, h_ref, y_ref = O.expert_ffn(np64(x), npi(off), np64(W1), np64(W2))
    assert np.array_equal(np64(u), u_ref)
    assert np.array_equal(np64(h), h_ref)
    assert np.array_equal(np64(yd), y_ref)


@pytest.mark.parametrize("R,D,F,E,empty,skew", SHAPES[1:5])
def test_grouped_gemm_single_launches_match_ffn(R, D, F, E, empty, skew):
    """moe_grouped_schedule + two moe_grouped_gemm launches reproduce
    moe_grouped_ffn bit for bit (same kernels, same schedule)."""
    g = torch.Generator().manual_seed(R + 17 * D)
    off = make_segments(R, E, seed=R + 3 * E, empty=empty, skew=skew).to(DEV)
    x = torch.randn((R, D), generator=g).to(torch.bfloat16).to(DEV)
    W1 = (torch.randn((E, D, F), generator=g) / np.sqrt(D)).to(torch.bfloat16).to(DEV)
    W2 = (torch.randn((E, F, D), generator=g) / np.sqrt(F)).to(torch.bfloat16).to(DEV)
    h, u, yd = layer.grouped_ffn(x, off, W1, W2, save_u=True)
    sched = layer.grouped_schedule(off, E, R)
    u2 = torch.empty_like(u)
    h2 = layer.grouped_gemm(x, sched, W1, 1, u_save=u2)
    y2 = layer.grouped_gemm(h2, sched, W2, 0)
    torch.cuda.synchronize()
    counts = np.diff(npi(off))
    ms = npi(sched[: E + 1])
    assert np.array_equal(np.diff(ms), (counts + 127) // 128)
    assert torch.equal(h, h2) and torch.equal(u, u2) and torch.equal(yd, y2)
    # each entry's run: the m-tiles of its expert cut into runs of at most 8 from the expert's first
    t0 = ((E + 1) * 4 + 15) // 16 * 16 // 4      # the table follows mtile_start, 16-byte aligned
    table = npi(sched[t0: t0 + 4 * int(ms[-1])]).reshape(-1, 4)
    for mt, (e, r0, r1, packed) in enumerate(table):
        g0, gs = packed >> 4, packed & 15
        assert (g0 - ms[e]) % 8 == 0 and g0 <= mt < g0 + gs and gs == min(8, ms[e + 1] - g0), (mt, e, g0, gs)


@pytest.mark.parametrize("S,D,F,E,K", [(1, 8, 8, 1, 1), (300, 136, 200, 5, 2), (2048, 256, 512, 64, 6),
                                       (777, 264, 392, 9, 3)])
def test_grouped_gemm_gather_matches_dispatched(S, D, F, E, K):
    """The up projection gathering its rows from x through perm equals the
    dispatch followed by the grouped GEMM on the dispatched rows, bit for bit
    (u saved too), on ragged experts and k / n tails."""
    from paper_2608_28511_amd import _lib as L
    g = torch.Generator().manual_seed(S + D + E)
    x = torch.randn((S, D), generator=g).to(torch.bfloat16).to(DEV)
    W1 = (torch.randn((E, D, F), generator=g) / np.sqrt(D)).to(torch.bfloat16).to(DEV)
    r = layer.route(make_logits("normal", S, E, seed=S + E).to(DEV), K)
    R = S * K
    xd, _ = layer.dispatch(x, None, r["inv_perm"], K)
    sched = layer.grouped_schedule(r["offsets"], E, R)
    u_ref = torch.empty((R, F), dtype=torch.bfloat16, device=DEV)
    h_ref = layer.grouped_gemm(xd, sched, W1, 1, u_save=u_ref)
    h = torch.full((R, F), float("nan"), dtype=torch.bfloat16, device=DEV)
    u = torch.full((R, F), float("nan"), dtype=torch.bfloat16, device=DEV)
    L.moe_grouped_gemm_gather(x, r["perm"], S, K, sched, E, R, D, F, W1, 1, h, u)
    torch.cuda.synchronize()
    assert torch.equal(h, h_ref) and torch.equal(u, u_ref)


def test_schedule_caps_overlapping_segments():
    """Offsets that are not monotone give segments that overlap after
    clamping and ask for more tiles than the table holds (here 8 + 4 > 8 + 3);
    the builder caps the count at the table size, so no reader of the table
    walks past it, and every entry it writes stays inside [0, R)."""
    E, R = 3, 1000
    off = torch.tensor([0, R, R // 2, R], dtype=torch.int32, device=DEV)
    sched = layer.grouped_schedule(off, E, R)
    torch.cuda.synchronize()
    ms = npi(sched[: E + 1])
    max_tiles = -(-R // 128) + min(R, E)
    assert ms[0] == 0 and np.all(np.diff(ms) >= 0) and ms[-1] == max_tiles
    t0 = ((E + 1) * 4 + 15) // 16 * 16 // 4      # the table follows mtile_start, 16-byte aligned
    table = npi(sched[t0: t0 + 4 * max_tiles]).reshape(max_tiles, 4)
    assert np.all((table[:, 0] >= 0) & (table[:, 0] < E))
    assert np.all((table[:, 1] >= 0) & (table[:, 1] < table[:, 2]) & (table[:, 2] <= R))
