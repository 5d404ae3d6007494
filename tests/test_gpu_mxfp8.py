"""GPU parity of the MX-FP8 dispatch payload (Section 1's precision lever on
b_x): codes, block scales and the decoded rows are integer/byte work and
must match the oracle bit for bit; the up projection that decodes the
payload in its operand path must equal decode-then-GEMM bit for bit (and
the oracle to the bf16 bar); the layer with the MX payload is held to the
bf16 output bar against the oracle's chain on the same payload."""
import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from paper_2608_28511_amd import layer
from paper_2608_28511_amd.workloads import PRODUCTION, WORKLOADS, make_inputs, make_segments

from gpu_helpers import LazyExperts, assert_bf16_close, np64, npi, takes_tall_tiles

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _rows(kind, S, D, seed):
    g = torch.Generator().manual_seed(seed)
    x = torch.randn((S, D), generator=g)
    if kind == "wide":        # per-row scales over ~2^-40 .. 2^40
        x = x * torch.exp2(torch.randint(-40, 40, (S, 1), generator=g).float())
    elif kind == "tiny":      # bf16 subnormals and blocks near the bottom of the range
        x = x * 2.0 ** -128
    elif kind == "edge":      # zero blocks, -0, block maxima just below a power of two (saturation)
        x[:, :32] = 0.0
        x[::2, 32:64] = -0.0
        x[:, 64] = 1.99 * torch.sign(x[:, 64] + 0.5)
        x[1::3, 96:128] = 0.0
        x[1::3, 97] = 2.0 ** 100
    return x.to(torch.bfloat16)


def _random_inv(S, K, seed):
    g = torch.Generator().manual_seed(seed)
    return torch.randperm(S * K, generator=g).to(torch.int32)


# the edge rows place their special blocks in the first four blocks of a row
_MX_CASES = [(kind, S, D, K) for kind in ("normal", "wide", "tiny", "edge")
             for (S, D, K) in [(1, 32, 1), (37, 96, 3), (256, 2048, 6), (100, 2688, 7), (513, 128, 8)]
             if not (kind == "edge" and D < 128)]


@pytest.mark.parametrize("kind,S,D,K", _MX_CASES)
def test_dispatch_mxfp8_bit_exact(kind, S, D, K):
    x = _rows(kind, S, D, S + D + K)
    inv = _random_inv(S, K, S * K)
    g = torch.Generator().manual_seed(S)
    p = torch.rand((S, K), generator=g)
    xq, xs, pd = layer.dispatch_mxfp8(x.to(DEV), p.to(DEV), inv.to(DEV), K)
    torch.cuda.synchronize()
    cd, sc, pref = O.dispatch_mxfp8(np64(x), p.numpy(), inv.numpy(), K)
    assert np.array_equal(xq.cpu().numpy(), cd), "codes"
    assert np.array_equal(xs.cpu().numpy(), sc), "scales"
    assert np.array_equal(pd.cpu().numpy(), pref), "p_disp"
    # receive side: the decoded bf16 rows are exact
    out = layer.mxfp8_dequant(xq, xs)
    torch.cuda.synchronize()
    want = O.round_bf16(O.mxfp8_dequantize(cd, sc))
    got = np64(out)
    assert np.array_equal(got, want) and np.array_equal(np.signbit(got), np.signbit(want)), "dequant"


def test_dequant_every_code_and_scale():
    # all 254 finite codes at every scale from 2^-127 to 2^119 (the bottom of
    # the range rounds below bf16's smallest normal)
    codes = np.array([c for c in range(256) if c & 0x7F != 0x7F], np.uint8)
    s = np.arange(-127, 120)
    R = len(s)
    cq = np.zeros((R, 256), np.uint8)
    cq[:, :254] = codes[None, :]
    sc = np.repeat((s + 127).astype(np.uint8)[:, None], 8, axis=1)
    out = layer.mxfp8_dequant(torch.as_tensor(cq).to(DEV), torch.as_tensor(sc).to(DEV))
    torch.cuda.synchronize()
    want = O.round_bf16(O.mxfp8_dequantize(cq, sc))
    got = np64(out)
    assert np.array_equal(got, want) and np.array_equal(np.signbit(got), np.signbit(want))


def test_mx_payload_bytes():
    from paper_2608_28511_amd import _lib as L
    for S, K, D in [(8192, 6, 2048), (16384, 7, 2688), (1, 1, 32)]:
        assert L.moe_mx_payload_bytes(S, K, D) == O.mx_payload_bytes(S, K, D)
    assert L.moe_mx_payload_bytes(8, 2, 48) == 0


@pytest.mark.parametrize("name,n_samples", [("tiny_s512_d256_e8_k2", None), ("base_s8192_d2048_e64_k6", 32)])
def test_layer_fwd_mxfp8(name, n_samples):
    s = WORKLOADS[name]
    inp = make_inputs(s, device=DEV)
    lf = layer.LayerFwd(s.S, s.D, s.E, s.K, s.F, export=True, payload="mxfp8")
    out = lf(inp["x"], inp["Wr"], inp["W1"], inp["W2"], bias=inp["bias"])
    torch.cuda.synchronize()
    x = np64(inp["x"])
    # the payload: each routed row holds its token's encoding, bit for bit
    c, sc = O.mxfp8_quantize(x)
    inv = npi(out["inv_perm"]).reshape(s.S, s.K)
    xq, xs = out["x_q"].cpu().numpy(), out["x_scale"].cpu().numpy()
    for k in range(s.K):
        assert np.array_equal(xq[inv[:, k]], c) and np.array_equal(xs[inv[:, k]], sc)
    assert np.array_equal(np64(out["x_disp"])[inv[:, 0]], O.round_bf16(O.mxfp8_dequantize(c, sc)))
    # outputs against the oracle's chain on the same MX payload (routing is
    # unchanged by the payload: the router reads x itself)
    rng = np.random.default_rng(s.seed)
    tok = np.arange(s.S) if n_samples is None else np.sort(rng.choice(s.S, n_samples, replace=False))
    ref = O.layer_fwd(x[tok], np64(inp["Wr"]), LazyExperts(inp["W1"]), LazyExperts(inp["W2"]), s.K,
                      bias=None if inp["bias"] is None else np64(inp["bias"]), payload="mxfp8",
                      round_payload=False)
    idx = npi(out["topk_idx"])[tok]
    ok = np.all(idx == ref["topk_idx"], axis=1)
    assert ok.mean() > 0.99
    assert_bf16_close(np64(out["y"][torch.as_tensor(tok[ok], device=DEV)]), ref["y"][ok], f"{name} y (mxfp8)")


# (rows kind, S, K, D = Kd, E, empty experts, N): Kd / 32 odd leaves half a
# 64-wide stage at the end of the contraction, and R * Kd / 32 not a multiple
# of 4 puts the last scale bytes in the allocation's padded word; the last
# case is long enough for the 256-row tiles.
_GEMM_MX_CASES = [
    ("normal", 1, 1, 32, 1, 0, 8),         # one row, one 32-element block, N = 8
    ("wide", 19, 2, 32, 3, 1, 24),         # Kd = 32: the only stage is half a stage
    ("tiny", 40, 4, 64, 7, 2, 264),        # Kd = 64: exactly one stage
    ("normal", 37, 3, 96, 5, 1, 72),
    ("normal", 256, 6, 2048, 8, 0, 1024),
    ("wide", 100, 7, 2688, 16, 3, 264),
    ("tiny", 513, 8, 128, 64, 20, 1032),
    ("edge", 201, 3, 160, 3, 0, 256),
    ("normal", 4096, 6, 512, 4, 0, 1024),
]


def _bits(t):
    return t.view(torch.int16)


@pytest.mark.parametrize("kind,S,K,D,E,empty,N", _GEMM_MX_CASES)
def test_grouped_gemm_mxfp8_equals_decode_then_gemm(kind, S, K, D, E, empty, N):
    seed = S + 7 * D + N
    R = S * K
    x = _rows(kind, S, D, seed)
    inv = _random_inv(S, K, seed + 1)
    xq, xs, _ = layer.dispatch_mxfp8(x.to(DEV), None, inv.to(DEV), K)
    off = make_segments(R, E, seed=seed + 2, empty=empty)
    sched = layer.grouped_schedule(off.to(DEV), E, R)
    g = torch.Generator().manual_seed(seed + 3)
    W = (torch.randn((E, D, N), generator=g) * D ** -0.5).to(torch.bfloat16).to(DEV)
    xd = layer.mxfp8_dequant(xq, xs)
    if (S, D) == (4096, 512):
        cus = torch.cuda.get_device_properties(0).multi_processor_count
        assert takes_tall_tiles(np.diff(npi(off)), N, cus), "the case must take the 256-row tiles"
    for epi in (1, 0):
        u_f = torch.empty((R, N), dtype=torch.bfloat16, device=DEV) if epi else None
        u_r = torch.empty((R, N), dtype=torch.bfloat16, device=DEV) if epi else None
        c_f = layer.grouped_gemm_mxfp8(xq, xs, sched, W, epi, u_save=u_f)
        c_r = layer.grouped_gemm(xd, sched, W, epi, u_save=u_r)
        torch.cuda.synchronize()
        assert torch.equal(_bits(c_f), _bits(c_r)), f"epilogue {epi}: C differs from decode-then-GEMM"
        if epi:
            assert torch.equal(_bits(u_f), _bits(u_r)), "u_save differs from decode-then-GEMM"
    if kind == "normal" and R * D <= 1 << 20:
        # and the oracle's chain: its own encoding, decode and expert FFN
        cd, sc, _ = O.dispatch_mxfp8(np64(x), None, inv.numpy(), K)
        xd_ref = O.round_bf16(O.mxfp8_dequantize(cd, sc))
        zero_w2 = [np.zeros((N, 8))] * E
        u_ref, _, _ = O.expert_ffn(xd_ref, npi(off), LazyExperts(W), zero_w2, round_payload=False)
        assert_bf16_close(np64(c_f), u_ref, f"{kind} u")   # epilogue 0: the plain product


def test_grouped_gemm_mxfp8_oracle_h():
    """The fused up projection's squared-ReLU output against the oracle."""
    S, K, D, E, N = 64, 4, 224, 6, 320
    R = S * K
    x = _rows("normal", S, D, 11)
    inv = _random_inv(S, K, 12)
    xq, xs, _ = layer.dispatch_mxfp8(x.to(DEV), None, inv.to(DEV), K)
    off = make_segments(R, E, seed=13, empty=1)
    sched = layer.grouped_schedule(off.to(DEV), E, R)
    W = (torch.randn((E, D, N), generator=torch.Generator().manual_seed(14)) * D ** -0.5).to(torch.bfloat16)
    W = W.to(DEV)
    u = torch.empty((R, N), dtype=torch.bfloat16, device=DEV)
    h = layer.grouped_gemm_mxfp8(xq, xs, sched, W, 1, u_save=u)
    torch.cuda.synchronize()
    cd, sc, _ = O.dispatch_mxfp8(np64(x), None, inv.numpy(), K)
    xd_ref = O.round_bf16(O.mxfp8_dequantize(cd, sc))
    u_ref, h_ref, _ = O.expert_ffn(xd_ref, npi(off), LazyExperts(W), [np.zeros((N, 8))] * E, round_payload=False)
    assert_bf16_close(np64(u), u_ref, "u")
    assert_bf16_close(np64(h), h_ref, "h")


def test_grouped_gemm_mxfp8_rejects_bad_shapes():
    from paper_2608_28511_amd import _lib as L
    R, D, E, N = 64, 48, 2, 64   # D not a multiple of 32
    xq = torch.zeros((R, D), dtype=torch.uint8, device=DEV)
    xs = layer.mx_scales(R, 64, DEV)
    off = make_segments(R, E, seed=1)
    sched = layer.grouped_schedule(off.to(DEV), E, R)
    W = torch.zeros((E, D, N), dtype=torch.bfloat16, device=DEV)
    C = torch.empty((R, N), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(RuntimeError):
        L.moe_grouped_gemm_mxfp8(xq, xs, sched, E, R, D, N, W, 0, C, None)
    with pytest.raises(ValueError):   # scale allocation not padded to whole words
        L.moe_grouped_gemm_mxfp8(xq[:, :32].contiguous(), torch.zeros(R * 1 - 1, dtype=torch.uint8, device=DEV),
                                 sched, E, R, 32, N, W[:, :32].contiguous(), 0, C, None)


def test_layer_fwd_mxfp8_without_decoded_export():
    """The MX layer that decodes only inside the up projection (x_disp not
    exported, no decode pass) gives the same outputs as with the export."""
    s = WORKLOADS["tiny_s512_d256_e8_k2"]
    inp = make_inputs(s, device=DEV)
    a = layer.LayerFwd(s.S, s.D, s.E, s.K, s.F, export=True, payload="mxfp8")
    b = layer.LayerFwd(s.S, s.D, s.E, s.K, s.F, export=False, payload="mxfp8")
    ya = a(inp["x"], inp["Wr"], inp["W1"], inp["W2"], bias=inp["bias"])["y"].clone()
    yb = b(inp["x"], inp["Wr"], inp["W1"], inp["W2"], bias=inp["bias"])["y"]
    torch.cuda.synchronize()
    assert torch.equal(_bits(ya), _bits(yb))


def _mx_layer_vs_oracle(s, inp, out, n_samples, **oracle_kw):
    """y of sampled tokens against the oracle's chain on the MX payload; tokens
    whose routing the oracle decides differently (near-ties) are left out,
    and may be at most one in fifty."""
    x = np64(inp["x"])
    rng = np.random.default_rng(s.seed)
    tok = np.arange(s.S) if n_samples is None else np.sort(rng.choice(s.S, n_samples, replace=False))
    ref = O.layer_fwd(x[tok], np64(inp["Wr"]), LazyExperts(inp["W1"]), LazyExperts(inp["W2"]), s.K,
                      round_payload=False, payload="mxfp8", **oracle_kw)
    ok = np.all(npi(out["topk_idx"])[tok] == ref["topk_idx"], axis=1)
    assert ok.sum() >= len(tok) - max(1, len(tok) // 50)
    assert_bf16_close(np64(out["y"][torch.as_tensor(tok[ok], device=DEV)]), ref["y"][ok], f"{s.name} y (mxfp8)")


@pytest.mark.parametrize("name,n_samples", [("prod_tiny_s512_d256_e8_k2", None), ("prod_s16384_d2688_e192_k7", 8)])
def test_prod_layer_fwd_mxfp8(name, n_samples):
    """The paper's production variant (sigmoid routing with a selection bias,
    shared expert, balance loss) on the MX payload."""
    s = PRODUCTION[name]
    inp = make_inputs(s, device=DEV)
    lf = layer.LayerFwd(s.S, s.D, s.E, s.K, s.F, export=False, payload="mxfp8", score="sigmoid", Fs=s.Fs,
                        seq_len=s.seq_len, aux_coeff=s.aux_coeff)
    lf.out["topk_idx"] = torch.empty((s.S, s.K), dtype=torch.int32, device=DEV)
    out = lf(inp["x"], inp["Wr"], inp["W1"], inp["W2"], sel_bias=inp["sel_bias"], Ws1=inp["Ws1"], Ws2=inp["Ws2"])
    torch.cuda.synchronize()
    _mx_layer_vs_oracle(s, inp, out, n_samples, score="sigmoid", sel_bias=np64(inp["sel_bias"]),
                        Ws1=np64(inp["Ws1"]), Ws2=np64(inp["Ws2"]))


def test_latent_layer_fwd_mxfp8():
    """The latent (LatentMoE-style) layer on the MX payload: the dispatch
    encodes the latent rows."""
    s = WORKLOADS["latent_s16384_h4096_d1024_e128_k6"]
    inp = make_inputs(s, device=DEV)
    lf = layer.LayerFwd(s.S, s.D, s.E, s.K, s.F, H=s.H, export=False, payload="mxfp8")
    lf.out["topk_idx"] = torch.empty((s.S, s.K), dtype=torch.int32, device=DEV)
    out = lf(inp["x"], inp["Wr"], inp["W1"], inp["W2"], bias=inp["bias"], Wdown=inp["Wdown"], Wup=inp["Wup"])
    torch.cuda.synchronize()
    _mx_layer_vs_oracle(s, inp, out, 16, bias=None if inp["bias"] is None else np64(inp["bias"]),
                        Wdown=np64(inp["Wdown"]), Wup=np64(inp["Wup"]))
