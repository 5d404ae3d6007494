"""moe_layer_fwd captured into a HIP graph and replayed.

Every entry point only enqueues kernels on the caller's stream (no
allocation, copy, memset or host synchronisation), so a layer call made while
the stream is captured (torch.cuda.CUDAGraph on the launch stream) records the
whole forward.  Each replay must reproduce the eager call bit for bit, in
every exported output: the outputs are overwritten with NaN / sentinel values
before each replay, eager layer calls on the same buffers run between
replays, and after new input values are copied into the captured input
buffer the replay must give the new eager result.  Covered: the plain layer
(materialised and fused dispatch), the MX-FP8 payload, the latent layer, the
production layer (sigmoid routing, shared expert, sequence loss) and a whole
forward and backward step through the separate entry points.
"""
import pytest
import torch

from paper_2608_28511_amd import layer
from paper_2608_28511_amd.workloads import MoEShape, make_inputs

pytestmark = pytest.mark.gpu
DEV = "cuda:0"

PLAIN = MoEShape("graph_s2048_d1024_e64_k6", S=2048, D=1024, E=64, K=6, F=1032, bias="normal", seed=21)
LATENT = MoEShape("graph_s1024_h2048_d512_e32_k4", S=1024, D=512, E=32, K=4, F=768, H=2048, seed=22)
PROD = MoEShape("graph_prod_s1024_d512_e32_k4", S=1024, D=512, E=32, K=4, F=512, seed=23, score="sigmoid",
                sel_bias_std=0.05, Fs=512, seq_len=256, aux_coeff=1e-4)

CASES = {
    "plain": (PLAIN, dict(export=True)),
    "plain_fused_dispatch": (PLAIN, dict(export=False)),
    "mxfp8_payload": (PLAIN, dict(export=True, payload="mxfp8")),
    "latent": (LATENT, dict(export=True)),
    "production": (PROD, dict(export=True, save_u=True, score="sigmoid", Fs=PROD.Fs, seq_len=PROD.seq_len,
                              aux_coeff=PROD.aux_coeff)),
}


def _call(lf, inp):
    return lf(inp["x"], inp["Wr"], inp["W1"], inp["W2"], bias=inp["bias"], Wdown=inp.get("Wdown"),
              Wup=inp.get("Wup"), sel_bias=inp.get("sel_bias"), Ws1=inp.get("Ws1"), Ws2=inp.get("Ws2"))


def _snapshot(out):
    return {k: v.clone() for k, v in out.items() if v is not None}


def _clobber(out):
    """Overwrite every output so that a replay that skipped a write shows."""
    for v in out.values():
        if v is None:
            continue
        if v.is_floating_point():
            v.fill_(float("nan"))
        elif v.dtype == torch.uint8:
            v.fill_(0xAB)
        else:
            v.fill_(-7)


def _assert_same(out, ref, what):
    for k, r in ref.items():
        # bitwise, NaN payloads included: compare the raw bytes
        got = out[k].contiguous().view(torch.uint8)
        assert torch.equal(got, r.contiguous().view(torch.uint8)), f"{what}: {k} differs from the eager call"


@pytest.mark.parametrize("name", list(CASES))
def test_layer_graph_replay(name):
    s, kw = CASES[name]
    inp = make_inputs(s, device=DEV)
    lf = layer.LayerFwd(s.S, s.D, s.E, s.K, s.F, H=s.H, **kw)
    _call(lf, inp)
    torch.cuda.synchronize()
    ref = _snapshot(lf.out)
    assert not torch.isnan(ref["y"].float()).any()

    # one call on a side stream before the capture, as torch's graph API asks
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        _call(lf, inp)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        _call(lf, inp)
    torch.cuda.synchronize()

    for rep in range(3):
        _clobber(lf.out)
        g.replay()
        torch.cuda.synchronize()
        _assert_same(lf.out, ref, f"{name}: replay {rep}")
        _clobber(lf.out)
        _call(lf, inp)
        torch.cuda.synchronize()
        _assert_same(lf.out, ref, f"{name}: eager call after replay {rep}")

    # new values in the captured input buffer: the replay reads them
    x2 = make_inputs(s.scaled(seed=s.seed + 100), device=DEV, with_experts=False)["x"]
    inp["x"].copy_(x2)
    _call(lf, inp)
    torch.cuda.synchronize()
    ref2 = _snapshot(lf.out)
    assert not torch.equal(ref2["y"], ref["y"])
    _clobber(lf.out)
    g.replay()
    torch.cuda.synchronize()
    _assert_same(lf.out, ref2, f"{name}: replay with new x")


SKEW = MoEShape("graph_skew_s2048_d512_e32_k4_bwd", S=2048, D=512, E=32, K=4, F=384, bias="zipf",
                backward=True, seed=24)


def _train_step(inp, K):
    """Router, route, dispatch, experts, combine and the whole backward
    (combine^T, expert dgrads and wgrads, router backward, dispatch^T with the
    router's input gradient added), on the current stream, no host sync."""
    x, Wr, W1, W2, dy = inp["x"], inp["Wr"], inp["W1"], inp["W2"], inp["dy"]
    S = x.shape[0]
    logits = layer.router_logits(x, Wr, inp["bias"])
    r = layer.route(logits, K)
    x_disp, p_disp = layer.dispatch(x, r["topk_prob"], r["inv_perm"], K)
    h, u, yd = layer.grouped_ffn(x_disp, r["offsets"], W1, W2, save_u=True)
    y = layer.combine(yd, p_disp, r["inv_perm"], S, K)
    dyd, dp = layer.combine_bwd(dy, yd, p_disp, r["inv_perm"], K)
    dxd, dW1, dW2 = layer.grouped_ffn_bwd(x_disp, u, h, dyd, r["offsets"], W1, W2)
    rb = layer.router_bwd(x, Wr, r["topk_idx"], r["topk_prob"], dp)
    dx = layer.dispatch_bwd(dxd, r["inv_perm"], S, K, dx_add=rb["dx_r"])
    return dict(logits=logits, topk_idx=r["topk_idx"], perm=r["perm"], y=y, dp=dp, dW1=dW1, dW2=dW2,
                dWr=rb["dWr"], dbias=rb["dbias"], dx=dx)


def test_train_step_graph_replay():
    """A forward and backward step on Zipf routing (dead experts included)
    captured once: every replay equals the eager step bit for bit, also after
    new x and dy are copied into the captured inputs."""
    s = SKEW
    inp = make_inputs(s, device=DEV)
    ref = _snapshot(_train_step(inp, s.K))
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        _train_step(inp, s.K)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        out = _train_step(inp, s.K)
    torch.cuda.synchronize()
    for rep in range(3):
        _clobber(out)
        g.replay()
        torch.cuda.synchronize()
        _assert_same(out, ref, f"train step: replay {rep}")
        _train_step(inp, s.K)   # eager work between the replays
        torch.cuda.synchronize()
    new = make_inputs(s.scaled(seed=s.seed + 100), device=DEV, with_experts=False)
    inp["x"].copy_(new["x"])
    inp["dy"].copy_(new["dy"])
    ref2 = _snapshot(_train_step(inp, s.K))
    torch.cuda.synchronize()
    assert not torch.equal(ref2["dW1"], ref["dW1"])
    _clobber(out)
    g.replay()
    torch.cuda.synchronize()
    _assert_same(out, ref2, "train step: replay with new x and dy")
