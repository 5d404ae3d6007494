"""Seeded random layer shapes on the GPU against the oracle, every token
compared: model and expert widths that are any multiple of 8 (k and n tails
in every GEMM), expert counts from 1 to 300, top-K up to 12, token counts
from 1 up, router biases that unbalance or empty experts, the MX-FP8 payload
and the production variant (sigmoid routing, shared expert, balance loss).
The checks are those of the fixed-shape layer tests: exact routing for
tokens away from score ties, valid routing for the rest, and the bf16
output bar; the backward chain (combine^T, both dgrads and wgrads,
dispatch^T) is held to its elementwise bounds."""
import numpy as np
import pytest
import torch

from paper_2608_28511_amd import layer
from paper_2608_28511_amd.workloads import PRODUCTION, WORKLOADS, make_inputs

from gpu_helpers import np64
from test_gpu_backward import check_backward_case
from test_gpu_layer import DEV, check_layer, run_layer
from test_gpu_mxfp8 import _mx_layer_vs_oracle
from test_gpu_production import check_prod_layer, run_prod_layer
from test_gpu_ffn import test_grouped_ffn_exact as _ffn_exact_case
from test_gpu_ffn import test_grouped_ffn_random as _ffn_random_case
from test_gpu_ffn import test_latent_proj as _latent_proj_case
from test_gpu_mxfp8 import test_dispatch_mxfp8_bit_exact as _mx_dispatch_case
from test_gpu_permute import test_combine_bwd_matches_oracle as _combine_bwd_case
from test_gpu_permute import test_combine_matches_oracle as _combine_case
from test_gpu_permute import test_dispatch_bit_exact_and_eq1_bytes as _dispatch_case
from test_gpu_production import test_combine_add as _combine_add_case
from test_gpu_production import test_route_sigmoid_suites as _route_sigmoid_case
from test_gpu_production import test_router_bwd_sigmoid_matches_oracle as _router_bwd_sigmoid_case
from test_gpu_production import test_seq_aux_loss as _seq_aux_case
from test_gpu_production import test_shared_expert_bwd as _shared_bwd_case
from test_gpu_production import test_shared_expert_fwd as _shared_fwd_case
from test_gpu_route import test_route_suites as _route_case
from test_gpu_route import test_router_logits as _router_logits_case
from test_gpu_router_bwd import test_latent_proj_bwd_matches_oracle as _latent_bwd_case
from test_gpu_router_bwd import test_router_bwd_matches_oracle as _router_bwd_case

pytestmark = pytest.mark.gpu


def _shape(i, mx=False):
    rng = np.random.default_rng(7000 + i)
    E = int(rng.integers(1, 301))
    bias = ["none", "normal", "zipf"][i % 3] if E >= 18 else "none"
    K = int(rng.integers(1, min(E - (5 if bias == "zipf" else 0), 12) + 1))
    S = int(rng.integers(1, 301))
    D = 32 * int(rng.integers(1, 25)) if mx else 8 * int(rng.integers(1, 97))
    F = 8 * int(rng.integers(1, 97))
    return WORKLOADS["tiny_s512_d256_e8_k2"].scaled(name=f"random{i}", S=S, D=D, E=E, K=K, F=F, bias=bias,
                                                    seed=100 + i)


def _ids(i, mx=False):
    s = _shape(i, mx)
    return f"s{s.S}_d{s.D}_e{s.E}_k{s.K}_f{s.F}_{s.bias}"


@pytest.mark.parametrize("i", range(24), ids=lambda i: _ids(i))
def test_random_layer_fwd(i):
    s = _shape(i)
    inp = make_inputs(s, device=DEV)
    out = run_layer(s, inp)
    n_amb = check_layer(s, inp, out)
    assert n_amb <= max(2, s.S // 8)
    # the fused dispatch (no exported intermediates) gives the same y bit for bit
    lf = layer.LayerFwd(s.S, s.D, s.E, s.K, s.F, export=False)
    y = lf(inp["x"], inp["Wr"], inp["W1"], inp["W2"], bias=inp["bias"])["y"]
    torch.cuda.synchronize()
    assert torch.equal(y, out["y"])


@pytest.mark.parametrize("i", range(8), ids=lambda i: _ids(i, mx=True))
def test_random_layer_fwd_mxfp8(i):
    s = _shape(i, mx=True)
    inp = make_inputs(s, device=DEV)
    lf = layer.LayerFwd(s.S, s.D, s.E, s.K, s.F, export=True, payload="mxfp8")
    out = lf(inp["x"], inp["Wr"], inp["W1"], inp["W2"], bias=inp["bias"])
    torch.cuda.synchronize()
    _mx_layer_vs_oracle(s, inp, out, None, bias=None if inp["bias"] is None else np64(inp["bias"]))


def _prod_shape(i):
    rng = np.random.default_rng(9000 + i)
    E = int(rng.integers(2, 129))
    K = int(rng.integers(1, min(E, 8) + 1))
    T = 8 * int(rng.integers(1, 17))
    S = T * int(rng.integers(1, 5))
    D = 8 * int(rng.integers(1, 65))
    F = 8 * int(rng.integers(1, 65))
    Fs = 8 * int(rng.integers(1, 65))
    return PRODUCTION["prod_tiny_s512_d256_e8_k2"].scaled(name=f"prod_random{i}", S=S, D=D, E=E, K=K, F=F, Fs=Fs,
                                                          seq_len=T, seed=200 + i)


@pytest.mark.parametrize("i", range(8), ids=lambda i: "s{S}_t{seq_len}_d{D}_e{E}_k{K}_f{F}_fs{Fs}".format(
    **_prod_shape(i).__dict__))
def test_random_prod_layer_fwd(i):
    s = _prod_shape(i)
    inp = make_inputs(s, device=DEV)
    out = run_prod_layer(s, inp)
    n_amb = check_prod_layer(s, inp, out, None, s.aux_coeff)
    assert n_amb <= max(2, s.S // 8)


def _bwd_shape(i):
    rng = np.random.default_rng(11000 + i)
    E = int(rng.integers(2, 201))
    K = int(rng.integers(1, min(E - 1, 10) + 1))
    S = int(rng.integers(1, 301))
    D = 8 * int(rng.integers(1, 65))
    F = 8 * int(rng.integers(1, 65))
    return S, D, E, K, F


@pytest.mark.parametrize("i", range(12), ids=lambda i: "s{}_d{}_e{}_k{}_f{}".format(*_bwd_shape(i)))
def test_random_backward(i):
    S, D, E, K, F = _bwd_shape(i)
    check_backward_case(S, D, E, K, F, seed=300 + i)


def _latent_shape(i):
    rng = np.random.default_rng(13000 + i)
    E = int(rng.integers(1, 97))
    K = int(rng.integers(1, min(E, 8) + 1))
    S = int(rng.integers(1, 257))
    H = 8 * int(rng.integers(1, 97))
    D = 8 * int(rng.integers(1, 65))
    F = 8 * int(rng.integers(1, 65))
    return WORKLOADS["latent_s16384_h4096_d1024_e128_k6"].scaled(name=f"latent_random{i}", S=S, H=H, D=D, E=E,
                                                                 K=K, F=F, seed=400 + i)


@pytest.mark.parametrize("i", range(6), ids=lambda i: "s{S}_h{H}_d{D}_e{E}_k{K}_f{F}".format(
    **_latent_shape(i).__dict__))
def test_random_latent_layer_fwd(i):
    """The latent layer (dense projections H -> D before routing and D -> H
    after the combine) at random widths: x_lat within its fp32/bf16 bound,
    routing from the GPU's own latent rows, y against the oracle."""
    s = _latent_shape(i)
    inp = make_inputs(s, device=DEV)
    out = run_layer(s, inp)
    n_amb = check_layer(s, inp, out)
    assert n_amb <= max(2, s.S // 8)


def _router_bwd_shape(i):
    rng = np.random.default_rng(15000 + i)
    E = int(rng.integers(2, 301))
    return (int(rng.integers(1, 601)), 8 * int(rng.integers(1, 129)), E, int(rng.integers(1, min(E, 12) + 1)))


@pytest.mark.parametrize("i", range(8), ids=lambda i: "s{}_d{}_e{}_k{}".format(*_router_bwd_shape(i)))
def test_random_router_bwd(i):
    """Router backward (softmax renormalisation gradient, dWr, dbias, dx_r)
    at random shapes, with the fixed-shape test's elementwise bounds."""
    _router_bwd_case(*_router_bwd_shape(i))


def _latent_bwd_shape(i):
    rng = np.random.default_rng(17000 + i)
    return int(rng.integers(1, 801)), 8 * int(rng.integers(1, 129)), 8 * int(rng.integers(1, 129))


@pytest.mark.parametrize("i", range(6), ids=lambda i: "m{}_k{}_n{}".format(*_latent_bwd_shape(i)))
def test_random_latent_proj_bwd(i):
    """Latent projection backward (dx_in, dW) at random shapes."""
    _latent_bwd_case(*_latent_bwd_shape(i))


# Every other entry point with shape arguments, at seeded random shapes that
# keep each test's own rules (widths multiples of 8, MX widths of 32, K <= E,
# sequences that divide the tokens).
def _r(i, salt):
    return np.random.default_rng(19000 + 100 * salt + i)


def _w(rng, hi):
    return 8 * int(rng.integers(1, hi + 1))


def _stage_cases():
    cases = []
    kinds = ["normal", "quantised", "equal", "signed0", "masked"]
    for i in range(5):
        rng = _r(i, 1)
        E = int(rng.integers(1, 1025)); S = int(rng.integers(1, 3001))
        cases.append(("route", (kinds[i], S, E, int(rng.integers(1, min(E, 32) + 1)))))
        rng = _r(i, 2)
        E = int(rng.integers(1, 1025)); S = int(rng.integers(1, 3001))
        cases.append(("route_sigmoid", (kinds[i], S, E, int(rng.integers(1, min(E, 32) + 1)), bool(i % 2))))
    for i in range(4):
        rng = _r(i, 3)
        cases.append(("router_logits", (int(rng.integers(1, 2001)), _w(rng, 300), int(rng.integers(1, 300)),
                                        bool(i % 2))))
        rng = _r(i, 4)
        T = int(rng.integers(1, 400)); E = int(rng.integers(1, 400))
        cases.append(("seq_aux", (T * int(rng.integers(1, 6)), E, int(rng.integers(1, min(E, 12) + 1)), T)))
        rng = _r(i, 5)
        T = int(rng.integers(1, 300)); E = int(rng.integers(2, 300))
        cases.append(("router_bwd_sigmoid", (T * int(rng.integers(1, 4)), _w(rng, 200), E,
                                             int(rng.integers(1, min(E, 8) + 1)), T, bool(i % 2))))
        rng = _r(i, 6)
        cases.append(("shared_fwd", (int(rng.integers(1, 1500)), _w(rng, 200), _w(rng, 200))))
        rng = _r(i, 7)
        cases.append(("shared_bwd", (int(rng.integers(1, 1500)), _w(rng, 200), _w(rng, 200))))
        rng = _r(i, 8)
        cases.append(("combine_add", (int(rng.integers(1, 1500)), _w(rng, 300), int(rng.integers(1, 13)))))
        for name, salt in (("dispatch", 9), ("combine", 10), ("combine_bwd", 11)):
            rng = _r(i, salt)
            E = int(rng.integers(1, 300))
            cases.append((name, (int(rng.integers(1, 1500)), _w(rng, 300), E, int(rng.integers(1, min(E, 12) + 1)))))
        rng = _r(i, 12)
        E = int(rng.integers(1, 200))
        cases.append(("ffn_exact" if i % 2 else "ffn_random",
                      (int(rng.integers(1, 4000)), _w(rng, 80), _w(rng, 80), E, int(rng.integers(0, E)),
                       float(rng.choice([0.0, 1.5])))))
        rng = _r(i, 13)
        cases.append(("latent_proj", (int(rng.integers(1, 3000)), _w(rng, 200), _w(rng, 200))))
        rng = _r(i, 14)
        D = 32 * int(rng.integers(4, 60))
        cases.append(("mx_dispatch", (["normal", "wide", "tiny", "edge"][i], int(rng.integers(1, 800)), D,
                                      int(rng.integers(1, 9)))))
    return cases


_STAGES = {"route": _route_case, "route_sigmoid": _route_sigmoid_case, "router_logits": _router_logits_case,
           "seq_aux": _seq_aux_case, "router_bwd_sigmoid": _router_bwd_sigmoid_case,
           "shared_fwd": _shared_fwd_case, "shared_bwd": _shared_bwd_case, "combine_add": _combine_add_case,
           "dispatch": _dispatch_case, "combine": _combine_case, "combine_bwd": _combine_bwd_case,
           "ffn_exact": _ffn_exact_case, "ffn_random": _ffn_random_case, "latent_proj": _latent_proj_case,
           "mx_dispatch": _mx_dispatch_case}
_STAGE_CASES = _stage_cases()


@pytest.mark.parametrize("name,args", _STAGE_CASES,
                         ids=[f"{n}-" + "_".join(str(a) for a in args) for n, args in _STAGE_CASES])
def test_random_stage(name, args):
    _STAGES[name](*args)
