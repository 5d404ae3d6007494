"""The layer forward called from plain C (tests/c_abi/layer_fwd_c.c: HIP
runtime allocations, no Python, no torch) gives bit for bit what the Python
binding gives on the same inputs: y, the router logits and the top-K
indices.  The C program also checks, before its call, that an invalid shape
and a short workspace are rejected with their status codes."""
import importlib.util
import subprocess
from pathlib import Path

import numpy as np
import pytest
import torch

from paper_2608_28511_amd import layer
from paper_2608_28511_amd.workloads import MoEShape, make_inputs

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
ROOT = Path(__file__).resolve().parents[1]

SHAPES = [MoEShape("c_s1000_d256_e16_k4", S=1000, D=256, E=16, K=4, F=264, bias="none", seed=31),
          MoEShape("c_s4096_d1024_e64_k6", S=4096, D=1024, E=64, K=6, F=1032, seed=32)]


def _consumer():
    spec = importlib.util.spec_from_file_location("c_abi_build", ROOT / "tests" / "c_abi" / "build.py")
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod.ensure_built()


@pytest.mark.parametrize("s", SHAPES, ids=lambda s: s.name)
def test_c_consumer_matches_binding(s, tmp_path):
    exe = _consumer()
    inp = make_inputs(s, device=DEV)
    lf = layer.LayerFwd(s.S, s.D, s.E, s.K, s.F, export=True)
    out = lf(inp["x"], inp["Wr"], inp["W1"], inp["W2"])
    torch.cuda.synchronize()

    def raw(t):
        return t.detach().contiguous().cpu().view(torch.uint8).numpy().tobytes()

    (tmp_path / "shape.txt").write_text(f"{s.S} {s.D} {s.E} {s.K} {s.F}\n")
    for name in ("x", "Wr", "W1", "W2"):
        (tmp_path / f"{name}.bin").write_bytes(raw(inp[name]))
    r = subprocess.run([str(exe), str(tmp_path)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    for name, dtype in (("y", np.uint16), ("logits", np.uint32), ("topk_idx", np.int32)):
        got = np.frombuffer((tmp_path / f"{name}.bin").read_bytes(), dtype=dtype)
        want = np.frombuffer(raw(out[name]), dtype=dtype)
        assert got.shape == want.shape and np.array_equal(got, want), f"{s.name}: {name} differs"
