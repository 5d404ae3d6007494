"""GPU check of moe_grouped_ffn_static, the grouped FFN entry point that
allocates nothing (its tile schedule lives in the library's fixed device
array): called through the C ABI, its outputs equal those of
moe_grouped_ffn on the same inputs bit for bit, on two calls in a row, the
second with a smaller input (fewer rows, fewer experts), so the second call
cannot lean on the first call's schedule left in the shared array."""
import numpy as np
import pytest
import torch

from paper_2608_28511_amd import _lib as L
from paper_2608_28511_amd import layer
from paper_2608_28511_amd.workloads import make_segments

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _case(R, D, F, E, seed, empty=0, skew=0.0):
    g = torch.Generator().manual_seed(seed)
    off = make_segments(R, E, seed=seed, empty=empty, skew=skew).to(DEV)
    x = torch.randn((R, D), generator=g).to(torch.bfloat16).to(DEV)
    W1 = (torch.randn((E, D, F), generator=g) / np.sqrt(D)).to(torch.bfloat16).to(DEV)
    W2 = (torch.randn((E, F, D), generator=g) / np.sqrt(F)).to(torch.bfloat16).to(DEV)
    return off, x, W1, W2


def _static(off, x, W1, W2, save_u):
    R, D = x.shape
    E, _, F = W1.shape
    h = torch.full((R, F), float("nan"), dtype=torch.bfloat16, device=DEV)
    u = torch.full((R, F), float("nan"), dtype=torch.bfloat16, device=DEV) if save_u else None
    y = torch.full((R, D), float("nan"), dtype=torch.bfloat16, device=DEV)
    L.moe_grouped_ffn_static(x, off, E, R, D, F, W1, W2, h, u, y)
    return h, u, y


def test_static_matches_workspace_entry_point_twice():
    # a large call (4096 rows over 64 experts, ragged and skewed, two empty),
    # then a smaller one (300 rows over 5 experts, one empty)
    for (R, D, F, E, seed, empty, skew) in [(4096, 256, 512, 64, 11, 2, 1.2), (300, 136, 200, 5, 12, 1, 0.0)]:
        off, x, W1, W2 = _case(R, D, F, E, seed, empty, skew)
        hs, us, ys = _static(off, x, W1, W2, save_u=True)
        h, u, y = layer.grouped_ffn(x, off, W1, W2, save_u=True)
        torch.cuda.synchronize()
        assert torch.equal(hs, h) and torch.equal(us, u) and torch.equal(ys, y), (R, E)
        assert not torch.isnan(ys).any()
