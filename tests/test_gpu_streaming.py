"""Transforms whose DFT launches move at least 128 MiB read their large input
(forward) or write their large output (inverse) with the non-temporal cache
hint.  The hint changes no arithmetic and every map is transformed on its
own, so the transform of such a batch must equal, bit for bit, the
transforms of its halves (launches just below the threshold that take the
same kernels: 2 B C >= 1024 keeps the direct-to-LDS latitude GEMMs); one
channel is also checked against the float64 oracle.  The bfloat16 form of
the hinted launches is exercised by the 256x256 parity tests."""

import numpy as np
import pytest
import torch

import oracle as O
from paper_2306_05420_amd import swsft as S
from helpers import TOL, from_device, rel_l2

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    S.lib()
    yield
    torch.cuda.synchronize()


def test_streamed_float_transforms_equal_itemwise():
    # 128x128 grid, L = 64, B = 8, C = 128, spin 0, float32: the forward DFT
    # moves x 134 MB + X 133 MB and the inverse DFT the same, both above the
    # 128 MiB threshold; half the batch moves 127.5 MiB
    H, L, B, C, spins = 128, 64, 8, 128, (0,)
    plan = S.Plan(H, H, L, spins, spins, "f32")
    gen = torch.Generator(device="cuda").manual_seed(20261202)
    x = torch.randn(B, 1, C, H, H, dtype=torch.complex64, device="cuda", generator=gen)
    coef = plan.forward(x)
    y = plan.inverse(coef)
    h = B // 2
    for b0 in (0, h):
        cb = plan.forward(x[b0:b0 + h].contiguous())
        assert torch.equal(cb, coef[:, b0:b0 + h]), f"forward, items {b0}..{b0 + h - 1}"
        yb = plan.inverse(coef[:, b0:b0 + h].contiguous())
        assert torch.equal(yb, y[b0:b0 + h]), f"inverse, items {b0}..{b0 + h - 1}"
    # one channel against the oracle (any input: the quadrature is the operator)
    xc = from_device(x[0:1, :, 0:1])
    ef = rel_l2(from_device(coef[:, 0:1, :, 0:1]), O.forward(xc, L, spins))
    ac = from_device(coef[:, 0:1, :, 0:1])
    ei = rel_l2(from_device(y[0:1, :, 0:1]), O.inverse(ac, H, H, spins))
    print(f"streamed float transforms: forward {ef:.2e}, inverse {ei:.2e}")
    assert ef <= TOL["f32"] and ei <= TOL["f32"]
    plan.close()
