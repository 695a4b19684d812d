"""The forward longitude stage as a dense DFT matrix product on MFMA (plans
created with longitude="matmul"): parity of swsft_forward, and of the layer,
against the float64 oracle, including grid widths that are not powers of two
(which only this route takes).  Tolerances as everywhere: relative L2
<= 1e-5 (float32 storage), <= 2e-2 (bfloat16 storage)."""

import numpy as np
import pytest
import torch

import oracle as O
from paper_2306_05420_amd import swsft as S
from paper_2306_05420_amd import synthetic as syn
from helpers import TOL, from_device, rel_l2, round_to, to_device, workload_inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    S.lib()
    yield
    torch.cuda.synchronize()


CASES = [  # H, L, spins, B, C, dtype, band-limited input
    (16, 8, (0,), 1, 4, "f32", True),
    (32, 16, (0, 1), 3, 16, "f32", True),
    (64, 32, (0, 1), 2, 16, "bf16", True),
    (96, 48, (0,), 2, 3, "f32", True),        # W = 96: not a power of two
    (96, 40, (0, -1), 1, 5, "f32", False),    # L < H/2, non-band-limited input
    (24, 12, (0, 1), 1, 8, "bf16", True),
    (6, 3, (0,), 2, 2, "bf16", True),         # 2W not a multiple of 8: element loads
    (128, 64, (0,), 2, 32, "f32", True),
]


@pytest.mark.parametrize("case", CASES, ids=[f"H{c[0]}L{c[1]}S{len(c[2])}C{c[4]}{c[5]}" for c in CASES])
def test_forward_matmul_parity(case):
    H, L, spins, B, C, dt, bl = case
    rng = np.random.default_rng(H * 13 + C)
    if bl:
        x = O.inverse(syn.random_coefficients(rng, L, B, spins, C, 1.0), H, H, spins)
    else:
        x = syn.complex_normal(rng, (B, len(spins), C, H, H))
    x = round_to(x, dt)
    plan = S.Plan(H, H, L, spins, spins, dt, longitude="matmul")
    got = from_device(plan.forward(to_device(x, dt)))
    ref = O.forward(x, L, spins)
    err = rel_l2(got, ref)
    print(f"matmul forward {case}: rel-L2 {err:.2e}")
    assert err <= TOL[dt]
    for si, s in enumerate(spins):
        assert np.all(got[: abs(s) ** 2, :, si] == 0)
    plan.close()


@pytest.mark.parametrize("name", ["small", "mol"])
def test_layer_with_matmul_longitude(name):
    w = syn.workload(name)
    x, K, _ = workload_inputs(w)
    plan = S.Plan(w.H, w.W, w.L, w.spins_in, w.spins_out, w.dtype, longitude="matmul")
    got = from_device(plan.conv(to_device(x, w.dtype), to_device(K, w.dtype)))
    err = rel_l2(got, O.conv(x, K, w.L, w.spins_in, w.spins_out))
    print(f"{name} conv with the matmul longitude stage: rel-L2 {err:.2e}")
    assert err <= TOL[w.dtype]
    plan.close()


def test_width_without_fft_rejects_the_inverse_stage():
    plan = S.Plan(96, 96, 48, (0,), (0,), "f32", longitude="matmul")
    c = plan.empty(48 * 48, 1, 1, 2)
    x = plan.empty(1, 1, 2, 96, 96)
    K = plan.empty(48, 1, 2, 1, 2)
    for call in (lambda: plan.inverse(c), lambda: plan.conv(x, K),
                 lambda: plan.conv_backward(x, K, x)):
        with pytest.raises(S.SwsftError) as e:
            call()
        assert e.value.status == S.E_UNSUPPORTED
    plan.close()


def test_wx256_matmul_forward_sampled():
    """Full 256 x 256 bf16 size through the matmul route: batch item 0."""
    w = syn.workload("wx256")
    x, _, _ = workload_inputs(w)
    plan = S.Plan(w.H, w.W, w.L, w.spins_in, w.spins_out, "bf16", longitude="matmul")
    coef = from_device(plan.forward(to_device(x, "bf16"))[:, :1])
    err = rel_l2(coef, O.forward(x[:1], w.L, w.spins_in))
    print(f"wx256 matmul forward rel-L2 {err:.3e}")
    assert err <= TOL["bf16"]
    plan.close()
