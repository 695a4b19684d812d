"""The longitude stages as dense DFT matrix products on MFMA (plans created
with longitude="matmul"): parity of swsft_forward, swsft_inverse, the layer
and its backward pass against the float64 oracle, including grid widths that
are not powers of two (which only this route takes: 96, 768).  Tolerances as
everywhere: relative L2 <= 1e-5 (float32 storage), <= 2e-2 (bfloat16
storage)."""

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


@pytest.mark.parametrize("case", CASES, ids=[f"H{c[0]}L{c[1]}S{len(c[2])}C{c[4]}{c[5]}" for c in CASES])
def test_inverse_matmul_parity(case):
    H, L, spins, B, C, dt, _ = case
    rng = np.random.default_rng(H * 17 + C)
    a = round_to(syn.random_coefficients(rng, L, B, spins, C, 1.0), dt)
    plan = S.Plan(H, H, L, spins, spins, dt, longitude="matmul")
    got = from_device(plan.inverse(to_device(a, dt)))
    err = rel_l2(got, O.inverse(a, H, H, spins))
    print(f"matmul inverse {case}: rel-L2 {err:.2e}")
    assert err <= TOL[dt]
    plan.close()


LAYERS = [  # H, L, spins_in, spins_out, B, C_in, C_out, dtype
    (96, 48, (0,), (0, 1), 2, 3, 5, "f32"),       # W = 96: no FFT of this width
    (96, 40, (0, 1), (1,), 1, 16, 8, "bf16"),     # L < H/2
    (24, 12, (0, 1), (0, 1), 2, 8, 8, "f32"),     # one latitude tile (H < 32)
]


@pytest.mark.parametrize("case", LAYERS, ids=[f"H{c[0]}L{c[1]}{c[7]}" for c in LAYERS])
def test_layer_and_backward_at_widths_without_fft(case):
    H, L, si, so, B, Ci, Co, dt = case
    rng = np.random.default_rng(H + 7 * L)
    x = round_to(O.inverse(syn.random_coefficients(rng, L, B, si, Ci, 1.0), H, H, si), dt)
    K = round_to(syn.random_filters(rng, L, si, Ci, so, Co, 1.0 / Ci), dt)
    gy = round_to(syn.complex_normal(rng, (B, len(so), Co, H, H)), dt)
    plan = S.Plan(H, H, L, si, so, dt, longitude="matmul")
    xd, Kd = to_device(x, dt), to_device(K, dt)
    err = rel_l2(from_device(plan.conv(xd, Kd)), O.conv(x, K, L, si, so))
    gx, gk = plan.conv_backward(xd, Kd, to_device(gy, dt))
    rx, rk = O.conv_backward(x, K, gy, L, si, so)
    ex, ek = rel_l2(from_device(gx), rx), rel_l2(from_device(gk), rk)
    print(f"matmul layer {case}: conv {err:.2e}, grad_x {ex:.2e}, grad_filters {ek:.2e}")
    assert err <= TOL[dt] and ex <= TOL[dt] and ek <= TOL[dt]
    plan.close()


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_768_grid_forward_inverse_layer(dt):
    """The largest grid of the paper's FFT-vs-DFT comparison (768 x 768,
    bandlimit 384), whole outputs: forward, inverse and the layer."""
    H, L, si, so, B, Ci, Co = 768, 384, (0, 1), (0, 1), 1, 4, 4
    rng = np.random.default_rng(768)
    a = syn.random_coefficients(rng, L, B, si, Ci, 1.0)
    x = round_to(O.inverse(a, H, H, si), dt)
    K = round_to(syn.random_filters(rng, L, si, Ci, so, Co, 1.0 / (2 * Ci)), dt)
    plan = S.Plan(H, H, L, si, so, dt, longitude="matmul")
    xd = to_device(x, dt)
    coef = from_device(plan.forward(xd))
    ref_a = O.forward(x, L, si)
    e_f = rel_l2(coef, ref_a)
    ac = round_to(a, dt)
    e_i = rel_l2(from_device(plan.inverse(to_device(ac, dt))), O.inverse(ac, H, H, si))
    e_c = rel_l2(from_device(plan.conv(xd, to_device(K, dt))),
                 O.inverse(O.mix(ref_a, K, si, so), H, H, so))
    print(f"768x768 {dt}: forward {e_f:.2e}, inverse {e_i:.2e}, conv {e_c:.2e}")
    assert e_f <= TOL[dt] and e_i <= TOL[dt] and e_c <= TOL[dt]
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
