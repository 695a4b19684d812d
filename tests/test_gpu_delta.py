"""The latitude stages by the Wigner-Delta route (eqs. (4)-(6)), with and
without the J / G symmetries: the same operators as the direct route, so the
GPU results are compared with the float64 oracle's transforms (themselves
pinned against the Delta-route oracle).  Tolerances as everywhere: relative
L2 <= 1e-5 (float32 storage), <= 2e-2 (bfloat16 storage)."""

import numpy as np
import pytest
import torch

import oracle as O
from paper_2306_05420_amd import swsft as S
from paper_2306_05420_amd import synthetic as syn
from helpers import TOL, from_device, rel_l2, round_to, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    S.lib()
    yield
    torch.cuda.synchronize()


CASES = [  # H, L, spins_in, spins_out, B, C_in, C_out, dtype
    (64, 32, (0,), (0,), 2, 4, 4, "f32"),
    (64, 32, (0, 1, -2), (1, 0), 2, 3, 5, "f32"),
    (128, 64, (0,), (0, 1), 1, 8, 8, "f32"),
    (64, 32, (0, 1), (0, 1), 2, 16, 16, "bf16"),
    (128, 32, (1,), (0,), 1, 8, 8, "f32"),      # L < H/2
]


@pytest.mark.parametrize("route", ["delta", "delta_sym"])
@pytest.mark.parametrize("case", CASES, ids=[f"H{c[0]}L{c[1]}S{len(c[2])}{len(c[3])}{c[7]}" for c in CASES])
def test_delta_route_parity(case, route):
    H, L, si, so, B, Ci, Co, dt = case
    rng = np.random.default_rng(H + L + Ci)
    x = round_to(syn.complex_normal(rng, (B, len(si), Ci, H, H)), dt)   # not band-limited
    a = round_to(syn.random_coefficients(rng, L, B, so, Co, 0.5), dt)
    K = round_to(syn.random_filters(rng, L, si, Ci, so, Co, 1.0 / (len(si) * Ci)), dt)
    plan = S.Plan(H, H, L, si, so, dt, latitude=route)
    plan.stage_timing(True)
    e_f = rel_l2(from_device(plan.forward(to_device(x, dt))), O.forward(x, L, si))
    assert plan.stage_times()["delta_theta"][1] == 1       # the route ran
    plan.stage_timing(False)
    e_i = rel_l2(from_device(plan.inverse(to_device(a, dt))), O.inverse(a, H, H, so))
    e_c = rel_l2(from_device(plan.conv(to_device(x, dt), to_device(K, dt))),
                 O.conv(x, K, L, si, so))
    print(f"{route} {case}: forward {e_f:.2e} inverse {e_i:.2e} conv {e_c:.2e}")
    assert e_f <= TOL[dt] and e_i <= TOL[dt] and e_c <= TOL[dt]
    plan.close()


def test_delta_route_rejects_backward():
    plan = S.Plan(64, 64, 32, (0,), (0,), "f32", latitude="delta_sym")
    x = plan.empty(1, 1, 2, 64, 64)
    K = plan.empty(32, 1, 2, 1, 2)
    with pytest.raises(S.SwsftError) as e:
        plan.conv_backward(x, K, x)
    assert e.value.status == S.E_UNSUPPORTED
    plan.close()
