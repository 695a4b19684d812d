"""GPU parity: the HIP library against the float64 oracle.

Every comparison is element by element on the same seeded inputs (inputs
rounded to the storage type first, so the tolerance covers the GPU's own
rounding only): relative L2 <= 1e-5 for float32 storage, <= 2e-2 for
bfloat16 storage with float32 accumulation.
"""

import math

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


def _plan(w, dtype=None):
    return S.Plan(w.H, w.W, w.L, w.spins_in, w.spins_out, dtype or w.dtype)


def _ref_table(plan, which, spin):
    """Oracle value of the plan's forward / inverse table for one spin."""
    H, W, L = plan.H, plan.W, plan.L
    theta, _ = O.grid(H, W)
    w = O.dh_weights(H)
    Hp, Lp = (H + 7) // 8 * 8, (L + 31) // 32 * 32
    M = 2 * L - 1
    N = np.sqrt((2 * np.arange(L) + 1) / (4 * np.pi))
    if which == 0:
        ref = np.zeros((M, L, Hp))
        for mi in range(M):
            d = O.wigner_d(L, mi - (L - 1), -spin, theta)
            ref[mi, :, :H] = (2 * np.pi / W) * w[None, :] * (-1.0) ** spin * N[:, None] * d
    else:
        ref = np.zeros((M, Hp, Lp))
        for mi in range(M):
            d = O.wigner_d(L, mi - (L - 1), -spin, theta)
            ref[mi, :H, :L] = ((-1.0) ** spin * N[:, None] * d).T
    return ref


@pytest.mark.parametrize("name", ["tiny", "wx256"])
def test_tables_match_oracle(name):
    w = syn.workload(name)
    plan = _plan(w)
    eps = 2.0 ** -24 if w.dtype == "f32" else 2.0 ** -8   # half an ulp, relative
    for which, spins in ((0, w.spins_in), (1, w.spins_out)):
        for si, s in enumerate(spins):
            got = plan.table(which, si).to(torch.float64).numpy()
            ref = _ref_table(plan, which, s)
            # one rounding of a float64 value, plus float64 differences
            bound = 2 * eps * np.abs(ref) + 1e-14 * np.abs(ref).max()
            assert np.all(np.abs(got - ref) <= bound), (name, which, s)
            assert np.all(got[ref == 0] == 0)
    plan.close()


def _x_and_plan(name):
    w = syn.workload(name)
    x, K, d = workload_inputs(w)
    return w, x, K, d, _plan(w)


@pytest.mark.parametrize("name", ["tiny", "small", "mol", "wx128"])
def test_forward_parity(name):
    w, x, K, d, plan = _x_and_plan(name)
    got = from_device(plan.forward(to_device(x, w.dtype)))
    ref = O.forward(x, w.L, w.spins_in)
    err = rel_l2(got, ref)
    print(f"{name} forward rel-L2 {err:.3e}")
    assert err <= TOL[w.dtype]
    # rows that do not exist for spin s (l < |s|) are exactly zero
    for si, s in enumerate(w.spins_in):
        assert np.all(got[: abs(s) ** 2, :, si] == 0)
    plan.close()


@pytest.mark.parametrize("name", ["tiny", "small", "mol", "wx128"])
def test_inverse_parity(name):
    w = syn.workload(name)
    rng = np.random.default_rng(w.seed + 77)
    a = round_to(syn.random_coefficients(rng, w.L, w.B, w.spins_out, w.C_out, 1.0), w.dtype)
    plan = _plan(w)
    got = from_device(plan.inverse(to_device(a, w.dtype)))
    ref = O.inverse(a, w.H, w.W, w.spins_out)
    err = rel_l2(got, ref)
    print(f"{name} inverse rel-L2 {err:.3e}")
    assert err <= TOL[w.dtype]
    plan.close()


@pytest.mark.parametrize("name", ["tiny", "small", "mol", "wx128"])
def test_conv_parity(name):
    w, x, K, d, plan = _x_and_plan(name)
    got = from_device(plan.conv(to_device(x, w.dtype), to_device(K, w.dtype)))
    ref = O.conv(x, K, w.L, w.spins_in, w.spins_out)
    err = rel_l2(got, ref)
    print(f"{name} conv rel-L2 {err:.3e}")
    assert err <= TOL[w.dtype]
    plan.close()


def test_two_layer_stack_with_phase_collapse():
    """The molecule-shaped workload's two stacked layers: conv -> phase
    collapse -> conv."""
    w, x, K, d, plan = _x_and_plan("mol")
    K2 = round_to(d["filters2"], w.dtype)
    W1, W2, b = (np.asarray(t, dtype=np.complex64) for t in d["pc"])
    plan2 = S.Plan(w.H, w.W, w.L, w.spins_out, w.spins_out, w.dtype)
    y1 = plan.conv(to_device(x, w.dtype), to_device(K, w.dtype))
    tW1, tW2, tb = (torch.from_numpy(t).cuda() for t in (W1, W2, b))
    z = plan.phase_collapse(y1, tW1, tW2, tb)
    y2 = plan2.conv(z, to_device(K2, w.dtype))
    r1 = O.conv(x, K, w.L, w.spins_in, w.spins_out)
    rz = O.phase_collapse(r1, w.spins_out, W1.astype(complex), W2.astype(complex),
                          b.astype(complex))
    r2 = O.conv(rz, K2, w.L, w.spins_out, w.spins_out)
    for got, ref, tag in ((y1, r1, "layer1"), (z, rz, "phase collapse"), (y2, r2, "layer2")):
        err = rel_l2(from_device(got), ref)
        print(f"mol stack {tag} rel-L2 {err:.3e}")
        assert err <= TOL[w.dtype], tag
    plan.close()
    plan2.close()


PC_CASES = [
    # H, L, spins_out, C, dtype
    (32, 16, (1, 0), 5, "f32"),        # C % 16 != 0: per-output loop kernel; spin 0 second
    (4, 2, (1, 0, -1), 32, "f32"),     # register form; 16 points (< one 32-point tile)
    (32, 16, (0, 1), 64, "f32"),       # register form at the molecule workload's width
    (32, 16, (0, 1), 32, "bf16"),      # bf16 storage
    (6, 3, (0,), 16, "f32"),           # register form, 36 points: a ragged 32-point tile
    (6, 3, (2, 0), 48, "f32"),         # register form, three row tiles (odd), ragged
    (8, 4, (0, 1, -1), 64, "f32"),     # LDS-staged MFMA kernel (no register form)
    (10, 5, (0,), 80, "bf16"),         # LDS-staged MFMA kernel, 100 points (ragged)
]


@pytest.mark.parametrize("case", PC_CASES, ids=[f"H{c[0]}S{len(c[2])}C{c[3]}{c[4]}" for c in PC_CASES])
def test_phase_collapse_in_place_and_passthrough(case):
    H, L, so, C, dt = case
    rng = np.random.default_rng(5 + C)
    x = round_to(syn.complex_normal(rng, (3, len(so), C, H, H)), dt)
    W1, W2, b = (np.asarray(t, np.complex64) for t in syn.phase_collapse_parameters(rng, len(so), C))
    # grids whose width is not a power of two need the matrix longitude route
    # to make a plan; the phase collapse itself does not depend on it
    lon = "fft" if H & (H - 1) == 0 else "matmul"
    plan = S.Plan(H, H, L, (0,), so, dt, longitude=lon)
    xd = to_device(x, dt)
    tW = [torch.from_numpy(t).cuda() for t in (W1, W2, b)]
    y = from_device(plan.phase_collapse(xd, *tW))
    ref = O.phase_collapse(x, so, W1.astype(complex), W2.astype(complex), b.astype(complex))
    s0 = so.index(0)
    for i in range(len(so)):
        if i != s0:
            assert np.array_equal(y[:, i], x[:, i])      # other spins bit-identical
    err = rel_l2(y, ref)
    print(f"phase collapse {case}: rel-L2 {err:.2e}")
    assert err <= (1e-6 if dt == "f32" else TOL[dt])
    plan.phase_collapse(xd, *tW, y=xd)                     # in place
    assert np.array_equal(from_device(xd), y)
    plan.close()


EDGE = [
    # H, L, spins_in, spins_out, B, C_in, C_out, dtype
    (16, 5, (0,), (0,), 1, 1, 1, "f32"),            # L < H/2, one channel
    (16, 8, (-1, 2, 0), (1, 0, -2), 3, 3, 5, "f32"),  # odd channel counts, |s| = 2
    (2, 1, (0,), (0,), 2, 2, 3, "f32"),            # smallest grid
    (4, 2, (0, 1), (1,), 1, 4, 2, "f32"),
    (8, 4, (0,), (0, 1), 5, 7, 9, "bf16"),
    (32, 16, (0, 1), (0, 1), 2, 40, 24, "bf16"),
    # bf16 mixing through the direct-to-LDS kernels (64-wide K steps when
    # 2 C_in % 64 == 0, else 32-wide):
    (32, 16, (0, 1), (0, 1, -1), 3, 32, 44, "bf16"),  # ragged row tiles, 2 column tiles (last 4 wide)
    (16, 8, (-2, 0), (0, 1), 3, 64, 8, "bf16"),       # input spin |s| = 2 skipped below l = 2
    (16, 8, (0, 1, -2), (2, 0), 5, 48, 12, "bf16"),   # 32-wide K steps, 3 per input spin
    # bf16 latitude GEMMs through the direct-to-LDS kernels (H a multiple of 64):
    (64, 32, (0,), (0, 1), 2, 20, 64, "bf16"),        # ragged forward columns, H < one latitude tile
    (64, 32, (1, -2), (2, 0), 2, 64, 64, "bf16"),     # |s| = 2: degree ranges start at max(|m|, |s|)
    (64, 32, (1,), (0, -1), 1, 33, 17, "f32"),     # ragged tiles everywhere
    (64, 20, (0,), (0,), 3, 8, 8, "f32"),          # spectral truncation L << H/2
    # f32 through the direct-to-LDS kernels (2 B C >= 1024, S_out C_out >= 128):
    (64, 32, (0, 1), (0, 1, 2), 4, 128, 132, "f32"),  # mixing: ragged outputs, dead output spin
                                                       # below l = 2; inverse: ragged n' tiles that
                                                       # span batch items
    (32, 16, (1, 0), (0, -1), 4, 130, 128, "f32"),    # one-stage latitude GEMMs (H = 32), ragged
                                                       # forward columns
]


@pytest.mark.parametrize("case", EDGE, ids=[f"H{c[0]}L{c[1]}{c[7]}" for c in EDGE])
def test_edge_cases(case):
    H, L, si, so, B, Ci, Co, dt = case
    rng = np.random.default_rng(H * 1000 + L)
    a = syn.random_coefficients(rng, L, B, si, Ci, 0.5)
    x = round_to(O.inverse(a, H, H, si), dt)
    K = round_to(syn.random_filters(rng, L, si, Ci, so, Co, 1.0 / Ci), dt)
    plan = S.Plan(H, H, L, si, so, dt)
    xd = to_device(x, dt)
    tol = TOL[dt]
    err_f = rel_l2(from_device(plan.forward(xd)), O.forward(x, L, si))
    ac = round_to(syn.random_coefficients(rng, L, B, so, Co, 0.5), dt)
    err_i = rel_l2(from_device(plan.inverse(to_device(ac, dt))), O.inverse(ac, H, H, so))
    err_c = rel_l2(from_device(plan.conv(xd, to_device(K, dt))), O.conv(x, K, L, si, so))
    print(f"edge {case}: fwd {err_f:.2e} inv {err_i:.2e} conv {err_c:.2e}")
    assert err_f <= tol and err_i <= tol and err_c <= tol
    plan.close()


def test_non_bandlimited_input_matches_oracle_operator():
    """The transform is the quadrature operator itself, aliasing included."""
    H, L = 32, 16
    rng = np.random.default_rng(9)
    x = round_to(syn.complex_normal(rng, (2, 2, 3, H, H)), "f32")
    plan = S.Plan(H, H, L, (0, 1), (0, 1), "f32")
    err = rel_l2(from_device(plan.forward(to_device(x, "f32"))), O.forward(x, L, (0, 1)))
    assert err <= 1e-5
    plan.close()


def test_deterministic():
    w, x, K, d, plan = _x_and_plan("small")
    xd, Kd = to_device(x, w.dtype), to_device(K, w.dtype)
    y1 = plan.conv(xd, Kd).clone()
    y2 = plan.conv(xd, Kd)
    assert torch.equal(y1, y2)
    plan.close()


def test_call_validation_with_plan():
    w = syn.workload("tiny")
    plan = _plan(w)
    L = S.lib()
    x = plan.empty(1, 1, 4, 16, 16)
    c = plan.empty(64, 1, 1, 4)
    need = plan.workspace_bytes(S.OP_FORWARD, 1, 4, 1)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    xp = torch.view_as_real(x).data_ptr()
    cp = torch.view_as_real(c).data_ptr()
    assert L.swsft_forward(plan._h, 1, 4, xp, cp, ws.data_ptr(), need - 1, None) == S.E_WORKSPACE
    assert L.swsft_forward(plan._h, 1, 4, xp, cp, None, need, None) == S.E_WORKSPACE
    assert L.swsft_forward(plan._h, 0, 4, xp, cp, ws.data_ptr(), need, None) == S.E_INVALID
    assert L.swsft_forward(plan._h, 1, 4, xp + 4, cp, ws.data_ptr(), need, None) == S.E_INVALID
    assert L.swsft_forward(plan._h, 1, 4, xp, cp, ws.data_ptr(), need, None) == S.OK
    # phase collapse needs spin 0 among the output spins
    p1 = S.Plan(16, 16, 8, (0,), (1,), "f32")
    assert L.spin_sph_phase_collapse(p1._h, 1, 4, xp, xp, xp, xp, xp, None) == S.E_INVALID
    torch.cuda.synchronize()
    plan.close()
    p1.close()


# ---------------------------------------------------------------------------
# The 256 x 256, C = 256, bfloat16 workload at its full size, in the launch
# configuration the benchmark times.  Every output element is compared with
# the oracle: the whole forward transform, the whole layer output (both batch
# items, both spins, all 256 output channels) and the whole inverse.
# ---------------------------------------------------------------------------

def report(tag, got, ref, spin_axis, spins):
    """Relative L2 over the whole tensor, printed with the per-spin relative
    L2 and the largest absolute error."""
    err = rel_l2(got, ref)
    parts = []
    for si, s in enumerate(spins):
        g = np.take(got, si, axis=spin_axis)
        r = np.take(ref, si, axis=spin_axis)
        parts.append(f"spin {s}: {rel_l2(g, r):.3e} (max-abs {np.abs(g - r).max():.3e})")
    print(f"{tag} rel-L2 {err:.3e}, max-abs {np.abs(got - ref).max():.3e}; " + "; ".join(parts))
    return err


@pytest.fixture(scope="module")
def wx256():
    w = syn.workload("wx256")
    x, K, d = workload_inputs(w)
    plan = _plan(w)
    xd, Kd = to_device(x, "bf16"), to_device(K, "bf16")
    a = O.forward(x, w.L, w.spins_in)          # oracle coefficients of every input map
    yield w, x, K, a, plan, xd, Kd
    plan.close()


def test_wx256_forward_full(wx256):
    w, x, K, a, plan, xd, Kd = wx256
    coef = from_device(plan.forward(xd))
    assert coef.shape == a.shape
    err = report("wx256 forward (whole)", coef, a, 2, w.spins_in)
    assert err <= TOL["bf16"]
    for si, s in enumerate(w.spins_in):
        assert np.all(coef[: abs(s) ** 2, :, si] == 0)


def test_wx256_conv_full(wx256):
    w, x, K, a, plan, xd, Kd = wx256
    y = from_device(plan.conv(xd, Kd))
    ref = O.inverse(O.mix(a, K, w.spins_in, w.spins_out), w.H, w.W, w.spins_out)
    assert y.shape == ref.shape == (w.B, len(w.spins_out), w.C_out, w.H, w.W)
    err = report("wx256 conv (whole)", y, ref, 1, w.spins_out)
    assert err <= TOL["bf16"]


def test_wx256_inverse_full(wx256):
    w, x, K, a, plan, xd, Kd = wx256
    rng = np.random.default_rng(4242)
    c = round_to(syn.random_coefficients(rng, w.L, w.B, w.spins_out, w.C_out, 1.0), "bf16")
    y = from_device(plan.inverse(to_device(c, "bf16")))
    ref = O.inverse(c, w.H, w.W, w.spins_out)
    err = report("wx256 inverse (whole)", y, ref, 1, w.spins_out)
    assert err <= TOL["bf16"]


def test_wx256_properties_at_full_size(wx256):
    """Round trip and exact longitude-shift equivariance on every map."""
    w, x, K, a, plan, xd, Kd = wx256
    coef = plan.forward(xd)
    back = plan.inverse(coef)
    xr = torch.view_as_complex(xd.float())
    br = torch.view_as_complex(back.float())
    err_rt = (torch.linalg.vector_norm(br - xr) / torch.linalg.vector_norm(xr)).item()
    r = 37
    c1 = torch.view_as_complex(coef.float())
    c2 = torch.view_as_complex(plan.forward(torch.roll(xd, r, dims=4)).float())
    m = torch.tensor([mm for l in range(w.L) for mm in range(-l, l + 1)], device="cuda")
    ph = torch.exp(-2j * math.pi * m.double() * r / w.W).to(torch.complex64)
    err_sh = (torch.linalg.vector_norm(c2 - c1 * ph[:, None, None, None])
              / torch.linalg.vector_norm(c1)).item()
    print(f"wx256 round trip {err_rt:.3e}, shift equivariance {err_sh:.3e}")
    assert err_rt <= TOL["bf16"] and err_sh <= TOL["bf16"]
