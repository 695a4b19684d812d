"""Pins of the oracle's convolution layer, phase collapse and bump synthesis.

Independent facts: brute-force spatial SO(3) convolution (eq. (1)) with a
zonal kernel on a tiny grid, evaluated with a Gauss--Legendre rule; identity,
scalar and channel-permutation filters; the spin-raising filter against
finite differences of the field; phase-collapse invariants and selector
matrices; the Funk--Hecke bump projection against direct evaluation."""

import math

import numpy as np
import pytest
from numpy.polynomial import legendre

import oracle as O
from paper_2306_05420_amd import synthetic as syn


def _identity_filters(L, spins_in, C_in, spins_out, C_out):
    K = np.zeros((L, len(spins_out), C_out, len(spins_in), C_in), complex)
    for ti, t in enumerate(spins_out):
        for si, s in enumerate(spins_in):
            if s == t:
                for c in range(min(C_in, C_out)):
                    K[:, ti, c, si, c] = 1.0
    return K


@pytest.mark.parametrize("spins", [(0,), (0, 1), (1, -1, 0)])
def test_identity_filter_is_identity(spins):
    H, L = 16, 8
    rng = np.random.default_rng(10)
    a = syn.random_coefficients(rng, L, 2, spins, 3)
    x = O.inverse(a, H, H, spins)
    K = _identity_filters(L, spins, 3, spins, 3)
    np.testing.assert_allclose(O.conv(x, K, L, spins, spins), x, atol=1e-13)


def test_scalar_and_permutation_filters():
    H, L, spins = 16, 8, (0, 1)
    rng = np.random.default_rng(11)
    a = syn.random_coefficients(rng, L, 1, spins, 3)
    x = O.inverse(a, H, H, spins)
    # scalar: K_l = c I
    K = 0.3j * _identity_filters(L, spins, 3, spins, 3)
    np.testing.assert_allclose(O.conv(x, K, L, spins, spins), 0.3j * x, atol=1e-13)
    # permutation of (spin, channel): out (t, c') <- in (s, c) with t = s, c' = (c+1) % 3,
    # and a spin swap in the output list
    spins_out = (1, 0)
    K = np.zeros((L, 2, 3, 2, 3), complex)
    for si, s in enumerate(spins):
        ti = spins_out.index(s)
        for c in range(3):
            K[:, ti, (c + 1) % 3, si, c] = 1.0
    y = O.conv(x, K, L, spins, spins_out)
    for si, s in enumerate(spins):
        ti = spins_out.index(s)
        for c in range(3):
            np.testing.assert_allclose(y[:, ti, (c + 1) % 3], x[:, si, c], atol=1e-13)


def test_mix_loop_and_masking():
    """mix against an explicit loop over (l, m), and the rule that spins with
    |s| > l or |t| > l take no part (even where the filter is not zero)."""
    rng = np.random.default_rng(12)
    L, B, spins_in, spins_out, C, Co = 4, 2, (0, 2), (1, -2), 2, 3
    a = syn.random_coefficients(rng, L, B, spins_in, C)
    K = syn.random_filters(rng, L, spins_in, C, spins_out, Co, 1.0)
    out = O.mix(a, K, spins_in, spins_out)
    for l in range(L):
        for m in range(-l, l + 1):
            r = O.coef_index(l, m)
            for b in range(B):
                for ti, t in enumerate(spins_out):
                    for co in range(Co):
                        acc = 0j
                        if abs(t) <= l:
                            for si, s in enumerate(spins_in):
                                if abs(s) <= l:
                                    for c in range(C):
                                        acc += K[l, ti, co, si, c] * a[r, b, si, c]
                        assert abs(out[r, b, ti, co] - acc) < 1e-14


def test_spin_raising_filter_gives_eth():
    """K_l = sqrt(l(l+1)) from spin 0 to spin 1 maps f to eth f; compare
    with central differences of the field evaluated off the grid."""
    H, L = 16, 8
    rng = np.random.default_rng(13)
    a = syn.random_coefficients(rng, L, 1, (0,), 1)
    x = O.inverse(a, H, H, (0,))
    K = np.zeros((L, 1, 1, 1, 1), complex)
    K[:, 0, 0, 0, 0] = np.sqrt(np.arange(L) * (np.arange(L) + 1.0))
    y = O.conv(x, K, L, (0,), (1,))[0, 0, 0]
    th, ph = O.grid(H, H)
    TH, PH = np.meshgrid(th, ph, indexing="ij")
    f = lambda t, p: O.evaluate(a, (0,), t, p)[0, 0, 0]
    h = 1e-5
    dth = (f(TH + h, PH) - f(TH - h, PH)) / (2 * h)
    dph = (f(TH, PH + h) - f(TH, PH - h)) / (2 * h)
    eth = -(dth + 1j * dph / np.sin(TH))
    np.testing.assert_allclose(y, eth, atol=5e-8 * np.abs(eth).max())


@pytest.mark.parametrize("H", [8, 12])
def test_brute_force_so3_convolution(H):
    """Eq. (1) with a zonal filter k(x) = k_z(nu . x), nu the north pole:
    (f*k)(x) = int_SO(3) f(g nu) k(g^-1 x) dg = 2 pi int_S2 f(y) k_z(x . y) dy
    (Haar measure of total mass 8 pi^2).  With k_z(t) = sum_l kh_l N_l P_l(t),
    Funk--Hecke gives the layer with K_l = 2 pi sqrt(4 pi/(2l+1)) kh_l."""
    L = H // 2
    rng = np.random.default_rng(14)
    a = syn.random_coefficients(rng, L, 1, (0,), 1)
    x = O.inverse(a, H, H, (0,))
    kh = syn.complex_normal(rng, (L,))
    K = np.zeros((L, 1, 1, 1, 1), complex)
    K[:, 0, 0, 0, 0] = 2 * np.pi * np.sqrt(4 * np.pi / (2 * np.arange(L) + 1)) * kh
    y = O.conv(x, K, L, (0,), (0,))[0, 0, 0]

    # brute force, integrating over y with Gauss--Legendre x uniform phi
    t, wq = legendre.leggauss(2 * L)
    nphi = 2 * L + 1
    phq = 2 * np.pi * np.arange(nphi) / nphi
    THq, PHq = np.meshgrid(np.arccos(t), phq, indexing="ij")
    fq = O.evaluate(a, (0,), THq, PHq)[0, 0, 0]
    wts = wq[:, None] * (2 * np.pi / nphi)
    uq = np.stack([np.sin(THq) * np.cos(PHq), np.sin(THq) * np.sin(PHq), np.cos(THq)], -1)
    th, ph = O.grid(H, H)
    TH, PH = np.meshgrid(th, ph, indexing="ij")
    ux = np.stack([np.sin(TH) * np.cos(PH), np.sin(TH) * np.sin(PH), np.cos(TH)], -1)
    coeffs = kh * np.sqrt((2 * np.arange(L) + 1) / (4 * np.pi))
    brute = np.zeros((H, H), complex)
    for j in range(H):
        for k in range(H):
            dots = np.clip((uq * ux[j, k]).sum(-1), -1, 1)
            kz = legendre.legval(dots, coeffs)
            brute[j, k] = 2 * np.pi * (wts * fq * kz).sum()
    np.testing.assert_allclose(y, brute, atol=1e-12 * np.abs(brute).max())


# ----------------------------- phase collapse -----------------------------

def _pc_case(rng, B=2, spins=(0, 1), C=3, H=4, W=4):
    x = syn.complex_normal(rng, (B, len(spins), C, H, W))
    W1, W2, b = syn.phase_collapse_parameters(rng, len(spins), C)
    return x, W1, W2, b


def test_phase_collapse_leaves_other_spins_bit_identical():
    rng = np.random.default_rng(20)
    x, W1, W2, b = _pc_case(rng, spins=(1, 0, 2))
    y = O.phase_collapse(x, (1, 0, 2), W1, W2, b)
    assert np.array_equal(y[:, 0], x[:, 0]) and np.array_equal(y[:, 2], x[:, 2])


def test_phase_collapse_selectors():
    rng = np.random.default_rng(21)
    spins, C = (0, 1), 3
    x, _, _, _ = _pc_case(rng, spins=spins, C=C)
    Z1 = np.zeros((C, C), complex)
    Z2 = np.zeros((C, 2 * C), complex)
    zb = np.zeros(C, complex)
    # W1 = I: identity on spin 0
    np.testing.assert_array_equal(O.phase_collapse(x, spins, np.eye(C), Z2, zb), x)
    # W2 selects |x| of (spin 1, channel 2) into output channel 0 (stack order: spin, channel)
    W2 = Z2.copy()
    W2[0, 1 * C + 2] = 1.0
    y = O.phase_collapse(x, spins, Z1, W2, zb)
    np.testing.assert_allclose(y[:, 0, 0], np.abs(x[:, 1, 2]), atol=0)
    assert np.all(y[:, 0, 1:] == 0)
    # W1 row/column orientation: out channel 2 <- in channel 0 times 2i
    W1 = Z1.copy()
    W1[2, 0] = 2j
    y = O.phase_collapse(x, spins, W1, Z2, zb)
    np.testing.assert_allclose(y[:, 0, 2], 2j * x[:, 0, 0], atol=0)
    # bias only
    b = np.array([1 + 1j, -2.0, 0.5j])
    y = O.phase_collapse(x, spins, Z1, Z2, b)
    np.testing.assert_allclose(y[:, 0], np.broadcast_to(b[None, :, None, None], y[:, 0].shape))


def test_phase_collapse_modulus_ignores_spin_phase():
    # a rotation about the pole multiplies spin-s features by a phase; the
    # modulus term must not see it
    rng = np.random.default_rng(22)
    spins = (0, 1)
    x, W1, W2, b = _pc_case(rng, spins=spins)
    x2 = x.copy()
    x2[:, 1] *= np.exp(0.7j)
    y1 = O.phase_collapse(x, spins, W1, W2, b)
    y2 = O.phase_collapse(x2, spins, W1, W2, b)
    np.testing.assert_allclose(y1[:, 0], y2[:, 0], atol=1e-14)


# ------------------------------ bump synthesis -----------------------------

def test_bump_projection_matches_direct_evaluation():
    rng = np.random.default_rng(30)
    (cent, amps), = syn.bump_parameters(rng, 1, 1, 2, max_bumps=5)
    L, width = 30, 0.3
    a = O.bump_coefficients(cent, amps[:, 0, :], width, L)        # [L^2, C]
    th = np.linspace(0.2, 2.9, 6)
    ph = np.linspace(0.1, 6.0, 6)
    TH, PH = np.meshgrid(th, ph, indexing="ij")
    ux = np.stack([np.sin(TH) * np.cos(PH), np.sin(TH) * np.sin(PH), np.cos(TH)], -1)
    psi = np.arccos(np.clip(ux @ cent.T, -1, 1))                 # [6, 6, n]
    direct = np.exp(-psi ** 2 / (2 * width ** 2)) @ amps[:, 0, :]
    got = O.evaluate(a[:, None, None, :], (0,), TH, PH)[0, 0]     # [C, 6, 6]
    np.testing.assert_allclose(np.moveaxis(got, 0, -1), direct, atol=1e-10)


def test_bump_spin_raise_is_eth():
    rng = np.random.default_rng(31)
    (cent, amps), = syn.bump_parameters(rng, 1, 1, 1, max_bumps=3)
    L, width = 30, 0.3
    a0 = O.bump_coefficients(cent, amps[:, 0, :], width, L)
    a1 = O.bump_coefficients(cent, amps[:, 0, :], width, L, spin_raise=True)
    th = np.linspace(0.4, 2.7, 5)
    ph = np.linspace(0.1, 6.0, 5)
    TH, PH = np.meshgrid(th, ph, indexing="ij")
    f = lambda t, p: O.evaluate(a0[:, None, None, :], (0,), t, p)[0, 0, 0]
    h = 1e-5
    eth = -((f(TH + h, PH) - f(TH - h, PH)) / (2 * h)
            + 1j * (f(TH, PH + h) - f(TH, PH - h)) / (2 * h) / np.sin(TH))
    got = O.evaluate(a1[:, None, None, :], (1,), TH, PH)[0, 0, 0]
    np.testing.assert_allclose(got, eth, atol=1e-7 * np.abs(eth).max())
