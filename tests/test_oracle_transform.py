"""Pins of the oracle's forward / inverse transforms (eqs. (2)-(3)).

Independent facts: the unseparated double sum, orthonormality of the
harmonics under the quadrature, the round trips, Parseval against a
Gauss--Legendre quadrature that does not use the Driscoll--Healy weights,
the mean, exact phase shifts under longitude rotation, and the conjugation
symmetry between spins s and -s."""

import math

import numpy as np
import pytest
from numpy.polynomial import legendre

import oracle as O
from paper_2306_05420_amd import synthetic as syn


def _field(rng, L, H, spins, B=2, C=3, decay=0.0):
    a = syn.random_coefficients(rng, L, B, spins, C, decay)
    return a, O.inverse(a, H, H, spins)


@pytest.mark.parametrize("H,L,spins", [(8, 4, (0,)), (8, 4, (1, -1)), (12, 6, (0, 2)),
                                       (16, 8, (0, 1))])
def test_separable_equals_direct_double_sum(H, L, spins):
    rng = np.random.default_rng(1)
    # arbitrary (not band-limited) input: the operator itself must agree
    x = syn.complex_normal(rng, (2, len(spins), 2, H, H))
    np.testing.assert_allclose(O.forward(x, L, spins), O.forward_direct(x, L, spins),
                               atol=1e-13)


@pytest.mark.parametrize("s", [0, 1, -2])
def test_orthonormality_on_grid(s):
    H, L = 16, 8
    th, ph = O.grid(H, H)
    TH, PH = np.meshgrid(th, ph, indexing="ij")
    for l in range(abs(s), L):
        for m in range(-l, l + 1):
            Y = O.spin_harmonic(s, l, m, TH, PH)
            a = O.forward(Y[None, None, None], L, (s,))[:, 0, 0, 0]
            e = np.zeros(L * L, complex)
            e[O.coef_index(l, m)] = 1.0
            np.testing.assert_allclose(a, e, atol=2e-14)


@pytest.mark.parametrize("H,L,spins", [(16, 8, (0, 1)), (32, 16, (0, 1, -1)), (16, 6, (2,))])
def test_round_trips(H, L, spins):
    rng = np.random.default_rng(2)
    a, x = _field(rng, L, H, spins)
    np.testing.assert_allclose(O.forward(x, L, spins), a, atol=1e-13)
    np.testing.assert_allclose(O.inverse(O.forward(x, L, spins), H, H, spins), x, atol=1e-13)


def test_inverse_matches_pointwise_evaluation():
    rng = np.random.default_rng(3)
    spins = (0, 1)
    a = syn.random_coefficients(rng, 6, 1, spins, 2)
    th, ph = O.grid(12, 12)
    TH, PH = np.meshgrid(th, ph, indexing="ij")
    np.testing.assert_allclose(O.inverse(a, 12, 12, spins), O.evaluate(a, spins, TH, PH),
                               atol=1e-13)


def test_parseval_against_gauss_legendre():
    rng = np.random.default_rng(4)
    L, spins = 8, (0, 1)
    a = syn.random_coefficients(rng, L, 1, spins, 2)
    # integrate |f|^2 with Gauss--Legendre in cos(theta) x uniform phi
    t, wq = legendre.leggauss(24)
    nphi = 40
    phi = 2 * np.pi * np.arange(nphi) / nphi
    TH, PH = np.meshgrid(np.arccos(t), phi, indexing="ij")
    f = O.evaluate(a, spins, TH, PH)
    integral = (np.abs(f) ** 2 * wq[None, None, None, :, None]).sum(axis=(-1, -2)) * 2 * np.pi / nphi
    np.testing.assert_allclose(integral, (np.abs(a) ** 2).sum(0), rtol=1e-12)


def test_constant_field_gives_mean_coefficient():
    # 0f^0_0 = sqrt(4 pi) * mean (Method, spectral batch norm paragraph)
    H, L = 16, 8
    x = np.full((1, 1, 1, H, H), 0.7 - 0.2j)
    a = O.forward(x, L, (0,))[:, 0, 0, 0]
    assert abs(a[0] - math.sqrt(4 * math.pi) * (0.7 - 0.2j)) < 1e-14
    assert np.abs(a[1:]).max() < 1e-14


@pytest.mark.parametrize("r", [1, 3, 7])
def test_longitude_shift_is_exact_phase(r):
    H, L, spins = 16, 8, (0, 1)
    rng = np.random.default_rng(5)
    x = syn.complex_normal(rng, (1, 2, 2, H, H))     # need not be band-limited
    a = O.forward(x, L, spins)
    a_shift = O.forward(np.roll(x, r, axis=-1), L, spins)
    m = np.array([m for l in range(L) for m in range(-l, l + 1)])
    np.testing.assert_allclose(a_shift, a * np.exp(-2j * np.pi * m * r / H)[:, None, None, None],
                               atol=1e-13)


def test_conjugate_field_maps_spin_s_to_minus_s():
    # conj(sY_lm) = (-1)^(m+s) (-s)Y_l(-m)  =>  (-s)[conj f]_lm = (-1)^(m+s) conj(s f_l(-m))
    H, L = 16, 8
    rng = np.random.default_rng(6)
    for s in (1, 2):
        a, x = _field(rng, L, H, (s,), B=1, C=1)
        b = O.forward(np.conj(x), L, (-s,))
        for l in range(abs(s), L):
            for m in range(-l, l + 1):
                want = (-1) ** (m + s) * np.conj(a[O.coef_index(l, -m)])
                np.testing.assert_allclose(b[O.coef_index(l, m)], want, atol=1e-13)


def test_low_spin_rows_are_zero():
    H, L = 16, 8
    rng = np.random.default_rng(7)
    x = syn.complex_normal(rng, (1, 1, 1, H, H))
    a = O.forward(x, L, (2,))
    for l in range(2):
        for m in range(-l, l + 1):
            assert a[O.coef_index(l, m)].max() == 0
