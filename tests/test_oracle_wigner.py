"""Pins of the oracle's Wigner-d recursion and spin-weighted harmonics.

Independent facts used: the textbook sum in exact rational arithmetic (at a
rotation angle with rational half-angle cosine and sine), the stored exact
values in tests/golden/wigner_d_exact.txt, scipy's spherical harmonics at
spin 0, orthogonality and symmetries of d^l, closed forms of low-degree spin
harmonics, spin raising by finite differences, and the paper's Wigner-Delta
identities behind eqs. (4) and (6)."""

import math
import os
from fractions import Fraction

import numpy as np
import pytest
import scipy.special as sp

import oracle as O

HERE = os.path.dirname(os.path.abspath(__file__))
BETA_345 = 2.0 * math.atan2(4.0, 3.0)      # cos(beta/2) = 3/5, sin(beta/2) = 4/5


def test_recursion_matches_exact_sum():
    worst = 0.0
    for l in range(0, 31):
        for m in range(-l, l + 1, max(1, l // 6)):
            for n in (-l, -2, -1, 0, 1, 2, l):
                if abs(n) > l:
                    continue
                d = O.wigner_d(l + 1, m, n, [BETA_345])[l, 0]
                e = O.wigner_d_sum_exact(l, m, n, Fraction(3, 5), Fraction(4, 5))
                worst = max(worst, abs(d - e))
    assert worst < 1e-13


def test_recursion_matches_golden_file():
    path = os.path.join(HERE, "golden", "wigner_d_exact.txt")
    rows = [ln.split() for ln in open(path) if ln.strip() and not ln.startswith("#")]
    assert len(rows) > 50
    for l, m, n, val in rows:
        l, m, n, val = int(l), int(m), int(n), float(val)
        d = O.wigner_d(l + 1, m, n, [BETA_345])[l, 0]
        assert abs(d - val) < 1e-13, (l, m, n)


def test_d1_sign_convention():
    b = np.linspace(0.1, 3.0, 5)
    np.testing.assert_allclose(O.wigner_d(2, 1, 0, b)[1], -np.sin(b) / math.sqrt(2), atol=1e-15)
    np.testing.assert_allclose(O.wigner_d(2, 1, 1, b)[1], (1 + np.cos(b)) / 2, atol=1e-15)
    np.testing.assert_allclose(O.wigner_d(2, 1, -1, b)[1], (1 - np.cos(b)) / 2, atol=1e-15)


def _dmatrix(l, beta):
    D = np.zeros((2 * l + 1, 2 * l + 1))
    for m in range(-l, l + 1):
        for n in range(-l, l + 1):
            D[m + l, n + l] = O.wigner_d(l + 1, m, n, [beta])[l, 0]
    return D


@pytest.mark.parametrize("l", [0, 1, 5, 17, 40])
def test_orthogonality(l):
    D = _dmatrix(l, 1.234)
    np.testing.assert_allclose(D @ D.T, np.eye(2 * l + 1), atol=5e-14)


@pytest.mark.parametrize("l", [3, 9])
def test_symmetries_and_identity(l):
    b = 0.77
    D = _dmatrix(l, b)
    idx = np.arange(-l, l + 1)
    sign = (-1.0) ** (idx[:, None] - idx[None, :])
    np.testing.assert_allclose(D, sign * D.T, atol=1e-14)          # d_mn = (-1)^(m-n) d_nm
    np.testing.assert_allclose(D, D[::-1, ::-1].T, atol=1e-14)      # d_mn = d_{-n,-m}
    np.testing.assert_allclose(_dmatrix(l, 0.0), np.eye(2 * l + 1), atol=1e-15)
    # d_mn(pi - b) = (-1)^(l+m) d_{m,-n}(b)
    Dp = _dmatrix(l, math.pi - b)
    np.testing.assert_allclose(Dp, ((-1.0) ** (l + idx))[:, None] * D[:, ::-1], atol=1e-13)


def test_spin0_matches_scipy():
    th = np.linspace(0.05, 3.1, 11)
    ph = np.linspace(-3.0, 6.0, 11)
    for l in range(0, 13):
        for m in range(-l, l + 1):
            np.testing.assert_allclose(O.spin_harmonic(0, l, m, th, ph),
                                       sp.sph_harm_y(l, m, th, ph), atol=1e-13)


def test_low_degree_closed_forms():
    th = np.linspace(0.05, 3.1, 9)
    ph = np.linspace(-1.0, 5.0, 9)
    pi = math.pi
    Y = O.spin_harmonic
    c = np.cos(th)
    s = np.sin(th)
    e = np.exp(1j * ph)
    np.testing.assert_allclose(Y(0, 0, 0, th, ph), 1 / math.sqrt(4 * pi) + 0 * th, atol=1e-15)
    np.testing.assert_allclose(Y(0, 1, 0, th, ph), math.sqrt(3 / (4 * pi)) * c, atol=1e-15)
    np.testing.assert_allclose(Y(0, 1, 1, th, ph), -math.sqrt(3 / (8 * pi)) * s * e, atol=1e-15)
    np.testing.assert_allclose(Y(0, 1, -1, th, ph), math.sqrt(3 / (8 * pi)) * s / e, atol=1e-15)
    np.testing.assert_allclose(Y(0, 2, 0, th, ph), math.sqrt(5 / (16 * pi)) * (3 * c * c - 1),
                               atol=1e-15)
    # spin 1 (Goldberg et al. / Huffenberger--Wandelt convention)
    np.testing.assert_allclose(Y(1, 1, 0, th, ph), math.sqrt(3 / (8 * pi)) * s, atol=1e-15)
    np.testing.assert_allclose(Y(1, 1, 1, th, ph), -math.sqrt(3 / (16 * pi)) * (1 - c) * e,
                               atol=1e-15)
    np.testing.assert_allclose(Y(1, 1, -1, th, ph), -math.sqrt(3 / (16 * pi)) * (1 + c) / e,
                               atol=1e-15)
    # spin >= l+1 does not exist
    assert np.all(Y(2, 1, 0, th, ph) == 0)


def _eth(fun, s, th, ph, h=1e-5):
    """eth eta = -(sin th)^s (d_th + i csc th d_ph) [(sin th)^-s eta], by
    central differences."""
    g = lambda t, p: np.sin(t) ** (-s) * fun(t, p)
    dth = (g(th + h, ph) - g(th - h, ph)) / (2 * h)
    dph = (g(th, ph + h) - g(th, ph - h)) / (2 * h)
    return -np.sin(th) ** s * (dth + 1j * dph / np.sin(th))


@pytest.mark.parametrize("s", [-1, 0, 1])
def test_spin_raising(s):
    th = np.linspace(0.3, 2.8, 7)
    ph = np.linspace(0.2, 5.0, 7)
    for l in range(max(abs(s), abs(s + 1)), 6):
        for m in range(-l, l + 1):
            lhs = _eth(lambda t, p: O.spin_harmonic(s, l, m, t, p), s, th, ph)
            rhs = math.sqrt((l - s) * (l + s + 1)) * O.spin_harmonic(s + 1, l, m, th, ph)
            np.testing.assert_allclose(lhs, rhs, atol=2e-8)


@pytest.mark.parametrize("s", [0, 1, -1, 2])
def test_paper_delta_identities(s):
    """Eq. (4) expresses conj(sY_lm) on the torus through
    (-1)^s i^(m+s) N_l sum_m' Delta_m'm Delta_m'(-s) e^{-i m' theta} e^{-i m phi};
    eq. (6) expresses sY_lm through
    (-1)^s i^(m+s) N_l sum_m' Delta_(-m')(-s) Delta_(-m')m e^{i m' theta} e^{i m phi}.
    Both must reproduce the oracle's harmonics, with Delta = d(pi/2)."""
    th = np.linspace(0.1, 3.0, 6)
    ph = np.linspace(0.3, 4.0, 6)
    for l in range(abs(s), 9):
        N = math.sqrt((2 * l + 1) / (4 * math.pi))
        D = _dmatrix(l, math.pi / 2)               # D[m'+l, m+l] = Delta_m'm
        for m in range(-l, l + 1):
            mp = np.arange(-l, l + 1)
            coef4 = D[mp + l, m + l] * D[mp + l, -s + l]
            conjY = ((-1.0) ** s) * (1j ** (m + s)) * N * (
                coef4[None, :] * np.exp(-1j * np.outer(th, mp))).sum(1) * np.exp(-1j * m * ph)
            np.testing.assert_allclose(conjY, np.conj(O.spin_harmonic(s, l, m, th, ph)),
                                       atol=1e-13)
            coef6 = D[-mp + l, -s + l] * D[-mp + l, m + l]
            Y = ((-1.0) ** s) * (1j ** (m + s)) * N * (
                coef6[None, :] * np.exp(1j * np.outer(th, mp))).sum(1) * np.exp(1j * m * ph)
            np.testing.assert_allclose(Y, O.spin_harmonic(s, l, m, th, ph), atol=1e-13)


def test_conjugation_symmetry():
    # conj(sY_lm) = (-1)^(m+s) (-s)Y_l(-m)
    th = np.linspace(0.1, 3.0, 5)
    ph = np.linspace(0.3, 4.0, 5)
    for s in (-1, 0, 1, 2):
        for l in range(abs(s), 6):
            for m in range(-l, l + 1):
                np.testing.assert_allclose(
                    np.conj(O.spin_harmonic(s, l, m, th, ph)),
                    (-1.0) ** (m + s) * O.spin_harmonic(-s, l, -m, th, ph), atol=1e-14)


def test_large_degree_stays_orthonormal_on_grid():
    # l up to 127 near the poles (seeds underflow gracefully)
    H = 256
    th, _ = O.grid(H, H)
    w = O.dh_weights(H)
    for m, n in [(0, 0), (5, -1), (100, 0), (127, -1), (-64, 1)]:
        d = O.wigner_d(128, m, n, th)
        G = (d * w) @ d.T
        lo = max(abs(m), abs(n))
        idx = np.arange(lo, 128)
        # int_0^pi d^l d^l' sin = 2/(2l+1) delta
        np.testing.assert_allclose(G[np.ix_(idx, idx)], np.diag(2.0 / (2 * idx + 1.0)),
                                   atol=1e-13)
        assert np.all(np.isfinite(d))
