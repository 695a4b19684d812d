"""Pins of the oracle's Wigner-Delta route (eqs. (4)-(6) and the J / G
symmetries), CPU only: both variants reproduce the direct-quadrature
transforms exactly (the Delta identity holds at every colatitude, so the
equality holds for any input, band-limited or not)."""

import numpy as np
import pytest

import oracle as O
from paper_2306_05420_amd import synthetic as syn

CASES = [  # H, L, spins
    (8, 4, (0,)),
    (12, 5, (0, 1, -2)),       # L < H/2, |s| = 2
    (16, 8, (1, -1)),
]


@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("symmetric", [False, True])
def test_forward_delta_equals_direct_quadrature(case, symmetric):
    H, L, spins = case
    rng = np.random.default_rng(H + L)
    x = syn.complex_normal(rng, (2, len(spins), 2, H, H))          # not band-limited
    a = O.forward(x, L, spins)
    b = O.forward_delta(x, L, spins, symmetric)
    assert np.allclose(b, a, rtol=1e-12, atol=1e-12 * np.abs(a).max())


@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("symmetric", [False, True])
def test_inverse_delta_equals_synthesis(case, symmetric):
    H, L, spins = case
    rng = np.random.default_rng(H * L)
    c = syn.random_coefficients(rng, L, 2, spins, 2, 0.0)
    y = O.inverse(c, H, H, spins)
    z = O.inverse_delta(c, H, H, spins, symmetric)
    assert np.allclose(z, y, rtol=1e-12, atol=1e-12 * np.abs(y).max())


def test_delta_matrix_orthogonal_and_symmetric():
    """Delta^l is orthogonal, and the product of eq. (5) obeys
    Delta_{-m'm} Delta_{-m'(-s)} = (-1)^(m+s) Delta_{m'm} Delta_{m'(-s)}."""
    L = 9
    D = O.delta_matrix(L)
    for l in range(L):
        idx = np.arange(L - 1 - l, L + l)
        Dl = D[l][np.ix_(idx, idx)]
        assert np.allclose(Dl.T @ Dl, np.eye(2 * l + 1), atol=1e-13)
        for s in range(-min(l, 2), min(l, 2) + 1):
            for m in range(-l, l + 1):
                for mp in range(0, l + 1):
                    lhs = D[l, L - 1 - mp, L - 1 + m] * D[l, L - 1 - mp, L - 1 - s]
                    rhs = (-1.0) ** (m + s) * D[l, L - 1 + mp, L - 1 + m] * D[l, L - 1 + mp, L - 1 - s]
                    assert abs(lhs - rhs) < 1e-13
