"""Pins of the oracle's grid and Driscoll--Healy weights against facts that do
not depend on the oracle: Fejer's first-rule closed form, exact integrals of
powers of cos(theta), Legendre orthogonality, a hand-computed case."""

import math

import numpy as np
import pytest
from numpy.polynomial import legendre

import oracle as O


@pytest.mark.parametrize("H", [2, 4, 8, 16, 32, 64])
def test_weights_sum_to_two(H):
    # int_0^pi sin(theta) dtheta = 2
    assert abs(O.dh_weights(H).sum() - 2.0) < 1e-14


def test_weights_h2_by_hand():
    # H = 2: theta = pi/4, 3pi/4; w = 2 sin^2(theta) = 1 each
    np.testing.assert_allclose(O.dh_weights(2), [1.0, 1.0], rtol=0, atol=1e-15)


@pytest.mark.parametrize("H", [4, 8, 16, 32])
def test_weights_equal_fejer_first_rule(H):
    # Fejer's first rule on the Chebyshev points x_j = cos(theta_j):
    # w_j = (2/H) [1 - 2 sum_{k=1}^{H/2} cos(2 k theta_j) / (4k^2 - 1)]
    theta, _ = O.grid(H, H)
    k = np.arange(1, H // 2 + 1)
    fej = (2.0 / H) * (1 - 2 * (np.cos(2 * np.outer(theta, k)) / (4 * k * k - 1)).sum(1))
    np.testing.assert_allclose(O.dh_weights(H), fej, rtol=0, atol=1e-15)


@pytest.mark.parametrize("H", [8, 16, 32])
def test_weights_exact_for_cos_powers(H):
    theta, _ = O.grid(H, H)
    w = O.dh_weights(H)
    for q in range(H):
        exact = (1 + (-1) ** q) / (q + 1.0)
        assert abs((w * np.cos(theta) ** q).sum() - exact) < 1e-13, q
    # and not exact at degree H: the Chebyshev polynomial T_H(cos theta) =
    # cos(H theta) vanishes at every node but integrates to 2/(1-H^2)
    assert abs((w * np.cos(H * theta)).sum()) < 1e-14
    assert abs(2.0 / (1.0 - H * H)) > 1e-4


@pytest.mark.parametrize("H", [8, 16])
def test_legendre_orthogonality(H):
    theta, _ = O.grid(H, H)
    w = O.dh_weights(H)
    x = np.cos(theta)
    for l in range(1, H):
        assert abs((w * legendre.legval(x, [0] * l + [1])).sum()) < 1e-14


def test_grid_points():
    th, ph = O.grid(4, 8)
    np.testing.assert_allclose(th, [math.pi / 8, 3 * math.pi / 8, 5 * math.pi / 8,
                                    7 * math.pi / 8])
    np.testing.assert_allclose(ph, np.arange(8) * math.pi / 4)


def test_odd_H_rejected():
    with pytest.raises(ValueError):
        O.dh_weights(5)
