"""Pins of the oracle's backward pass (adjoints and gradients), CPU only.

The backward pass is fixed by the mathematics rather than by the paper: for a
real loss with output gradient g (dL = Re <g, dy>), the input gradient of a
linear map A is A^H g.  Each adjoint is checked against its forward map
through <A x, y> = <x, A^H y> on random data, the gradients against finite
differences of the loss, and the filter gradient against an explicit loop.
"""

import numpy as np
import pytest

import oracle as O
from paper_2306_05420_amd import synthetic as syn



def _cn(rng, shape):
    return syn.complex_normal(rng, shape)


def _vdot(u, v):
    return np.vdot(np.ravel(u), np.ravel(v))   # sum conj(u) v


def _rel(a, b):
    return abs(a - b) / max(abs(a), abs(b))


CASES = [  # H, L, spins_in, spins_out, B, C_in, C_out
    (8, 4, (0,), (0, 1), 2, 3, 2),
    (12, 6, (1, -2), (0, 2), 1, 2, 3),   # non-power-of-two grid, |s| = 2
    (16, 5, (0, 1), (1,), 2, 2, 2),      # L < H/2
]


@pytest.mark.parametrize("case", CASES)
def test_forward_adjoint_identity(case):
    H, L, si, so, B, Ci, Co = case
    rng = np.random.default_rng(1)
    x = _cn(rng, (B, len(si), Ci, H, H))       # not band-limited: the operator itself
    a = syn.random_coefficients(rng, L, B, si, Ci, 0.0)
    lhs = _vdot(O.forward(x, L, si), a)
    rhs = _vdot(x, O.forward_adjoint(a, H, H, si))
    assert _rel(lhs, rhs) < 1e-12


@pytest.mark.parametrize("case", CASES)
def test_inverse_adjoint_identity(case):
    H, L, si, so, B, Ci, Co = case
    rng = np.random.default_rng(2)
    a = syn.random_coefficients(rng, L, B, so, Co, 0.0)
    y = _cn(rng, (B, len(so), Co, H, H))
    lhs = _vdot(O.inverse(a, H, H, so), y)
    rhs = _vdot(a, O.inverse_adjoint(y, L, so))
    assert _rel(lhs, rhs) < 1e-12


@pytest.mark.parametrize("case", CASES)
def test_mix_adjoint_identity(case):
    H, L, si, so, B, Ci, Co = case
    rng = np.random.default_rng(3)
    a = syn.random_coefficients(rng, L, B, si, Ci, 0.0)
    g = syn.random_coefficients(rng, L, B, so, Co, 0.0)
    K = _cn(rng, (L, len(so), Co, len(si), Ci))
    lhs = _vdot(O.mix(a, K, si, so), g)
    rhs = _vdot(a, O.mix_adjoint(g, K, si, so))
    assert _rel(lhs, rhs) < 1e-12


def test_inverse_adjoint_is_unweighted_analysis():
    """On a band-limited field, G^H y = F(y / q) must give back
    sum_{jk} conj(Y) y: for y = one harmonic sY_lm that is the discrete
    inner product of sY_lm with itself and the other harmonics; check it
    against a direct double sum with spin_harmonic."""
    H, L, s = 8, 4, 1
    theta, phi = O.grid(H, H)
    TH, PH = np.meshgrid(theta, phi, indexing="ij")
    y = O.spin_harmonic(s, 2, -1, TH, PH)[None, None, None]
    got = O.inverse_adjoint(y, L, (s,))
    for l in range(abs(s), L):
        for m in range(-l, l + 1):
            ref = np.sum(np.conj(O.spin_harmonic(s, l, m, TH, PH)) * y[0, 0, 0])
            assert abs(got[O.coef_index(l, m), 0, 0, 0] - ref) < 1e-12


def test_filter_grad_explicit_loop():
    L, B, si, so, Ci, Co = 4, 2, (0, 1), (1, 0), 2, 3
    rng = np.random.default_rng(4)
    g = syn.random_coefficients(rng, L, B, so, Co, 0.0)
    a = syn.random_coefficients(rng, L, B, si, Ci, 0.0)
    got = O.filter_grad(g, a, si, so)
    ref = np.zeros_like(got)
    for l in range(L):
        for ti, t in enumerate(so):
            for si_, s in enumerate(si):
                if abs(t) > l or abs(s) > l:
                    continue
                for m in range(-l, l + 1):
                    r = O.coef_index(l, m)
                    for b in range(B):
                        for co in range(Co):
                            for c in range(Ci):
                                ref[l, ti, co, si_, c] += g[r, b, ti, co] * np.conj(a[r, b, si_, c])
    assert np.allclose(got, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("case", CASES[:2])
def test_conv_backward_finite_differences(case):
    """L(x, K) = Re <g, conv(x, K)>: the directional derivatives along random
    dx and dK equal Re <grad_x, dx> and Re <grad_K, dK> (central differences;
    the loss is linear in each argument, so they are exact up to rounding)."""
    H, L, si, so, B, Ci, Co = case
    rng = np.random.default_rng(5)
    x = _cn(rng, (B, len(si), Ci, H, H))
    K = _cn(rng, (L, len(so), Co, len(si), Ci))
    g = _cn(rng, (B, len(so), Co, H, H))
    dx = _cn(rng, x.shape)
    dK = _cn(rng, K.shape)

    def loss(x_, K_):
        return np.real(_vdot(g, O.conv(x_, K_, L, si, so)))

    gx, gK = O.conv_backward(x, K, g, L, si, so)
    h = 1e-3
    fd_x = (loss(x + h * dx, K) - loss(x - h * dx, K)) / (2 * h)
    fd_K = (loss(x, K + h * dK) - loss(x, K - h * dK)) / (2 * h)
    assert _rel(fd_x, np.real(_vdot(gx, dx))) < 1e-9
    assert _rel(fd_K, np.real(_vdot(gK, dK))) < 1e-9
    # filter entries whose spins do not exist at a degree get no gradient
    for l in range(L):
        for ti, t in enumerate(so):
            for s_i, s in enumerate(si):
                if abs(t) > l or abs(s) > l:
                    assert np.all(gK[l, ti, :, s_i] == 0)
