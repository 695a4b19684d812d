"""Pins of the oracle's spectral batch norm, spectral pooling and residual
block (Method, "Spectral batch normalization", "Spectral pooling and
efficient residual block", Fig. 2), CPU only.

Spatial statistics are integrated on a Gauss--Legendre x uniform-longitude
grid from the direct sum of eq. (3) (`evaluate`), which shares nothing with
the batch norm's coefficient formula and is exact for band-limited fields.
"""

import numpy as np
import pytest

import oracle as O
from paper_2306_05420_amd import synthetic as syn


def _gl_grid(L):
    """Nodes and weights that integrate |f|^2 and f exactly for l < L:
    Gauss--Legendre in cos(theta) with L + 2 nodes, 2L + 2 longitudes."""
    t, wt = np.polynomial.legendre.leggauss(L + 2)
    n_phi = 2 * L + 2
    theta = np.arccos(t)
    phi = 2 * np.pi * np.arange(n_phi) / n_phi
    TH, PH = np.meshgrid(theta, phi, indexing="ij")
    wq = np.outer(wt, np.full(n_phi, 2 * np.pi / n_phi))   # sums to 4 pi
    return TH, PH, wq


def _spatial_mean_var(coef, spins):
    """Per (b, s, c) the spatial mean (1/4pi) int f of the spin-0 maps (0 for
    other spins: a spin-weighted field has no l = 0 part to remove), and per
    (s, c) the batch average of (1/4pi) int |f - mean|^2."""
    L = int(round(np.sqrt(coef.shape[0])))
    TH, PH, wq = _gl_grid(L)
    f = O.evaluate(coef, spins, TH, PH)                      # [B, S, C, n_t, n_p]
    mean = np.sum(f * wq, axis=(-2, -1)) / (4 * np.pi)       # [B, S, C]
    mean[:, [s != 0 for s in spins]] = 0.0
    dev = f - mean[..., None, None]
    var = np.mean(np.sum(np.abs(dev) ** 2 * wq, axis=(-2, -1)) / (4 * np.pi), axis=0)
    return mean, var


SPINS = [(0,), (0, 1), (1, -2, 0)]


@pytest.mark.parametrize("spins", SPINS)
def test_batch_norm_normalizes_the_function(spins):
    L, B, C = 6, 3, 2
    rng = np.random.default_rng(11)
    a = syn.random_coefficients(rng, L, B, spins, C, 0.5)
    a[0] += 3.0                                              # a large mean
    gamma = np.ones((len(spins), C))
    out, var = O.spectral_batch_norm(a, spins, gamma, eps=0.0)
    mean_in, var_in = _spatial_mean_var(a, spins)
    mean_out, var_out = _spatial_mean_var(out, spins)
    # the statistic is the spatial variance about each sample's own mean
    # (spin 0), the mean square of the field (other spins)
    assert np.allclose(var, var_in, rtol=1e-12)
    assert np.allclose(mean_out, 0, atol=1e-12)
    assert np.allclose(var_out, 1.0, rtol=1e-12)


def test_batch_norm_affine_bias_skip_and_given_variance():
    L, B, C = 5, 2, 3
    spins = (0, 1)
    rng = np.random.default_rng(12)
    a = syn.random_coefficients(rng, L, B, spins, C, 0.0)
    gamma = rng.uniform(0.5, 2.0, size=(2, C))
    beta = syn.complex_normal(rng, (C,))
    out, var = O.spectral_batch_norm(a, spins, gamma, beta, eps=0.0)
    mean_out, var_out = _spatial_mean_var(out, spins)
    # the bias sets the spin-0 coefficient l = 0: mean beta Y_00 = beta / sqrt(4 pi)
    assert np.allclose(mean_out[:, 0], beta[None, :] / np.sqrt(4 * np.pi), rtol=1e-12)
    assert np.allclose(var_out, gamma ** 2, rtol=1e-12)
    # given variance (inference): used as is; eps adds under the root
    v = rng.uniform(0.5, 3.0, size=(2, C))
    out2, v2 = O.spectral_batch_norm(a, spins, gamma, None, eps=0.25, var=v)
    assert np.array_equal(v2, v)
    assert np.allclose(out2[1:], a[1:] * (gamma / np.sqrt(v + 0.25))[None, None], rtol=1e-14)
    assert np.all(out2[0] == 0)
    # skip is added after the normalization
    skip = syn.complex_normal(rng, a.shape)
    out3, _ = O.spectral_batch_norm(a, spins, gamma, beta, eps=0.0, skip=skip)
    assert np.allclose(out3, out + skip, rtol=1e-14, atol=1e-14)
    # rows that do not exist for spin 1 stay zero
    assert np.all(out[:1, :, 1] == 0)


def _identity_filters(L, S, C):
    K = np.zeros((L, S, C, S, C), dtype=np.complex128)
    for s in range(S):
        K[:, s, :, s, :] = np.eye(C)[None]
    return K


def _identity_pc(S, C):
    return (np.eye(C, dtype=np.complex128), np.zeros((C, S * C), dtype=np.complex128),
            np.zeros(C, dtype=np.complex128))


def _block_params(rng, L, S, C):
    K1 = syn.random_filters(rng, L, range(S), C, range(S), C, 1.0 / (S * C))
    K2 = syn.random_filters(rng, L, range(S), C, range(S), C, 1.0 / (S * C))
    bn1 = (rng.uniform(0.5, 1.5, size=(S, C)), syn.complex_normal(rng, (C,)))
    bn2 = (rng.uniform(0.5, 1.5, size=(S, C)), syn.complex_normal(rng, (C,)))
    pc1 = syn.phase_collapse_parameters(rng, S, C)
    pc2 = syn.phase_collapse_parameters(rng, S, C)
    return K1, K2, bn1, bn2, pc1, pc2


@pytest.mark.parametrize("pool", [False, True])
def test_block_without_second_branch_is_the_phase_collapse_of_its_input(pool):
    """K2 = 0 and no bias: the block returns sigma2 of the input itself on the
    output grid (the skip coefficients are the input's)."""
    L, B, C, spins = 4, 2, 2, (0, 1)
    H_out = 2 * L
    H_in = 2 * H_out if pool else H_out
    rng = np.random.default_rng(13)
    a = syn.random_coefficients(rng, L, B, spins, C, 0.0)
    x = O.inverse(a, H_in, H_in, spins)
    K1, K2, bn1, bn2, pc1, pc2 = _block_params(rng, L, len(spins), C)
    K2 = np.zeros_like(K2)
    bn2 = (bn2[0], None)
    y = O.residual_block(x, L, H_out, spins, K1, K2, bn1, bn2, pc1, pc2)
    th, ph = O.grid(H_out, H_out)
    TH, PH = np.meshgrid(th, ph, indexing="ij")
    x_out = O.evaluate(a, spins, TH, PH)                     # the input on the output grid
    assert np.allclose(y, O.phase_collapse(x_out, spins, *pc2), rtol=1e-10, atol=1e-10)


def test_block_with_identity_parameters():
    """Identity filters and activations, unit scale, no bias, eps = 0:
    y = x + (x - mean) / std with the per-sample spatial mean (spin-0 maps
    only) and the batch-averaged spatial standard deviation about it, both
    integrated independently of the transform."""
    L, B, C, spins = 5, 3, 2, (0, 1)
    H = 2 * L
    rng = np.random.default_rng(14)
    a = syn.random_coefficients(rng, L, B, spins, C, 0.0)
    a[0] += 2.0
    x = O.inverse(a, H, H, spins)
    S = len(spins)
    K = _identity_filters(L, S, C)
    bn = (np.ones((S, C)), None)
    pc = _identity_pc(S, C)
    y = O.residual_block(x, L, H, spins, K, K, bn, bn, pc, pc, eps=0.0)
    mean, var = _spatial_mean_var(a, spins)
    ref = x + (x - mean[..., None, None]) / np.sqrt(var)[None, :, :, None, None]
    assert np.allclose(y, ref, rtol=1e-10, atol=1e-10)


@pytest.mark.parametrize("pool", [False, True])
def test_block_longitude_shift_equivariance(pool):
    L, B, C, spins = 4, 2, 2, (0, 1)
    H_out = 2 * L
    H_in = 2 * H_out if pool else H_out
    rng = np.random.default_rng(15)
    x = syn.complex_normal(rng, (B, len(spins), C, H_in, H_in))   # not band-limited
    params = _block_params(rng, L, len(spins), C)
    y = O.residual_block(x, L, H_out, spins, *params)
    r = 2 if pool else 3
    y_shift = O.residual_block(np.roll(x, r, axis=-1), L, H_out, spins, *params)
    assert np.allclose(y_shift, np.roll(y, r * H_out // H_in, axis=-1), rtol=1e-10, atol=1e-10)
