"""Plain float64 oracle of the spectral spin-weighted spherical convolution layer.

TEST INFRASTRUCTURE ONLY (see the package docstring): slow, obviously correct
numpy code that the GPU library is compared against.  Nothing here is tuned.

What it computes (Esteves, Slotine, Makadia, "Scaling Spherical CNNs",
ICML 2023):

* the forward spin-weighted spherical Fourier transform, eq. (2) of the
  Background section, evaluated by Driscoll--Healy quadrature on the
  equiangular grid (the paper's "Computing generalized convolutions"
  paragraph cites Driscoll--Healy and Kostelec--Rockmore for it);
* the inverse transform, eq. (3);
* the convolution as per-degree products of coefficients with filters shared
  across the order m ("Spherical CNNs" paragraph: spin-weighted convolutions
  are products of spin-weighted harmonic coefficients; Fig. 2's "*K");
* the phase-collapse nonlinearity (Method, "Phase collapse nonlinearity");
* the backward pass of the layer (adjoints of the linear maps above);
* the transforms by the paper's Wigner-Delta route, eqs. (4)-(6), with and
  without the J / G symmetries;
* spectral batch normalization, spectral pooling and the residual block with
  its skip connection between Fourier coefficients (Method, "Spectral batch
  normalization", "Spectral pooling and efficient residual block", Fig. 2);
* the Funk--Hecke projection of isotropic bumps used to synthesise the
  molecule-shaped inputs.

Conventions (the paper fixes them only through eqs. (4) and (6)):

* grid: theta_j = pi (2j+1) / (2H), phi_k = 2 pi k / W;
* Wigner d: d^1_{10}(beta) = -sin(beta)/sqrt(2);
* spin harmonics: sY_lm(theta, phi) = (-1)^s N_l d^l_{m,-s}(theta) e^{i m phi},
  N_l = sqrt((2l+1)/(4 pi)); 0Y_lm is the Condon--Shortley Y_lm;
* coefficient layout: row l^2 + l + m of a [L^2, ...] array; rows with
  l < |s| do not exist and hold 0;
* filter layout: K[l, t, c_out, s, c_in] (output spin/channel first).

Parity: every function here is pinned by tests/test_oracle_*.py against
closed forms, exact rational arithmetic, library routines, invariants or
brute force (see each docstring's "Pinned by").
"""

from __future__ import annotations

import math

import numpy as np

__all__ = [
    "grid",
    "dh_weights",
    "wigner_d",
    "wigner_d_sum_exact",
    "spin_harmonic",
    "coef_index",
    "forward",
    "forward_direct",
    "inverse",
    "evaluate",
    "mix",
    "conv",
    "forward_adjoint",
    "inverse_adjoint",
    "mix_adjoint",
    "filter_grad",
    "conv_backward",
    "delta_matrix",
    "forward_delta",
    "inverse_delta",
    "phase_collapse",
    "spectral_batch_norm",
    "residual_block",
    "bump_coefficients",
]


# --------------------------------------------------------------------------
# Grid and quadrature
# --------------------------------------------------------------------------

def grid(H: int, W: int):
    """Equiangular sample points: colatitudes theta_j and longitudes phi_k.

    The paper only requires an equiangular grid with the same number of
    samples on both axes (appendix, WeatherBench details); we take the
    pole-free Driscoll--Healy / Kostelec--Rockmore offset grid
    theta_j = pi (2j+1)/(2H), phi_k = 2 pi k / W.
    Pinned by: tests/test_oracle_quadrature.py (exactness of the rule built
    on it).
    """
    j = np.arange(H, dtype=np.float64)
    k = np.arange(W, dtype=np.float64)
    theta = np.pi * (2.0 * j + 1.0) / (2.0 * H)
    phi = 2.0 * np.pi * k / W
    return theta, phi


def dh_weights(H: int) -> np.ndarray:
    """Driscoll--Healy latitude weights on the offset grid (H even).

    w_j = (4/H) sin(theta_j) sum_{p=0}^{H/2-1} sin((2p+1) theta_j) / (2p+1),
    so that (2 pi / W) sum_{j,k} w_j g(theta_j, phi_k) integrates g over the
    sphere exactly when g is band-limited to degree < H in latitude and
    |order| < W in longitude.
    Pinned by: Fejer's first-rule closed form, exact integrals of cos^q,
    orthogonality of Legendre polynomials (tests/test_oracle_quadrature.py).
    """
    if H % 2:
        raise ValueError("H must be even")
    theta, _ = grid(H, 1)
    p = np.arange(H // 2, dtype=np.float64)
    s = np.sin(np.outer(theta, 2.0 * p + 1.0)) / (2.0 * p + 1.0)
    return (4.0 / H) * np.sin(theta) * s.sum(axis=1)


# --------------------------------------------------------------------------
# Wigner small-d functions
# --------------------------------------------------------------------------

def _wigner_seed(j: int, m: int, n: int, c: np.ndarray, sg: np.ndarray) -> np.ndarray:
    """d^j_{mn} at the lowest degree j = max(|m|, |n|), where the textbook
    sum has a single term.  c = cos(beta/2), sg = sin(beta/2)."""
    if m == j:
        return math.sqrt(math.comb(2 * j, j + n)) * c ** (j + n) * (-sg) ** (j - n)
    if m == -j:
        return math.sqrt(math.comb(2 * j, j - n)) * c ** (j - n) * sg ** (j + n)
    if n == j:
        return math.sqrt(math.comb(2 * j, j + m)) * c ** (j + m) * sg ** (j - m)
    # n == -j
    return math.sqrt(math.comb(2 * j, j - m)) * c ** (j - m) * (-sg) ** (j + m)


def wigner_d(L: int, m: int, n: int, beta) -> np.ndarray:
    """d^l_{mn}(beta) for l = 0..L-1 (rows), zero where l < max(|m|, |n|).

    The paper uses Wigner Delta = d(pi/2) in eqs. (4)-(6); we evaluate d at
    the grid colatitudes directly.  Seed at l0 = max(|m|,|n|) from the
    single-term textbook sum, then the standard three-term recurrence in l:

      d^{l+1} = (l+1)(2l+1) / sqrt(((l+1)^2-m^2)((l+1)^2-n^2))
                * [ (cos b - m n/(l(l+1))) d^l
                    - sqrt((l^2-m^2)(l^2-n^2)) / (l(2l+1)) d^{l-1} ]

    (the m n/(l(l+1)) term is absent at l = 0).
    Pinned by: exact rational evaluation of the full textbook sum, scipy's
    associated Legendre functions at n = 0, orthogonality, symmetries,
    d(0) = I, and the paper's Delta identity of eqs. (4)/(6)
    (tests/test_oracle_wigner.py).
    """
    beta = np.atleast_1d(np.asarray(beta, dtype=np.float64))
    out = np.zeros((L, beta.size), dtype=np.float64)
    l0 = max(abs(m), abs(n))
    if l0 >= L:
        return out
    c = np.cos(beta / 2.0)
    sg = np.sin(beta / 2.0)
    cb = np.cos(beta)
    out[l0] = _wigner_seed(l0, m, n, c, sg)
    prev = np.zeros_like(beta)
    cur = out[l0].copy()
    for l in range(l0, L - 1):
        lp = l + 1
        a = lp * (2 * l + 1) / math.sqrt((lp * lp - m * m) * (lp * lp - n * n))
        if l == 0:
            t1 = cb * cur
        else:
            t1 = (cb - m * n / (l * (l + 1.0))) * cur
        if l > l0:
            t2 = math.sqrt((l * l - m * m) * (l * l - n * n)) / (l * (2 * l + 1.0)) * prev
        else:
            t2 = 0.0
        nxt = a * (t1 - t2)
        out[lp] = nxt
        prev, cur = cur, nxt
    return out


def wigner_d_sum_exact(l: int, m: int, n: int, cos_half, sin_half) -> float:
    """Full textbook sum for d^l_{mn}(beta) in exact rational arithmetic.

    d^l_{mn} = sqrt((l+m)!(l-m)!(l+n)!(l-n)!) *
               sum_k (-1)^(k-n+m) c^(2l-2k+n-m) s^(2k-n+m)
                     / ((l+n-k)! k! (l-k-m)! (k-n+m)!)
    with c = cos(beta/2), s = sin(beta/2) given as fractions.Fraction, so the
    sum (which cancels badly in floating point) is exact; only the final
    square-root factor is rounded.  Used only as a pin for wigner_d.
    """
    from fractions import Fraction

    c = Fraction(cos_half)
    s = Fraction(sin_half)
    total = Fraction(0)
    for k in range(0, 2 * l + 1):
        a1, a2, a3, a4 = l + n - k, k, l - k - m, k - n + m
        if min(a1, a2, a3, a4) < 0:
            continue
        den = (math.factorial(a1) * math.factorial(a2) * math.factorial(a3)
               * math.factorial(a4))
        term = c ** (2 * l - 2 * k + n - m) * s ** (2 * k - n + m) / den
        total += -term if (k - n + m) % 2 else term
    pref = (math.factorial(l + m) * math.factorial(l - m)
            * math.factorial(l + n) * math.factorial(l - n))
    # sqrt(pref) * total, with the irrational factor rounded once at the end
    return float(total) * math.sqrt(pref) if pref < 2 ** 1000 else \
        float(total * math.isqrt(pref * 10 ** 40)) / 1e20


# --------------------------------------------------------------------------
# Spin-weighted spherical harmonics
# --------------------------------------------------------------------------

def _norm(l):
    return np.sqrt((2.0 * np.asarray(l, dtype=np.float64) + 1.0) / (4.0 * np.pi))


def spin_harmonic(s: int, l: int, m: int, theta, phi) -> np.ndarray:
    """sY_lm(theta, phi) = (-1)^s sqrt((2l+1)/(4pi)) d^l_{m,-s}(theta) e^{i m phi}.

    Zero for l < max(|m|, |s|).  This is the convention under which the
    paper's eqs. (4) and (6) hold and 0Y_lm is the standard harmonic
    (Background, after eqs. (2)-(3)).
    Pinned by: scipy's sph_harm_y at s = 0, closed forms for l <= 2, spin
    raising by finite differences, eqs. (4)/(6) (tests/test_oracle_wigner.py).
    """
    theta = np.asarray(theta, dtype=np.float64)
    phi = np.asarray(phi, dtype=np.float64)
    if l < max(abs(m), abs(s)):
        return np.zeros(np.broadcast(theta, phi).shape, dtype=np.complex128)
    d = wigner_d(l + 1, m, -s, theta.ravel())[l].reshape(theta.shape)
    return ((-1.0) ** s) * _norm(l) * d * np.exp(1j * m * phi)


def coef_index(l: int, m: int) -> int:
    """Row of coefficient (l, m) in the packed [L^2] layout."""
    return l * l + l + m


# --------------------------------------------------------------------------
# Forward / inverse transforms, eqs. (2) and (3)
# --------------------------------------------------------------------------

def _orders(L: int) -> np.ndarray:
    return np.arange(-(L - 1), L)


def _lon_dft_matrix(W: int, L: int, sign: int) -> np.ndarray:
    """e^{sign * 2 pi i (m k mod W)/W}, shape [W, 2L-1]; phases are reduced
    exactly in integers before the float64 exponential."""
    k = np.arange(W)
    m = _orders(L)
    r = np.mod(np.outer(k, m), W).astype(np.float64)
    return np.exp(sign * 2j * np.pi * r / W)


def forward(x: np.ndarray, L: int, spins) -> np.ndarray:
    """Forward SWSFT, eq. (2), by separable Driscoll--Healy quadrature.

    x: complex [B, S, C, H, W] on the grid of `grid`; returns complex
    coefficients [L^2, B, S, C] with
      a[l^2+l+m, b, s, c] = (2pi/W) sum_j w_j sum_k x[b,s,c,j,k] conj(sY_lm(theta_j, phi_k)),
    evaluated as a longitude DFT with exactly reduced phases followed by the
    latitude sum.  Rows with l < |s| are zero.
    Pinned by: forward_direct on tiny grids, orthonormality, Parseval,
    round trip, the mean, longitude-shift equivariance
    (tests/test_oracle_transform.py).
    """
    x = np.asarray(x, dtype=np.complex128)
    B, S, C, H, W = x.shape
    spins = list(spins)
    assert S == len(spins)
    theta, _ = grid(H, W)
    w = dh_weights(H)
    E = _lon_dft_matrix(W, L, -1)
    # X[b, s, c, j, mi] = (2pi/W) sum_k x[b,s,c,j,k] e^{-i m phi_k}
    X = (2.0 * np.pi / W) * (x.reshape(-1, W) @ E).reshape(B, S, C, H, 2 * L - 1)
    # the same numbers laid out [s, mi, j, (b, c)] so each (s, m) slice is contiguous
    X = np.ascontiguousarray(X.transpose(1, 4, 3, 0, 2)).reshape(S, 2 * L - 1, H, B * C)
    coef = np.zeros((L * L, B, S, C), dtype=np.complex128)
    lvals = np.arange(L)
    for si, s in enumerate(spins):
        for mi, m in enumerate(_orders(L)):
            lo = max(abs(m), abs(s))
            if lo >= L:
                continue
            d = wigner_d(L, m, -s, theta)  # [L, H]
            tab = ((-1.0) ** s) * _norm(lvals)[:, None] * d * w[None, :]
            a = (tab @ X[si, mi]).reshape(L, B, C)     # [L, H] x [H, B*C]
            for l in range(lo, L):
                coef[coef_index(l, m), :, si, :] = a[l]
    return coef


def forward_direct(x: np.ndarray, L: int, spins) -> np.ndarray:
    """Eq. (2) as one unseparated double sum over every grid point, with the
    harmonics evaluated by `spin_harmonic` and np.exp of the raw angle.
    O(H W L^2) per map: tiny grids only."""
    x = np.asarray(x, dtype=np.complex128)
    B, S, C, H, W = x.shape
    theta, phi = grid(H, W)
    w = dh_weights(H)
    TH, PH = np.meshgrid(theta, phi, indexing="ij")
    q = (2.0 * np.pi / W) * w[:, None] * np.ones((H, W))
    coef = np.zeros((L * L, B, S, C), dtype=np.complex128)
    for si, s in enumerate(spins):
        for l in range(abs(s), L):
            for m in range(-l, l + 1):
                Y = spin_harmonic(s, l, m, TH, PH)
                coef[coef_index(l, m), :, si, :] = np.einsum(
                    "bcjk,jk->bc", x[:, si], q * np.conj(Y))
    return coef


def inverse(coef: np.ndarray, H: int, W: int, spins) -> np.ndarray:
    """Inverse SWSFT, eq. (3): y = sum_{l >= |s|} sum_{|m| <= l} a_lm sY_lm.

    coef: complex [L^2, B, S, C]; returns complex [B, S, C, H, W].  Separable:
    first G[j, m] = sum_l a_lm (-1)^s N_l d^l_{m,-s}(theta_j), then the
    longitude sum over m with exactly reduced phases.  Rows with l < |s| are
    ignored.
    Pinned by: evaluate (direct sum at arbitrary points), round trip,
    orthonormality (tests/test_oracle_transform.py).
    """
    coef = np.asarray(coef, dtype=np.complex128)
    L2, B, S, C = coef.shape
    L = int(round(math.sqrt(L2)))
    assert L * L == L2
    spins = list(spins)
    theta, _ = grid(H, W)
    lvals = np.arange(L)
    G = np.zeros((S, 2 * L - 1, H, B * C), dtype=np.complex128)
    for si, s in enumerate(spins):
        for mi, m in enumerate(_orders(L)):
            lo = max(abs(m), abs(s))
            if lo >= L:
                continue
            d = wigner_d(L, m, -s, theta)
            tab = ((-1.0) ** s) * _norm(lvals)[:, None] * d  # [L, H]
            a = np.zeros((L, B * C), dtype=np.complex128)
            for l in range(lo, L):
                a[l] = coef[coef_index(l, m), :, si, :].reshape(B * C)
            G[si, mi] = tab.T @ a                              # [H, L] x [L, B*C]
    # [s, mi, j, (b, c)] -> [b, s, c, j, mi], then the longitude sum over m
    G = np.ascontiguousarray(G.reshape(S, 2 * L - 1, H, B, C).transpose(3, 0, 4, 2, 1))
    E = _lon_dft_matrix(W, L, +1)  # [W, 2L-1]
    y = G.reshape(-1, 2 * L - 1) @ E.T
    return y.reshape(B, S, C, H, W)


def evaluate(coef: np.ndarray, spins, theta, phi) -> np.ndarray:
    """Direct sum of eq. (3) at arbitrary points (theta, phi) (same shape);
    returns complex [B, S, C, *theta.shape].  Slow; tiny cases only."""
    coef = np.asarray(coef, dtype=np.complex128)
    L2, B, S, C = coef.shape
    L = int(round(math.sqrt(L2)))
    theta = np.asarray(theta, dtype=np.float64)
    phi = np.asarray(phi, dtype=np.float64)
    out = np.zeros((B, S, C) + theta.shape, dtype=np.complex128)
    for si, s in enumerate(spins):
        for l in range(abs(s), L):
            for m in range(-l, l + 1):
                Y = spin_harmonic(s, l, m, theta, phi)
                out[:, si] += np.multiply.outer(coef[coef_index(l, m), :, si, :], Y)
    return out


# --------------------------------------------------------------------------
# Convolution: per-degree products with filters shared across m
# --------------------------------------------------------------------------

def mix(coef: np.ndarray, K: np.ndarray, spins_in, spins_out) -> np.ndarray:
    """a'[l^2+l+m, b, t, c'] = sum_{s, |s|<=l} sum_c K[l, t, c', s, c] a[l^2+l+m, b, s, c]
    for |t| <= l, else 0.

    The spin-weighted convolution is a product of coefficients per degree l
    with filters shared across the order m (Background, "Spherical CNNs";
    Fig. 2's "*K"); spins are mixed as channels.
    coef: [L^2, B, S_in, C_in]; K: [L, S_out, C_out, S_in, C_in]; returns
    [L^2, B, S_out, C_out].
    Pinned by: an explicit loop over (l, m) on small cases, identity and
    scalar filters, the spin-raising filter, brute-force SO(3) convolution
    (tests/test_oracle_conv.py).
    """
    coef = np.asarray(coef, dtype=np.complex128)
    K = np.asarray(K, dtype=np.complex128)
    L2, B, S, C = coef.shape
    L = K.shape[0]
    assert L * L == L2
    T, Co = K.shape[1], K.shape[2]
    out = np.zeros((L2, B, T, Co), dtype=np.complex128)
    sin_ = np.abs(np.asarray(list(spins_in)))
    sout = np.abs(np.asarray(list(spins_out)))
    for l in range(L):
        Kl = K[l] * (sout[:, None, None, None] <= l) * (sin_[None, None, :, None] <= l)
        rows = slice(l * l, (l + 1) * (l + 1))
        a = coef[rows].reshape(-1, S * C)                    # [(2l+1) B, S C]
        out[rows] = (a @ Kl.reshape(T * Co, S * C).T).reshape(2 * l + 1, B, T, Co)
    return out


def conv(x: np.ndarray, K: np.ndarray, L: int, spins_in, spins_out) -> np.ndarray:
    """The layer: inverse(mix(forward(x))).  x: [B, S_in, C_in, H, W];
    returns [B, S_out, C_out, H, W]."""
    H, W = x.shape[-2:]
    a = forward(x, L, spins_in)
    return inverse(mix(a, K, spins_in, spins_out), H, W, spins_out)


# --------------------------------------------------------------------------
# Backward pass of the layer (adjoints of the linear maps above)
#
# For a real loss of the complex output y with gradient g = dL/dy in the
# convention dL = Re <g, dy> (complex inner product <u, v> = sum conj(u) v),
# a linear map y = A x has input gradient A^H g.  The layer is
# y = G(K . F(x)): F the weighted analysis (eq. (2) by quadrature), K the
# per-degree mixing, G the synthesis (eq. (3)).
# --------------------------------------------------------------------------

def _quadrature_weights(H: int, W: int) -> np.ndarray:
    """q_j = (2 pi / W) w_j: the weight of every sample of latitude j in eq. (2)."""
    return (2.0 * np.pi / W) * dh_weights(H)


def forward_adjoint(coef: np.ndarray, H: int, W: int, spins) -> np.ndarray:
    """F^H: the forward transform's matrix has entries q_j conj(sY_lm(theta_j, phi_k)),
    so its adjoint is x[j, k] = q_j sum_lm a_lm sY_lm(theta_j, phi_k), i.e. the
    synthesis of eq. (3) weighted by q_j.  coef [L^2, B, S, C] -> [B, S, C, H, W].
    Pinned by: <F x, a> = <x, F^H a> (tests/test_oracle_backward.py).
    """
    q = _quadrature_weights(H, W)
    return inverse(coef, H, W, spins) * q[:, None]


def inverse_adjoint(y: np.ndarray, L: int, spins) -> np.ndarray:
    """G^H: a_lm = sum_{j,k} conj(sY_lm(theta_j, phi_k)) y[j, k], the analysis
    sum of eq. (2) without quadrature weights: forward(y / q_j) (the weights
    q_j are positive on this grid).  y [B, S, C, H, W] -> [L^2, B, S, C].
    Pinned by: <G a, y> = <a, G^H y> (tests/test_oracle_backward.py).
    """
    y = np.asarray(y, dtype=np.complex128)
    H, W = y.shape[-2:]
    q = _quadrature_weights(H, W)
    return forward(y / q[:, None], L, spins)


def mix_adjoint(coef_out: np.ndarray, K: np.ndarray, spins_in, spins_out) -> np.ndarray:
    """The adjoint of `mix`: a[l^2+l+m, b, s, c] = sum_{t, c'} conj(K[l, t, c', s, c])
    a'[l^2+l+m, b, t, c'] over |t| <= l, for |s| <= l (else 0).
    coef_out [L^2, B, S_out, C_out] -> [L^2, B, S_in, C_in].
    Pinned by: <mix(a), a'> = <a, mix^H(a')> (tests/test_oracle_backward.py).
    """
    coef_out = np.asarray(coef_out, dtype=np.complex128)
    K = np.asarray(K, dtype=np.complex128)
    L2, B, T, Co = coef_out.shape
    L, S, C = K.shape[0], K.shape[3], K.shape[4]
    out = np.zeros((L2, B, S, C), dtype=np.complex128)
    sin_ = np.abs(np.asarray(list(spins_in)))
    sout = np.abs(np.asarray(list(spins_out)))
    for l in range(L):
        Kl = K[l] * (sout[:, None, None, None] <= l) * (sin_[None, None, :, None] <= l)
        rows = slice(l * l, (l + 1) * (l + 1))
        g = coef_out[rows].reshape(-1, T * Co)               # [(2l+1) B, T Co]
        out[rows] = (g @ np.conj(Kl.reshape(T * Co, S * C))).reshape(2 * l + 1, B, S, C)
    return out


def filter_grad(coef_out_grad: np.ndarray, coef: np.ndarray, spins_in, spins_out) -> np.ndarray:
    """Gradient of the filters of `mix`: since a' = K a per degree,
    dL/dK[l, t, c', s, c] = sum_{|m| <= l, b} g'[l^2+l+m, b, t, c'] conj(a[l^2+l+m, b, s, c]),
    zero where |s| > l or |t| > l.  Returns [L, S_out, C_out, S_in, C_in].
    Pinned by: Re <dL/dK, dK> = d/dh Re <g', mix(a; K + h dK)> and an explicit
    loop over (l, m, b) (tests/test_oracle_backward.py).
    """
    g = np.asarray(coef_out_grad, dtype=np.complex128)
    a = np.asarray(coef, dtype=np.complex128)
    L2, B, T, Co = g.shape
    S, C = a.shape[2], a.shape[3]
    L = int(round(math.sqrt(L2)))
    gK = np.zeros((L, T, Co, S, C), dtype=np.complex128)
    sin_ = np.abs(np.asarray(list(spins_in)))
    sout = np.abs(np.asarray(list(spins_out)))
    for l in range(L):
        rows = slice(l * l, (l + 1) * (l + 1))
        gl = g[rows].reshape(-1, T * Co)                     # [(2l+1) B, T Co]
        al = a[rows].reshape(-1, S * C)
        gK[l] = (gl.T @ np.conj(al)).reshape(T, Co, S, C)
        gK[l] *= (sout[:, None, None, None] <= l) * (sin_[None, None, :, None] <= l)
    return gK


def conv_backward(x: np.ndarray, K: np.ndarray, grad_y: np.ndarray, L: int, spins_in,
                  spins_out):
    """Input and filter gradients of `conv` for output gradient grad_y:
    grad_x = F^H (K^H (G^H grad_y)), grad_K = filter_grad(G^H grad_y, F x)."""
    H, W = x.shape[-2:]
    g_out = inverse_adjoint(grad_y, L, spins_out)
    a = forward(x, L, spins_in)
    grad_K = filter_grad(g_out, a, spins_in, spins_out)
    grad_x = forward_adjoint(mix_adjoint(g_out, K, spins_in, spins_out), H, W, spins_in)
    return grad_x, grad_K


# --------------------------------------------------------------------------
# The Wigner-Delta route of eqs. (4)-(6) (Background, "Computing generalized
# convolutions"): Delta = d(pi/2) and Fourier sums in theta
# --------------------------------------------------------------------------

def delta_matrix(L: int) -> np.ndarray:
    """D[l, m' + L - 1, m + L - 1] = Delta^l_{m'm} = d^l_{m'm}(pi/2), zero
    where |m'| > l or |m| > l.
    Pinned by: the Delta identities of eqs. (4) and (6) against the
    harmonics and the symmetry used by eq. (5) (tests/test_oracle_wigner.py,
    tests/test_oracle_delta.py)."""
    D = np.zeros((L, 2 * L - 1, 2 * L - 1))
    for mp in range(-(L - 1), L):
        for m in range(-(L - 1), L):
            D[:, mp + L - 1, m + L - 1] = wigner_d(L, mp, m, np.pi / 2)[:, 0]
    return D


def forward_delta(x: np.ndarray, L: int, spins, symmetric: bool = False) -> np.ndarray:
    """Forward SWSFT by eq. (4):
        a_lm = (-1)^s i^(m+s) N_l sum_{m'=-l..l} Delta^l_{m'm} Delta^l_{m'(-s)} I_{m'm},
        I_{m'm} = sum_j q_j e^{-i m' theta_j} X_m(theta_j),
    with X_m(theta_j) = sum_k x e^{-i m phi_k} and q_j = (2 pi / W) w_j, so that
    I is the quadrature of eq. (2)'s inner product on the grid.  With
    `symmetric`, eq. (5): the sum runs over m' = 0..l with
    J_{m'm} = I_{m'm} + (-1)^(m+s) I_{-m'm} (m' > 0), J_{0m} = I_{0m}.
    Pinned by: equality with `forward` on non-band-limited input
    (tests/test_oracle_delta.py)."""
    x = np.asarray(x, dtype=np.complex128)
    B, S, C, H, W = x.shape
    spins = list(spins)
    theta, _ = grid(H, W)
    q = (2.0 * np.pi / W) * dh_weights(H)
    E = _lon_dft_matrix(W, L, -1)
    X = (x.reshape(-1, W) @ E).reshape(B, S, C, H, 2 * L - 1)     # [..., j, m]
    mp = _orders(L)
    Eth = q[None, :] * np.exp(-1j * np.outer(mp, theta))           # [m', j]
    I = np.einsum("pj,bscjm->bscpm", Eth, X)                        # [b, s, c, m', m]
    D = delta_matrix(L)
    coef = np.zeros((L * L, B, S, C), dtype=np.complex128)
    for si, s in enumerate(spins):
        for m in range(-(L - 1), L):
            ph = ((-1.0) ** s) * (1j ** ((m + s) % 4))
            for l in range(max(abs(m), abs(s)), L):
                if symmetric:
                    acc = 0.0
                    for p in range(0, l + 1):
                        if p == 0:
                            J = I[:, si, :, L - 1, m + L - 1]
                        else:
                            J = (I[:, si, :, L - 1 + p, m + L - 1]
                                 + (-1.0) ** (m + s) * I[:, si, :, L - 1 - p, m + L - 1])
                        acc = acc + D[l, L - 1 + p, m + L - 1] * D[l, L - 1 + p, -s + L - 1] * J
                else:
                    idx = np.arange(L - 1 - l, L + l)                 # m' = -l..l
                    w = D[l, idx, m + L - 1] * D[l, idx, -s + L - 1]
                    acc = np.einsum("p,bcp->bc", w, I[:, si, :, idx, m + L - 1].transpose(1, 2, 0))
                coef[coef_index(l, m), :, si, :] = ph * _norm(l) * acc
    return coef


def inverse_delta(coef: np.ndarray, H: int, W: int, spins, symmetric: bool = False) -> np.ndarray:
    """Inverse SWSFT by eq. (6):
        f(theta, phi) = sum_{m'} sum_m e^{i m' theta} e^{i m phi} G_{m'm},
        G_{m'm} = (-1)^s i^(m+s) sum_l N_l Delta^l_{(-m')(-s)} Delta^l_{(-m')m} a_lm,
    evaluated on the grid.  With `symmetric`, only G_{m'm} for m' >= 0 is
    computed and G_{(-m')m} = (-1)^(m+s) G_{m'm} fills the rest.
    Pinned by: equality with `inverse` (tests/test_oracle_delta.py)."""
    coef = np.asarray(coef, dtype=np.complex128)
    L2, B, S, C = coef.shape
    L = int(round(math.sqrt(L2)))
    spins = list(spins)
    theta, _ = grid(H, W)
    D = delta_matrix(L)
    mps = _orders(L)
    Y = np.zeros((B, S, C, H, 2 * L - 1), dtype=np.complex128)      # [..., j, m]
    for si, s in enumerate(spins):
        for m in range(-(L - 1), L):
            lo = max(abs(m), abs(s))
            if lo >= L:
                continue
            ph = ((-1.0) ** s) * (1j ** ((m + s) % 4))
            G = np.zeros((2 * L - 1, B, C), dtype=np.complex128)
            for p in (range(0, L) if symmetric else mps):
                for l in range(max(lo, abs(p)), L):
                    G[p + L - 1] += (_norm(l) * D[l, -p + L - 1, -s + L - 1]
                                     * D[l, -p + L - 1, m + L - 1]) * coef[coef_index(l, m), :, si, :]
            if symmetric:
                for p in range(1, L):
                    G[L - 1 - p] = (-1.0) ** (m + s) * G[L - 1 + p]
            Eth = np.exp(1j * np.outer(theta, mps))                  # [j, m']
            Y[:, si, :, :, m + L - 1] = ph * np.einsum("jp,pbc->bcj", Eth, G)
    E = _lon_dft_matrix(W, L, +1)                                    # [k, m]
    return (Y.reshape(-1, 2 * L - 1) @ E.T).reshape(B, S, C, H, W)


# --------------------------------------------------------------------------
# Phase collapse (Method, "Phase collapse nonlinearity")
# --------------------------------------------------------------------------

def phase_collapse(x: np.ndarray, spins, W1: np.ndarray, W2: np.ndarray,
                   bias: np.ndarray) -> np.ndarray:
    """At every grid point, x0 <- W1 x0 + W2 |x| + b; other spins unchanged.

    x: complex [B, S, C, H, W]; x0 = x[:, spins.index(0)] (C channels);
    |x| stacks the moduli of all S*C channels in (spin, channel) order;
    W1: complex [C, C]; W2: complex [C, S*C]; bias: complex [C].
    Pinned by: invariants and selector-matrix cases
    (tests/test_oracle_conv.py).
    """
    x = np.asarray(x, dtype=np.complex128)
    B, S, C, H, W = x.shape
    spins = list(spins)
    s0 = spins.index(0)
    y = x.copy()
    z0 = x[:, s0]                                   # [B, C, H, W]
    mag = np.abs(x).reshape(B, S * C, H, W)         # [B, S*C, H, W]
    y[:, s0] = (np.einsum("oc,bchw->bohw", W1, z0)
                + np.einsum("oc,bchw->bohw", W2, mag)
                + bias[None, :, None, None])
    return y


# --------------------------------------------------------------------------
# Spectral batch normalization and the residual block (Method, "Spectral
# batch normalization", "Spectral pooling and efficient residual block")
# --------------------------------------------------------------------------

def spectral_batch_norm(coef: np.ndarray, spins, gamma: np.ndarray, beta=None,
                        eps: float = 1e-5, var=None, skip=None):
    """Batch normalization computed on the coefficients.

    The l = 0 coefficient is the function's mean (times sqrt(4 pi)) and, by
    Parseval, (1/4pi) sum_{l>=1, m} |a_lm|^2 is the variance of the function
    over the sphere.  Per (spin s, channel c), with batch statistics
        var[s, c] = (1 / (4 pi B)) sum_b sum_{l >= 1} sum_m |a_lm[b, s, c]|^2
    (or the given `var`, e.g. running statistics at inference):
        out_lm = gamma[s, c] a_lm / sqrt(var[s, c] + eps)   for l >= 1,
        out_00 = beta[c] for spin 0 (0 without beta): the mean is removed by
                 zeroing the l = 0 coefficient and the bias sets it,
    then `skip` (same shape as coef) is added if given.
    coef [L^2, B, S, C] complex; gamma [S, C] real; beta [C] complex.
    Returns (out, var).
    Pinned by: the spatial mean and variance of the synthesised output,
    integrated by Gauss--Legendre quadrature independently of the transform
    (tests/test_oracle_block.py).
    """
    a = np.asarray(coef, dtype=np.complex128)
    L2, B, S, C = a.shape
    spins = list(spins)
    if var is None:
        var = np.sum(np.abs(a[1:]) ** 2, axis=(0, 1)) / (4.0 * np.pi * B)   # [S, C]
    var = np.asarray(var, dtype=np.float64)
    scale = np.asarray(gamma, dtype=np.float64) / np.sqrt(var + eps)
    out = a * scale[None, None]
    out[0] = 0.0
    if beta is not None and 0 in spins:
        out[0, :, spins.index(0), :] = np.asarray(beta, dtype=np.complex128)[None, :]
    if skip is not None:
        out = out + np.asarray(skip, dtype=np.complex128)
    return out, var


def residual_block(x: np.ndarray, L: int, H_out: int, spins, K1, K2, bn1, bn2, pc1, pc2,
                   eps: float = 1e-5) -> np.ndarray:
    """The residual block of Fig. 2 with the skip connection in Fourier space:
        a = FT(x)                          (bandlimit L: spectral pooling when L < H_in/2)
        z = sigma1(IFT(BN1(K1 * a)))       on the H_out x H_out grid
        y = sigma2(IFT(BN2(K2 * FT(z)) + a))
    FT / IFT are `forward` / `inverse`, K * the per-degree mixing `mix`,
    BN the spectral batch norm with batch statistics, sigma the phase collapse.
    x [B, S, C, H_in, W_in]; K1, K2 [L, S, C, S, C]; bn = (gamma, beta);
    pc = (W1, W2, bias).  Returns [B, S, C, H_out, H_out].
    Pinned by: K2 = 0 reductions to the phase collapse of the input (same grid)
    and of the input evaluated on the coarse grid (pooling), and exact
    longitude-shift equivariance (tests/test_oracle_block.py).
    """
    a = forward(x, L, spins)
    h = spectral_batch_norm(mix(a, K1, spins, spins), spins, *bn1, eps=eps)[0]
    z = phase_collapse(inverse(h, H_out, H_out, spins), spins, *pc1)
    b = forward(z, L, spins)
    c = spectral_batch_norm(mix(b, K2, spins, spins), spins, *bn2, eps=eps, skip=a)[0]
    return phase_collapse(inverse(c, H_out, H_out, spins), spins, *pc2)


# --------------------------------------------------------------------------
# Input synthesis helper: isotropic bumps projected to a bandlimit
# --------------------------------------------------------------------------

def bump_coefficients(centres: np.ndarray, amps: np.ndarray, width: float,
                      L: int, spin_raise: bool = False) -> np.ndarray:
    """Coefficients of f(x) = sum_i A_i exp(-psi_i(x)^2 / (2 width^2)),
    psi_i the geodesic angle from centre u_i, truncated to l < L.

    Funk--Hecke: f_lm = sum_i A_i g_l conj(Y_lm(u_i)),
    g_l = 2 pi int_{-1}^{1} exp(-arccos(t)^2/(2 width^2)) P_l(t) dt
    (Gauss--Legendre, 400 nodes).  With spin_raise, returns the spin-1
    coefficients sqrt(l(l+1)) f_lm of eth f.
    centres: unit vectors [n, 3]; amps: [n, ...] (trailing dims kept).
    Returns [L^2, ...].
    """
    from numpy.polynomial import legendre

    centres = np.asarray(centres, dtype=np.float64)
    amps = np.asarray(amps, dtype=np.float64)
    t, wq = legendre.leggauss(400)
    g = np.exp(-np.arccos(np.clip(t, -1.0, 1.0)) ** 2 / (2.0 * width ** 2))
    gl = np.array([2.0 * np.pi * np.sum(wq * g * legendre.legval(t, [0] * l + [1]))
                   for l in range(L)])
    th = np.arccos(np.clip(centres[:, 2], -1.0, 1.0))
    ph = np.arctan2(centres[:, 1], centres[:, 0])
    out = np.zeros((L * L,) + amps.shape[1:], dtype=np.complex128)
    for l in range(L):
        fac = gl[l] * (math.sqrt(l * (l + 1.0)) if spin_raise else 1.0)
        for m in range(-l, l + 1):
            Yc = np.conj(spin_harmonic(0, l, m, th, ph))        # [n]
            out[coef_index(l, m)] = fac * np.tensordot(Yc, amps, axes=(0, 0))
    return out
