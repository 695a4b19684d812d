"""Seeded synthetic inputs for the spin-weighted spherical convolution layer.

This module only draws random numbers and shapes them; it contains none of
the transform's arithmetic (no harmonics, quadrature or DFT).  It is the one
module that both the float64 oracle's tests and the GPU benchmarks use.

Workloads (molecule- and weather-shaped stand-ins for the paper's QM9 and
ERA5 experiments, which need data that is not available here):

====  =======  ====  ==  ==========  =============  ======  =====================
name  grid     L     B   spins       C_in -> C_out  dtype   input field
====  =======  ====  ==  ==========  =============  ======  =====================
tiny  16x16    8     1   {0}->{0,1}  4 -> 4         f32     CN(0,1) coefficients
small 32x32    16    8   {0}->{0,1}  16 -> 32       f32     CN(0,1)/(l+1)
mol   32x32    16    32  {0,1}->{0,1} 64 -> 64      f32     1..29 Gaussian bumps
wx128 128x128  64    4   {0}->{0}    128 -> 128     f32     CN(0,1)/(l+1)
wx256 256x256  128   2   {0,1}->{0,1} 256 -> 256    bf16    CN(0,1)/(l+1)
====  =======  ====  ==  ==========  =============  ======  =====================

Seeds: numpy Generator(PCG64(1000 + i)) for workload i (1-based, table
order); draws in the order coefficients-or-bumps, filters, phase-collapse
parameters.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class Workload:
    index: int
    name: str
    H: int
    W: int
    L: int
    B: int
    spins_in: tuple
    spins_out: tuple
    C_in: int
    C_out: int
    dtype: str          # "f32" or "bf16": storage type of the GPU path
    field: str          # "white", "decay1" (amplitude (l+1)^-1) or "bumps"
    filter_var: float   # variance of each complex filter entry
    notes: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def seed(self) -> int:
        return 1000 + self.index

    def rng(self) -> np.random.Generator:
        return np.random.Generator(np.random.PCG64(self.seed))


WORKLOADS = (
    Workload(1, "tiny", 16, 16, 8, 1, (0,), (0, 1), 4, 4, "f32", "white", 1.0 / 4),
    Workload(2, "small", 32, 32, 16, 8, (0,), (0, 1), 16, 32, "f32", "decay1", 1.0 / 16),
    Workload(3, "mol", 32, 32, 16, 32, (0, 1), (0, 1), 64, 64, "f32", "bumps", 1.0 / 128,
             notes="also a two-layer stack with phase collapse in between"),
    Workload(4, "wx128", 128, 128, 64, 4, (0,), (0,), 128, 128, "f32", "decay1", 1.0 / 128,
             notes="transform-only throughput reported too"),
    Workload(5, "wx256", 256, 256, 128, 2, (0, 1), (0, 1), 256, 256, "bf16", "decay1",
             1.0 / 512, notes="bf16 storage, fp32 accumulation"),
)


def workload(name_or_index) -> Workload:
    for w in WORKLOADS:
        if w.name == name_or_index or w.index == name_or_index:
            return w
    raise KeyError(name_or_index)


def complex_normal(rng: np.random.Generator, shape, var: float = 1.0) -> np.ndarray:
    """Circular complex normal: real and imaginary parts i.i.d. N(0, var/2)."""
    sd = np.sqrt(var / 2.0)
    return rng.normal(0.0, sd, size=shape) + 1j * rng.normal(0.0, sd, size=shape)


def random_coefficients(rng: np.random.Generator, L: int, B: int, spins, C: int,
                        decay: float = 0.0) -> np.ndarray:
    """Complex [L^2, B, S, C] coefficients, row l^2+l+m, CN(0,1) times
    (l+1)^-decay; rows with l < |s| (which do not exist for spin s) are 0."""
    spins = list(spins)
    a = complex_normal(rng, (L * L, B, len(spins), C))
    l_of_row = np.floor(np.sqrt(np.arange(L * L))).astype(np.int64)
    a *= ((l_of_row + 1.0) ** (-decay))[:, None, None, None]
    for si, s in enumerate(spins):
        a[l_of_row < abs(s), :, si, :] = 0.0
    return a


def random_filters(rng: np.random.Generator, L: int, spins_in, C_in: int,
                   spins_out, C_out: int, var: float) -> np.ndarray:
    """Complex filters [L, S_out, C_out, S_in, C_in], each entry CN(0, var)."""
    return complex_normal(rng, (L, len(spins_out), C_out, len(spins_in), C_in), var)


def bump_parameters(rng: np.random.Generator, B: int, S: int, C: int,
                    max_bumps: int = 29):
    """Per batch item: n ~ U{1..max_bumps} centres uniform on the sphere
    (normalised N(0, I_3) draws) and N(0,1) amplitudes per (bump, spin,
    channel).  Returns a list of (centres [n,3], amps [n,S,C])."""
    out = []
    for _ in range(B):
        n = int(rng.integers(1, max_bumps + 1))
        v = rng.normal(size=(n, 3))
        v /= np.linalg.norm(v, axis=1, keepdims=True)
        amps = rng.normal(size=(n, S, C))
        out.append((v, amps))
    return out


def phase_collapse_parameters(rng: np.random.Generator, S: int, C: int):
    """W1 ~ CN(0, 1/C) [C, C]; W2 ~ CN(0, 1/(S C)) [C, S C]; b ~ CN(0, 0.01) [C]."""
    W1 = complex_normal(rng, (C, C), 1.0 / C)
    W2 = complex_normal(rng, (C, S * C), 1.0 / (S * C))
    b = complex_normal(rng, (C,), 0.01)
    return W1, W2, b


def draw(w: Workload):
    """All random draws for a workload, in the fixed order.

    Returns a dict with either 'coef' ([L^2, B, S_in, C_in]) or 'bumps'
    (list from bump_parameters), 'filters', and for the bump workload a
    second filter bank 'filters2' and the phase-collapse parameters 'pc'.
    """
    rng = w.rng()
    out = {}
    if w.field == "bumps":
        out["bumps"] = bump_parameters(rng, w.B, len(w.spins_in), w.C_in)
    else:
        decay = {"white": 0.0, "decay1": 1.0}[w.field]
        out["coef"] = random_coefficients(rng, w.L, w.B, w.spins_in, w.C_in, decay)
    out["filters"] = random_filters(rng, w.L, w.spins_in, w.C_in, w.spins_out,
                                    w.C_out, w.filter_var)
    if w.field == "bumps":
        out["pc"] = phase_collapse_parameters(rng, len(w.spins_out), w.C_out)
        out["filters2"] = random_filters(rng, w.L, w.spins_out, w.C_out,
                                         w.spins_out, w.C_out, w.filter_var)
    return out


# ---------------------------------------------------------------------------
# The same recipes drawn on the GPU with torch's seeded generator, for
# benchmarks that only need inputs of the right shape and distribution (not
# the exact values the float64 oracle sees in the parity tests).
# ---------------------------------------------------------------------------

def torch_complex_normal(gen, shape, var: float = 1.0, device="cuda"):
    import torch

    sd = (var / 2.0) ** 0.5
    re = torch.randn(shape, generator=gen, device=device, dtype=torch.float32) * sd
    im = torch.randn(shape, generator=gen, device=device, dtype=torch.float32) * sd
    return torch.complex(re, im)


def torch_random_coefficients(gen, L: int, B: int, spins, C: int, decay: float = 0.0,
                              device="cuda"):
    """Complex64 [L^2, B, S, C]: CN(0,1) (l+1)^-decay, zero where l < |s|."""
    import torch

    spins = list(spins)
    a = torch_complex_normal(gen, (L * L, B, len(spins), C), 1.0, device)
    l_of_row = torch.arange(L * L, device=device).float().sqrt().floor()
    a *= ((l_of_row + 1.0) ** (-decay)).to(a.dtype)[:, None, None, None]
    for si, s in enumerate(spins):
        a[l_of_row < abs(s), :, si, :] = 0
    return a


def torch_random_filters(gen, L: int, spins_in, C_in: int, spins_out, C_out: int,
                         var: float, device="cuda"):
    """Complex64 filters [L, S_out, C_out, S_in, C_in], each entry CN(0, var)."""
    return torch_complex_normal(gen, (L, len(spins_out), C_out, len(spins_in), C_in), var,
                                device)
