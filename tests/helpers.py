"""Shared helpers for the tests: dtype rounding, device transfer, relative
error, and the per-workload inputs (random draws from the synthetic module,
band-limited fields synthesised by the float64 oracle)."""

from __future__ import annotations

import numpy as np
import torch

import oracle as O
from paper_2306_05420_amd import synthetic as syn

# Relative-L2 tolerances of the GPU path against the float64 oracle.
TOL = {"f32": 1e-5, "bf16": 2e-2}


def rel_l2(got, ref) -> float:
    got = np.asarray(got, dtype=np.complex128)
    ref = np.asarray(ref, dtype=np.complex128)
    return float(np.linalg.norm((got - ref).ravel()) / np.linalg.norm(ref.ravel()))


def round_to(a: np.ndarray, dtype: str) -> np.ndarray:
    """The complex128 values a GPU buffer of `dtype` holds for `a`."""
    a = np.asarray(a, dtype=np.complex128)
    if dtype == "f32":
        return a.astype(np.complex64).astype(np.complex128)
    r = torch.from_numpy(np.ascontiguousarray(np.stack([a.real, a.imag], -1)))
    r = r.to(torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    return r[..., 0] + 1j * r[..., 1]


def to_device(a: np.ndarray, dtype: str, device="cuda") -> torch.Tensor:
    a = np.asarray(a, dtype=np.complex128)
    if dtype == "f32":
        return torch.from_numpy(a.astype(np.complex64)).to(device)
    r = torch.from_numpy(np.ascontiguousarray(np.stack([a.real, a.imag], -1)))
    return r.to(torch.float32).to(torch.bfloat16).to(device)


def from_device(t: torch.Tensor) -> np.ndarray:
    t = t.detach().cpu()
    if t.dtype == torch.complex64:
        return t.numpy().astype(np.complex128)
    r = t.to(torch.float64).numpy()
    return r[..., 0] + 1j * r[..., 1]


def bump_coefficients(w: syn.Workload, bumps) -> np.ndarray:
    """[L^2, B, S, C] coefficients of the bump fields: spin 0 channels are the
    Funk--Hecke projection of the bumps, spin 1 channels eth of an
    independent bump field (same centres, independent amplitudes)."""
    L = w.L
    a = np.zeros((L * L, w.B, len(w.spins_in), w.C_in), dtype=np.complex128)
    for b, (cent, amps) in enumerate(bumps):
        for si, s in enumerate(w.spins_in):
            if s == 0:
                a[:, b, si, :] = O.bump_coefficients(cent, amps[:, si, :], 0.3, L)
            elif s == 1:
                a[:, b, si, :] = O.bump_coefficients(cent, amps[:, si, :], 0.3, L,
                                                     spin_raise=True)
            else:
                raise ValueError("bump fields are defined for spins 0 and 1")
    return a


def workload_inputs(w: syn.Workload):
    """(x, filters, extras) as complex128 arrays already rounded to the
    workload's storage dtype; x is band-limited, synthesised by the oracle."""
    d = syn.draw(w)
    coef = bump_coefficients(w, d["bumps"]) if w.field == "bumps" else d["coef"]
    x = round_to(O.inverse(coef, w.H, w.W, w.spins_in), w.dtype)
    K = round_to(d["filters"], w.dtype)
    return x, K, d
