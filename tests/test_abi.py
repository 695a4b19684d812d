"""CPU tests of the C ABI: the library loads, exports every function that
include/swsft.h declares, and rejects invalid arguments on the host before
any HIP call (so they need no GPU)."""

import ctypes

import pytest

from paper_2306_05420_amd import swsft as S


@pytest.fixture(scope="module")
def L():
    return S.lib()


def test_exports_every_declared_function(L):
    names = S.header_functions()
    assert len(names) == 22
    for n in names:
        assert hasattr(L, n), n


def _create(L, H, W, Lb, si, so, dtype=0, out=True):
    a = (ctypes.c_int * max(1, len(si)))(*si)
    b = (ctypes.c_int * max(1, len(so)))(*so)
    h = ctypes.c_void_p()
    return L.swsft_plan_create(H, W, Lb, a, len(si), b, len(so), dtype,
                               ctypes.byref(h) if out else None)


@pytest.mark.parametrize("args,status", [
    ((16, 8, 8, [0], [0]), S.E_INVALID),          # H != W
    ((15, 15, 7, [0], [0]), S.E_INVALID),         # odd H
    ((16, 16, 9, [0], [0]), S.E_INVALID),         # L > H/2
    ((16, 16, 0, [0], [0]), S.E_INVALID),         # L < 1
    ((16, 16, 8, [0, 0], [0]), S.E_INVALID),      # repeated spin
    ((16, 16, 8, [8], [0]), S.E_INVALID),         # |s| >= L
    ((16, 16, 8, [0], [-8]), S.E_INVALID),
    ((16, 16, 8, [], [0]), S.E_INVALID),          # no spins
    ((16, 16, 8, list(range(-4, 5)), [0]), S.E_INVALID),  # 9 spins
    ((24, 24, 8, [0], [0]), S.E_UNSUPPORTED),     # W not a power of two
    ((1024, 1024, 8, [0], [0]), S.E_UNSUPPORTED),  # W > 512
])
def test_plan_create_validation(L, args, status):
    assert _create(L, *args) == status
    assert L.swsft_last_error().decode() != ""


def test_plan_create_flags(L):
    a = (ctypes.c_int * 1)(0)
    h = ctypes.c_void_p()
    # unknown flag bits; the two Delta routes together
    assert L.swsft_plan_create_ex(16, 16, 8, a, 1, a, 1, 0, 8, ctypes.byref(h)) == S.E_INVALID
    assert L.swsft_plan_create_ex(64, 64, 32, a, 1, a, 1, 0, 6, ctypes.byref(h)) == S.E_INVALID
    # the Delta route takes L a multiple of 32
    assert L.swsft_plan_create_ex(32, 32, 16, a, 1, a, 1, 0, 4, ctypes.byref(h)) == S.E_UNSUPPORTED
    # a width that is not a power of two needs the DFT-matrix longitude stage
    assert L.swsft_plan_create_ex(96, 96, 48, a, 1, a, 1, 0, 0, ctypes.byref(h)) == S.E_UNSUPPORTED
    assert L.swsft_plan_create(96, 96, 48, a, 1, a, 1, 0, ctypes.byref(h)) == S.E_UNSUPPORTED
    # grids above 32 take whole latitude tiles of 32 rows
    assert L.swsft_plan_create_ex(48, 48, 24, a, 1, a, 1, 0, 1, ctypes.byref(h)) == S.E_UNSUPPORTED


def test_plan_create_bad_dtype_and_null_out(L):
    assert _create(L, 16, 16, 8, [0], [0], dtype=7) == S.E_INVALID
    assert _create(L, 16, 16, 8, [0], [0], out=False) == S.E_INVALID


def test_calls_reject_null_plan(L):
    vp = ctypes.c_void_p
    x = vp(1 << 20)
    assert L.swsft_forward(None, 1, 1, x, x, x, 1 << 30, None) == S.E_INVALID
    assert L.swsft_inverse(None, 1, 1, x, x, x, 1 << 30, None) == S.E_INVALID
    assert L.spin_sph_conv_forward(None, 1, 1, 1, x, x, x, x, 1 << 30, None) == S.E_INVALID
    assert L.spin_sph_conv_backward(None, 1, 1, 1, x, x, x, x, x, x, x, 1 << 30, None) == S.E_INVALID
    assert L.spin_sph_conv_forward_train(None, 1, 1, 1, x, x, x, x, x, 1 << 30, None) == S.E_INVALID
    assert L.spin_sph_conv_forward_noalloc(None, 1, 1, 1, x, x, x, None) == S.E_INVALID
    assert L.spin_sph_phase_collapse(None, 1, 1, x, x, x, x, x, None) == S.E_INVALID
    assert L.spin_sph_mix(None, 1, 1, 1, x, x, x, None) == S.E_INVALID
    assert L.spin_sph_spectral_batch_norm(None, 1, 1, x, x, None, 0.0, None, None, None, x, x,
                                          1 << 30, None) == S.E_INVALID
    assert L.swsft_block_workspace_bytes(None, None, 1, 1) == 0
    assert L.spin_sph_residual_block_forward(None, None, 1, 1, x, None, x, x, 1 << 30,
                                             None) == S.E_INVALID
    assert L.swsft_stage_timing(None, 1) == S.E_INVALID
    assert L.swsft_workspace_bytes(None, 0, 1, 1, 1) == 0
    assert L.swsft_stage_times(None, None, None, 0) == 0
    L.swsft_plan_destroy(None)


def test_status_strings_and_stage_names(L):
    for st in range(6):
        assert L.swsft_status_string(st).decode().startswith("SWSFT_")
    assert L.swsft_status_string(99).decode() == "unknown swsft status"
    assert [L.swsft_stage_name(i).decode() for i in range(len(S.STAGES))] == list(S.STAGES)
    assert L.swsft_stage_name(len(S.STAGES)).decode() == ""


def test_mfma_probe_validation(L):
    # refused on the host before any launch: dtype, iteration and wave counts, NULL out
    out = ctypes.c_void_p(1 << 20)
    f = ctypes.c_double(0.0)
    assert L.swsft_probe_mfma(7, 1, 10, 8, out, ctypes.byref(f), None) == S.E_INVALID
    assert L.swsft_probe_mfma(S.BF16, 1, 0, 8, out, ctypes.byref(f), None) == S.E_INVALID
    assert L.swsft_probe_mfma(S.BF16, 1, 1 << 25, 8, out, ctypes.byref(f), None) == S.E_INVALID
    assert L.swsft_probe_mfma(S.BF16, 1, 10, 6, out, ctypes.byref(f), None) == S.E_INVALID
    assert L.swsft_probe_mfma(S.F32, 1, 10, 0, out, ctypes.byref(f), None) == S.E_INVALID
    assert L.swsft_probe_mfma(S.BF16, 1, 10, 8, None, ctypes.byref(f), None) == S.E_INVALID
    assert L.swsft_last_error().decode() != ""
