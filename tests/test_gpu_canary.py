"""Overrun detection: every entry point of the C ABI, called on buffers that
carry guard bands.

Each buffer a call receives (inputs, outputs and the workspace, sized exactly
as include/swsft.h states) sits between two 4 KiB bands of a fixed byte
pattern.  After the call the bands must be intact (no kernel wrote before or
past its buffer) and every input must be bit-identical to what it was (no
kernel wrote into a buffer it only reads).  The cases cover the five
workloads and shapes that take the ragged, clamped and masked edges of each
kernel family (direct-to-LDS bf16 and float kernels, register-staged
kernels, the small-grid path).
"""

import ctypes

import numpy as np
import pytest
import torch

from paper_2306_05420_amd import swsft as S
from paper_2306_05420_amd import synthetic as syn

pytestmark = pytest.mark.gpu

GUARD = 4096
PATTERN = 0xA5


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    S.lib()
    yield
    torch.cuda.synchronize()


class Guarded:
    """`nbytes` bytes of device memory between two guard bands."""

    def __init__(self, nbytes: int, name: str, gen: torch.Generator = None):
        self.n = int(nbytes)
        self.name = name
        self.raw = torch.full((self.n + 2 * GUARD,), PATTERN, dtype=torch.uint8, device="cuda")
        if gen is not None and self.n:
            # inputs: random bfloat16 values in [-1, 1); read as float32, each
            # 4 bytes hold such a value in the high half, so they are finite too
            body = self.raw[GUARD:GUARD + self.n]
            v = (torch.rand(self.n // 2, generator=gen, device="cuda") * 2 - 1).to(torch.bfloat16)
            body[: 2 * (self.n // 2)].copy_(v.view(torch.uint8))
        self.ptr = self.raw.data_ptr() + GUARD
        self.before = self.raw[GUARD:GUARD + self.n].clone() if gen is not None else None

    def check(self):
        assert bool((self.raw[:GUARD] == PATTERN).all()), f"{self.name}: band before overwritten"
        assert bool((self.raw[GUARD + self.n:] == PATTERN).all()), \
            f"{self.name}: band after overwritten"
        if self.before is not None:
            assert torch.equal(self.raw[GUARD:GUARD + self.n], self.before), \
                f"{self.name}: an input was modified"


def _sizes(plan, B, Ci, Co):
    e = 2 if plan.dtype == "bf16" else 4
    H, W, L = plan.H, plan.W, plan.L
    Si, So = len(plan.spins_in), len(plan.spins_out)
    return {
        "x": B * Si * Ci * H * W * 2 * e,
        "y": B * So * Co * H * W * 2 * e,
        "a_in": L * L * B * Si * Ci * 2 * e,
        "a_out": L * L * B * So * Co * 2 * e,
        "K": L * So * Co * Si * Ci * 2 * e,
    }


def _run(call, bufs):
    print(f"  {call.__name__}: " + ", ".join(f"{b.name} {b.n}" for b in bufs), flush=True)
    torch.cuda.synchronize()
    for b in bufs:
        b.check()


def _all_calls(plan, B, Ci, Co, seed):
    """Call every entry point the plan takes on guarded buffers."""
    Lib = S.lib()
    h = plan._h
    st = torch.cuda.current_stream().cuda_stream
    gen = torch.Generator(device="cuda")
    gen.manual_seed(seed)
    sz = _sizes(plan, B, Ci, Co)

    def ws(op):
        n = Lib.swsft_workspace_bytes(h, op, B, Ci, Co)
        assert n > 0
        return Guarded(n, "workspace")

    def ok(status, what):
        assert status == S.OK, (what, Lib.swsft_last_error().decode())

    # forward transform
    x, a, w = Guarded(sz["x"], "x", gen), Guarded(sz["a_in"], "coef"), ws(S.OP_FORWARD)
    ok(Lib.swsft_forward(h, B, Ci, x.ptr, a.ptr, w.ptr, w.n, st), "swsft_forward")
    _run(Lib.swsft_forward, [x, a, w])
    # inverse transform
    c, y = Guarded(sz["a_out"], "coef", gen), Guarded(sz["y"], "y")
    w = Guarded(Lib.swsft_workspace_bytes(h, S.OP_INVERSE, B, 1, Co), "workspace")
    ok(Lib.swsft_inverse(h, B, Co, c.ptr, y.ptr, w.ptr, w.n, st), "swsft_inverse")
    _run(Lib.swsft_inverse, [c, y, w])
    # the layer, and the layer saving F x
    K = Guarded(sz["K"], "filters", gen)
    y, w = Guarded(sz["y"], "y"), ws(S.OP_CONV)
    ok(Lib.spin_sph_conv_forward(h, B, Ci, Co, x.ptr, K.ptr, y.ptr, w.ptr, w.n, st),
       "spin_sph_conv_forward")
    _run(Lib.spin_sph_conv_forward, [x, K, y, w])
    y, cx, w = Guarded(sz["y"], "y"), Guarded(sz["a_in"], "coef_x"), ws(S.OP_CONV)
    ok(Lib.spin_sph_conv_forward_train(h, B, Ci, Co, x.ptr, K.ptr, y.ptr, cx.ptr, w.ptr, w.n,
                                       st), "spin_sph_conv_forward_train")
    _run(Lib.spin_sph_conv_forward_train, [x, K, y, cx, w])
    cx.before = cx.raw[GUARD:GUARD + cx.n].clone()          # an input from now on
    # the layer on the library's static workspace, where it fits (128 MiB)
    if Lib.swsft_workspace_bytes(h, S.OP_CONV, B, Ci, Co) <= (128 << 20):
        y = Guarded(sz["y"], "y")
        ok(Lib.spin_sph_conv_forward_noalloc(h, B, Ci, Co, x.ptr, K.ptr, y.ptr, st),
           "spin_sph_conv_forward_noalloc")
        _run(Lib.spin_sph_conv_forward_noalloc, [x, K, y])
    # the backward pass: from x, and from the saved coefficients
    gy = Guarded(sz["y"], "grad_y", gen)
    for use_saved in (False, True):
        gx, gk, w = Guarded(sz["x"], "grad_x"), Guarded(sz["K"], "grad_filters"), \
            ws(S.OP_CONV_BACKWARD)
        ok(Lib.spin_sph_conv_backward(h, B, Ci, Co, None if use_saved else x.ptr,
                                      cx.ptr if use_saved else None, K.ptr, gy.ptr, gx.ptr,
                                      gk.ptr, w.ptr, w.n, st), "spin_sph_conv_backward")
        _run(Lib.spin_sph_conv_backward, [x, cx, K, gy, gx, gk, w])
    # the mixing alone
    a_in = Guarded(sz["a_in"], "coef", gen)
    a_out = Guarded(sz["a_out"], "coef_out")
    ok(Lib.spin_sph_mix(h, B, Ci, Co, a_in.ptr, K.ptr, a_out.ptr, st), "spin_sph_mix")
    _run(Lib.spin_sph_mix, [a_in, K, a_out])
    # batch norm on the output spins (batch statistics, skip, variance out)
    So = len(plan.spins_out)
    if So * Co <= 2048:
        gamma = Guarded(So * Co * 4, "gamma", gen)
        beta = Guarded(Co * 8, "beta", gen)
        skip = Guarded(sz["a_out"], "skip", gen)
        var = Guarded(So * Co * 4, "var_out")
        out = Guarded(sz["a_out"], "out")
        w = Guarded(Lib.swsft_workspace_bytes(h, S.OP_BATCH_NORM, B, 1, Co), "workspace")
        ok(Lib.spin_sph_spectral_batch_norm(h, B, Co, c.ptr, gamma.ptr, beta.ptr, 1e-5, None,
                                            var.ptr, skip.ptr, out.ptr, w.ptr, w.n, st),
           "spin_sph_spectral_batch_norm")
        _run(Lib.spin_sph_spectral_batch_norm, [c, gamma, beta, skip, var, out, w])
    # phase collapse (spin 0 among the output spins, C within the LDS limit)
    if 0 in plan.spins_out:
        W1 = Guarded(Co * Co * 8, "W1", gen)
        W2 = Guarded(Co * So * Co * 8, "W2", gen)
        bias = Guarded(Co * 8, "bias", gen)
        yin = Guarded(sz["y"], "x", gen)
        yout = Guarded(sz["y"], "y")
        st_pc = Lib.spin_sph_phase_collapse(h, B, Co, yin.ptr, W1.ptr, W2.ptr, bias.ptr,
                                            yout.ptr, st)
        assert st_pc in (S.OK, S.E_UNSUPPORTED), Lib.swsft_last_error().decode()
        if st_pc == S.OK:
            _run(Lib.spin_sph_phase_collapse, [W1, W2, bias, yin, yout])


WORKLOADS = ["tiny", "small", "mol", "wx128", "wx256"]


@pytest.mark.parametrize("name", WORKLOADS)
def test_guard_bands_workloads(name):
    w = syn.workload(name)
    print(f"canary workload {name}", flush=True)
    plan = S.Plan(w.H, w.W, w.L, w.spins_in, w.spins_out, w.dtype)
    _all_calls(plan, w.B, w.C_in, w.C_out, w.seed)
    plan.close()


EDGE = [
    # H, L, spins_in, spins_out, B, C_in, C_out, dtype
    (16, 5, (0,), (0,), 1, 1, 1, "f32"),              # small path, one channel
    (2, 1, (0,), (0,), 2, 2, 3, "f32"),               # smallest grid
    (8, 4, (0,), (0, 1), 5, 7, 9, "bf16"),            # odd channels, bf16 small path
    (32, 16, (0, 1), (0, 1), 2, 40, 24, "bf16"),      # register-staged bf16 shapes
    (32, 16, (0, 1), (0, 1, -1), 3, 32, 44, "bf16"),  # ragged mixing tiles (last 4 outputs)
    (16, 8, (0, 1, -2), (2, 0), 5, 48, 12, "bf16"),   # 32-wide mixing K steps, |s| = 2
    (64, 32, (0,), (0, 1), 2, 20, 64, "bf16"),        # ragged latitude columns
    (64, 32, (1, -2), (2, 0), 2, 64, 64, "bf16"),     # degree ranges from max(|m|, |s|)
    (64, 32, (1,), (0, -1), 1, 33, 17, "f32"),        # ragged float tiles everywhere
    (64, 20, (0,), (0,), 3, 8, 8, "f32"),             # L << H/2
    (64, 32, (0, 1), (0, 1, 2), 4, 128, 132, "f32"),  # float direct-to-LDS, ragged outputs
    (32, 16, (1, 0), (0, -1), 4, 130, 128, "f32"),    # one-stage float latitude GEMMs
    (128, 64, (0, 1), (1, 0), 3, 96, 160, "bf16"),    # bf16 direct-to-LDS, ragged tiles
]


@pytest.mark.parametrize("case", EDGE, ids=[f"H{c[0]}L{c[1]}B{c[4]}{c[7]}" for c in EDGE])
def test_guard_bands_edge_cases(case):
    H, L, si, so, B, Ci, Co, dt = case
    print(f"canary edge case {case}", flush=True)
    plan = S.Plan(H, H, L, si, so, dt)
    _all_calls(plan, B, Ci, Co, H * 100 + L)
    plan.close()


def test_guard_bands_residual_block_with_pooling():
    w = syn.workload("mol")
    print("canary residual block 64 -> 32", flush=True)
    blk = S.ResidualBlock(2 * w.H, w.H, w.spins_in, w.C_in, "f32", L=w.L)
    Lib = S.lib()
    st = torch.cuda.current_stream().cuda_stream
    gen = torch.Generator(device="cuda")
    gen.manual_seed(77)
    Sn, C, L, B = len(w.spins_in), w.C_in, w.L, w.B
    x = Guarded(B * Sn * C * (2 * w.H) ** 2 * 8, "x", gen)
    y = Guarded(B * Sn * C * w.H ** 2 * 8, "y")
    K1, K2 = (Guarded(L * Sn * C * Sn * C * 8, n, gen) for n in ("K1", "K2"))
    g1, g2 = (Guarded(Sn * C * 4, n, gen) for n in ("gamma1", "gamma2"))
    b1, b2 = (Guarded(C * 8, n, gen) for n in ("beta1", "beta2"))
    pcs = [Guarded(n, nm, gen) for n, nm in ((C * C * 8, "pc1_W1"), (C * Sn * C * 8, "pc1_W2"),
                                             (C * 8, "pc1_b"), (C * C * 8, "pc2_W1"),
                                             (C * Sn * C * 8, "pc2_W2"), (C * 8, "pc2_b"))]
    v1, v2 = Guarded(Sn * C * 4, "var1"), Guarded(Sn * C * 4, "var2")
    prm = S.BlockParams(K1.ptr, K2.ptr, g1.ptr, b1.ptr, g2.ptr, b2.ptr,
                        *[p.ptr for p in pcs], 1e-5, v1.ptr, v2.ptr)
    n = Lib.swsft_block_workspace_bytes(blk.p_in._h, blk.p_out._h, B, C)
    ws = Guarded(n, "workspace")
    assert Lib.spin_sph_residual_block_forward(blk.p_in._h, blk.p_out._h, B, C, x.ptr,
                                               ctypes.byref(prm), y.ptr, ws.ptr, ws.n,
                                               st) == S.OK, Lib.swsft_last_error().decode()
    _run(Lib.spin_sph_residual_block_forward, [x, y, K1, K2, g1, g2, b1, b2, v1, v2, ws] + pcs)
    blk.close()
