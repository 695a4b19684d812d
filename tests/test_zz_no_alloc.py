"""spin_sph_conv_forward_noalloc (the layer on the library's static
workspace) against spin_sph_conv_forward with a caller workspace, through
the C ABI: the same kernels run in the same launch configuration, so the
outputs must be bit-identical.  Two calls in a row on one plan, the second
with a smaller batch (the static array keeps the first call's contents),
then a layer whose workspace exceeds the static array, which is refused
with nothing enqueued."""

import numpy as np
import pytest
import torch

from paper_2306_05420_amd import swsft as S
from paper_2306_05420_amd import synthetic as syn

pytestmark = pytest.mark.gpu

STATIC_BYTES = 128 << 20


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    S.lib()
    yield
    torch.cuda.synchronize()


def _inputs(plan, w, B, seed):
    gen = torch.Generator(device="cuda")
    gen.manual_seed(seed)
    x = plan.empty(B, len(w.spins_in), w.C_in, w.H, w.W)
    K = plan.empty(w.L, len(w.spins_out), w.C_out, len(w.spins_in), w.C_in)
    for t in (x, K):
        r = torch.view_as_real(t) if t.dtype == torch.complex64 else t
        r.copy_(torch.randn(r.shape, generator=gen, device="cuda").to(r.dtype))
    return x, K


@pytest.mark.parametrize("name", ["wx128", "mol"])
def test_noalloc_matches_caller_workspace(name):
    w = syn.workload(name)
    Lib = S.lib()
    plan = S.Plan(w.H, w.W, w.L, w.spins_in, w.spins_out, w.dtype)
    st = torch.cuda.current_stream().cuda_stream
    for B, seed in ((w.B, 1), (max(1, w.B // 2), 2)):     # the second call smaller
        print(f"noalloc {name} B={B}", flush=True)
        need = plan.workspace_bytes(S.OP_CONV, B, w.C_in, w.C_out)
        assert 0 < need <= STATIC_BYTES
        x, K = _inputs(plan, w, B, seed)
        y_ref = plan.conv(x, K)
        y = plan.empty(*y_ref.shape)
        xr, kr, yr = (plan.real_view(t) for t in (x, K, y))
        assert Lib.spin_sph_conv_forward_noalloc(plan._h, B, w.C_in, w.C_out, xr.data_ptr(),
                                                 kr.data_ptr(), yr.data_ptr(), st) == S.OK, \
            Lib.swsft_last_error().decode()
        torch.cuda.synchronize()
        assert torch.equal(y, y_ref), name
    plan.close()


def test_noalloc_refuses_layers_above_the_static_workspace():
    w = syn.workload("wx256")
    Lib = S.lib()
    plan = S.Plan(w.H, w.W, w.L, w.spins_in, w.spins_out, w.dtype)
    assert plan.workspace_bytes(S.OP_CONV, w.B, w.C_in, w.C_out) > STATIC_BYTES
    x = torch.zeros(16, dtype=torch.bfloat16, device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    status = Lib.spin_sph_conv_forward_noalloc(plan._h, w.B, w.C_in, w.C_out, x.data_ptr(),
                                               x.data_ptr(), x.data_ptr(), st)
    assert status == S.E_UNSUPPORTED
    assert "static workspace" in Lib.swsft_last_error().decode()
    torch.cuda.synchronize()
    plan.close()


@pytest.mark.parametrize("name", ["mol", "wx128"])
def test_noalloc_graph_replays_match_eager(name):
    """The entry point captured in a HIP graph (the callers it is for): every
    replay reproduces the eager call bit for bit, with an eager call of the
    same entry point on another input between replays (it rewrites the
    static workspace the replay then reuses)."""
    w = syn.workload(name)
    Lib = S.lib()
    plan = S.Plan(w.H, w.W, w.L, w.spins_in, w.spins_out, w.dtype)
    x, K = _inputs(plan, w, w.B, 3)
    x2, _ = _inputs(plan, w, w.B, 4)
    shape = (w.B, len(w.spins_out), w.C_out, w.H, w.W)
    y, y2 = plan.empty(*shape), plan.empty(*shape)

    def call(xx, yy):
        st = torch.cuda.current_stream().cuda_stream
        xr, kr, yr = (plan.real_view(t) for t in (xx, K, yy))
        status = Lib.spin_sph_conv_forward_noalloc(plan._h, w.B, w.C_in, w.C_out, xr.data_ptr(),
                                                   kr.data_ptr(), yr.data_ptr(), st)
        assert status == S.OK, Lib.swsft_last_error().decode()

    print(f"noalloc graph {name}", flush=True)
    call(x, y)
    call(x2, y2)
    torch.cuda.synchronize()
    ref, ref2 = y.clone(), y2.clone()
    assert torch.equal(ref, plan.conv(x, K)) and torch.equal(ref2, plan.conv(x2, K))
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call(x, y)
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call(x, y)
    for rep in range(4):
        y.zero_()
        y2.zero_()
        call(x2, y2)                         # eager, same static workspace
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, ref), (name, rep)
        assert torch.equal(y2, ref2), (name, rep)
    del g
    plan.close()
