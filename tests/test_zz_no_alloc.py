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
