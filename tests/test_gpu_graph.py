"""The layer and its backward pass captured in a HIP graph (through torch's
graph capture): every replay must reproduce the eager result bit for bit,
with the program's own eager work and synchronizations between replays (the
per-call path issues kernel launches only: no memset, allocation or host
synchronization)."""

import numpy as np
import pytest
import torch

from paper_2306_05420_amd import swsft as S
from paper_2306_05420_amd import synthetic as syn
from helpers import to_device, workload_inputs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["tiny", "small", "mol"])
def test_graph_replays_match_eager(name):
    assert torch.cuda.is_available()
    w = syn.workload(name)
    x, K, _ = workload_inputs(w)
    rng = np.random.default_rng(w.seed + 11)
    gy = syn.complex_normal(rng, (w.B, len(w.spins_out), w.C_out, w.H, w.W))
    plan = S.Plan(w.H, w.W, w.L, w.spins_in, w.spins_out, w.dtype)
    xd, Kd, gd = to_device(x, w.dtype), to_device(K, w.dtype), to_device(gy, w.dtype)
    y = plan.empty(w.B, len(w.spins_out), w.C_out, w.H, w.W)
    gx = plan.empty(*xd.shape[:-1] if w.dtype == "bf16" else xd.shape)
    gk = plan.empty(*Kd.shape[:-1] if w.dtype == "bf16" else Kd.shape)

    def step():
        plan.conv(xd, Kd, y)
        plan.conv_backward(xd, Kd, gd, grad_x=gx, grad_filters=gk)

    step()                                   # eager; allocates the workspaces
    torch.cuda.synchronize()
    ref = [y.clone(), gx.clone(), gk.clone()]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for rep in range(4):
        for t in (y, gx, gk):
            t.zero_()
        plan.forward(xd)                     # unrelated eager work between replays
        g.replay()
        torch.cuda.synchronize()
        for got, want in zip((y, gx, gk), ref):
            assert torch.equal(got, want), (name, rep)
    del g
    plan.close()


def test_graph_replays_match_eager_bf16_wx256():
    """The 256 x 256, C = 256, bfloat16 layer and backward (direct-to-LDS
    GEMMs, the adjoint mixing from the filters as stored, the streamed DFTs,
    the inverse over batch items) captured and replayed; random inputs of the
    workload's shapes (a replay is compared with the eager call, not with the
    oracle)."""
    assert torch.cuda.is_available()
    w = syn.workload("wx256")
    plan = S.Plan(w.H, w.W, w.L, w.spins_in, w.spins_out, w.dtype)
    gen = torch.Generator(device="cuda").manual_seed(5)

    def rnd(*shape, scale=1.0):
        t = plan.empty(*shape)
        t.copy_((torch.randn(t.shape, device="cuda", generator=gen) * scale).to(torch.bfloat16))
        return t

    Si, So = len(w.spins_in), len(w.spins_out)
    xd = rnd(w.B, Si, w.C_in, w.H, w.W)
    Kd = rnd(w.L, So, w.C_out, Si, w.C_in, scale=0.05)
    gd = rnd(w.B, So, w.C_out, w.H, w.W)
    y = plan.empty(w.B, So, w.C_out, w.H, w.W)
    gx = plan.empty(w.B, Si, w.C_in, w.H, w.W)
    gk = plan.empty(w.L, So, w.C_out, Si, w.C_in)

    def step():
        plan.conv(xd, Kd, y)
        plan.conv_backward(xd, Kd, gd, grad_x=gx, grad_filters=gk)

    step()
    torch.cuda.synchronize()
    ref = [y.clone(), gx.clone(), gk.clone()]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for rep in range(3):
        for t in (y, gx, gk):
            t.zero_()
        plan.forward(xd)
        g.replay()
        torch.cuda.synchronize()
        for got, want in zip((y, gx, gk), ref):
            assert torch.equal(got, want), ("wx256", rep)
    del g
    plan.close()


def test_two_streams_with_one_call_shape_use_separate_workspaces():
    """The binding caches one workspace per call shape and stream: two layer
    calls of the same shape running concurrently on two streams must each
    give their eager single-stream result bit for bit."""
    w = syn.workload("mol")
    plan = S.Plan(w.H, w.W, w.L, w.spins_in, w.spins_out, w.dtype)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(3)
    xs = [syn.torch_complex_normal(gen, (w.B, len(w.spins_in), w.C_in, w.H, w.W)) for _ in range(2)]
    K = syn.torch_random_filters(gen, w.L, w.spins_in, w.C_in, w.spins_out, w.C_out, w.filter_var)
    refs = [plan.conv(x, K).clone() for x in xs]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    ys = [plan.empty(*r.shape) for r in refs]
    for rep in range(3):
        for st in streams:
            st.wait_stream(torch.cuda.current_stream())
        for st, x, y in zip(streams, xs, ys):
            with torch.cuda.stream(st):
                plan.conv(x, K, y)
        torch.cuda.synchronize()
        for y, r in zip(ys, refs):
            assert torch.equal(y, r), rep
        for y in ys:
            y.zero_()
    plan.close()
