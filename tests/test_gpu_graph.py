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
