"""The register-only MFMA probe behind bench.py's measured MFMA rates
(swsft_probe_mfma): with constant operands (all ones) every lane's checksum
is exact, which pins the instruction shape and the number of MFMAs issued:
each of the 16 accumulator registers of each of the 4 chains gains K per
MFMA (K = 16 for 32x32x16 bf16, 2 for 32x32x2 f32), so the sum of a lane's
64 accumulator values after `iters` rounds is 64 K iters.  Random operands
give finite checksums."""

import pytest
import torch

from paper_2306_05420_amd import swsft as S

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype,k", [("bf16", 16), ("f32", 2)])
def test_probe_constant_operands_exact(dtype, k):
    n_waves, iters = 16, 100
    out = torch.full((64 * n_waves,), -1.0, dtype=torch.float32, device="cuda")
    flops = S.probe_mfma(dtype, False, iters, n_waves, out)
    torch.cuda.synchronize()
    assert flops == n_waves * iters * 4 * 2 * 32 * 32 * k
    assert torch.equal(out, torch.full_like(out, 64.0 * k * iters))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_probe_random_operands_finite(dtype):
    n_waves = 8
    out = torch.zeros(64 * n_waves, dtype=torch.float32, device="cuda")
    S.probe_mfma(dtype, True, 50, n_waves, out)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(out).all())
    assert float(out.abs().sum()) > 0.0
