"""The measurement probes compute what they say.  psc_probe_fma: per lane, 8
chains a_j = fma(a_j, b, c) started at lane + j, summed (fp32).
psc_probe_mfma: 4 chains of fp32 MFMA 16x16x4 with A all 1 and B all 1/4,
each instruction adding exactly 1 to each result, so every lane's 16 results
sum to 16 * iters."""
import numpy as np
import pytest

from paper_2003_06513_amd import binding as B

pytestmark = pytest.mark.gpu


def test_probe_fma_values():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    blocks, iters = 3, 5
    out = torch.full((blocks * 256,), -1.0, dtype=torch.float32, device="cuda")
    B.probe_fma(blocks, iters, out)
    torch.cuda.synchronize()
    b, c = np.float32(1.0000001), np.float32(1e-7)
    lane = np.arange(256, dtype=np.float64)
    s = np.zeros(256, dtype=np.float32)
    for j in range(8):
        a = (lane + j).astype(np.float32)
        for _ in range(iters):
            # a*b is exact in fp64 (24 + 24 bits); one rounding to fp32 after the add
            a = (a.astype(np.float64) * np.float64(b) + np.float64(c)).astype(np.float32)
        s = (s + a).astype(np.float32)
    got = out.cpu().numpy().reshape(blocks, 256)
    for k in range(blocks):
        np.testing.assert_allclose(got[k], s, rtol=1e-6, atol=0)


@pytest.mark.parametrize("iters", [0, 1, 1000])
def test_probe_mfma_values(iters):
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    blocks = 5
    out = torch.full((blocks * 256,), -1.0, dtype=torch.float32, device="cuda")
    B.probe_mfma(blocks, iters, out)
    torch.cuda.synchronize()
    assert bool((out == 16.0 * iters).all())
