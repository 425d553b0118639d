"""HIP graph capture of the conv and pool launches (the benchmark replays a
captured step, with the pool either its own launch or fused into the conv
launch): every replay must equal the eager result bit for bit, also with
eager work and synchronisations between the replays."""
import numpy as np
import pytest

from paper_2003_06513_amd import binding as B
from synthetic import inputs
from gpu_cases import dev, note, torch_mod

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    B.lib()


@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_graph_replays_match_eager(dtype, fused):
    torch = torch_mod()
    tdt = torch.float32 if dtype == np.float32 else torch.float16
    # conv 8->16 @ 28x28 (+ReLU, pool) -> conv 16->32 @ 14x14 (split shares) -> conv 32->32 @ 14x14
    n = 2
    shapes = [(8, 16, 28), (16, 32, 14), (32, 32, 14)]
    preps, bufs = [], []
    masks = None
    ws = [inputs.he_weights(70 + i, co, ci, dtype) for i, (ci, co, _) in enumerate(shapes)]
    masks = B.select_library(np.concatenate([w.reshape(-1, 3, 3) for w in ws]), 8)
    for (ci, co, s), w in zip(shapes, ws):
        preps.append(B.prepare(dev(w), masks, inputs.keep_after_drop(ci * co, 60)))
        bufs.append(torch.empty((n, co, s, s), dtype=tdt, device="cuda"))
    pooled = torch.empty((n, 16, 14, 14), dtype=tdt, device="cuda")
    x = dev(inputs.normal_activations(71, (n, 8, 28, 28), dtype))

    def step():
        if fused:
            B.conv3x3_fwd_pool2(preps[0].layer, preps[0].packed, x, pooled, relu=True)
        else:
            B.conv3x3_fwd(preps[0].layer, preps[0].packed, x, bufs[0], relu=True)
            B.maxpool2x2(bufs[0], pooled)
        B.conv3x3_fwd(preps[1].layer, preps[1].packed, pooled, bufs[1], relu=True)
        B.conv3x3_fwd(preps[2].layer, preps[2].packed, bufs[1], bufs[2], relu=False)

    note("graph eager reference %s fused=%s" % (np.dtype(dtype).name, fused))
    step()
    torch.cuda.synchronize()
    ref = bufs[2].clone()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    note("graph capture")
    with torch.cuda.graph(g):
        step()
    for rep in range(3):
        bufs[2].fill_(123.0)                 # eager work between replays
        torch.cuda.synchronize()
        note("graph replay %d" % rep)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(bufs[2], ref), "replay %d differs from the eager result" % rep
