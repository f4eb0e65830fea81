"""qnet_forward inside a captured HIP graph (run with -m gpu): the forward
launches only kernels on the caller's stream (no allocation, copy or memset),
so it can be captured; every replay must reproduce the eager logits bit for
bit, with the program's own eager work and synchronisations between replays
(the output is overwritten with NaN before each replay)."""
import pytest
import torch

from paper_2003_04296_amd import synth
from paper_2003_04296_amd.nets import build_convnet, build_resnet18

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


@pytest.mark.parametrize("net", ["convnet", "resnet18"])
def test_forward_replays_from_a_captured_graph(dev, net):
    if net == "convnet":
        p = synth.convnet_params(seed=1003, batch=8)
        qn = build_convnet(p, dev)
    else:
        p = synth.resnet18_params(seed=1004, batch=2)
        qn = build_resnet18(p, dev)
    x = p["x"].to(dev)
    n = x.shape[0]
    logits = torch.empty((n, qn.out_features), dtype=torch.float32, device=dev)
    qn.workspace(n)
    qn.forward(x, logits)
    torch.cuda.synchronize()
    want = logits.clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        qn.forward(x, logits)
    torch.cuda.synchronize()
    for r in range(4):
        logits.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(logits, want), f"replay {r}"
        # eager work between replays: a forward of other images into another buffer
        other = qn.forward(torch.flip(x, dims=[3]))
        torch.cuda.synchronize()
        assert torch.isfinite(other).all()
