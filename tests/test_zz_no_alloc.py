"""qnet_forward_noalloc (the network entry point for callers that cannot
allocate device memory) against qnet_forward with a caller workspace, through
the C ABI, on the GPU: bit-identical logits on two calls in a row, the second
with a smaller batch, and the refusal of a network that does not fit the
library's fixed scratch array."""
import numpy as np
import pytest
import torch

import paper_2003_04296_amd as q
from paper_2003_04296_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    q.lib()
    return torch.device("cuda:0")


def _both(qn, x, dev):
    """(logits of qnet_forward with a workspace, logits of qnet_forward_noalloc)."""
    n = x.shape[0]
    want = qn.forward(x)
    got = torch.full((n, qn.out_features), float("nan"), dtype=torch.float32, device=dev)
    qn.net.forward_noalloc(x, got)
    torch.cuda.synchronize()
    return want.cpu().numpy(), got.cpu().numpy()


def test_noalloc_convnet_matches_workspace_forward(dev):
    from paper_2003_04296_amd.nets import build_convnet

    p = synth.convnet_params(seed=1003, batch=24)
    qn = build_convnet(p, dev)
    assert 0 < qn.net.noalloc_bytes(24) <= q.lib().qnet_noalloc_limit()
    x = p["x"].to(dev)
    for n in (24, 7):  # the second call reuses the scratch with a smaller batch
        want, got = _both(qn, x[:n].contiguous(), dev)
        np.testing.assert_array_equal(got, want, err_msg=f"batch {n}")


def test_noalloc_resnet18_matches_workspace_forward(dev):
    from paper_2003_04296_amd.nets import build_resnet18

    p = synth.resnet18_params(seed=1004, batch=3)
    qn = build_resnet18(p, dev)
    x = p["x"].to(dev)
    for n in (3, 1):
        want, got = _both(qn, x[:n].contiguous(), dev)
        np.testing.assert_array_equal(got, want, err_msg=f"batch {n}")


def test_noalloc_refuses_networks_past_the_scratch(dev):
    """A batch whose plan exceeds the array returns QCONV_ESCRATCH before any
    launch: the logits buffer keeps its sentinel."""
    from paper_2003_04296_amd.nets import build_resnet18

    p = synth.resnet18_params(seed=1004, batch=1)
    qn = build_resnet18(p, dev)
    limit = q.lib().qnet_noalloc_limit()
    big = 1
    while qn.net.noalloc_bytes(big) <= limit:
        big *= 2
    x = torch.zeros((big, 3, 224, 224), dtype=torch.float32, device=dev)
    logits = torch.full((big, qn.out_features), 7.0, dtype=torch.float32, device=dev)
    with pytest.raises(q.QconvError) as e:
        qn.net.forward_noalloc(x, logits)
    assert e.value.status == q.QCONV_ESCRATCH
    torch.cuda.synchronize()
    assert bool((logits == 7.0).all())
