"""Guard bands around every output the library writes (run with -m gpu).

Each output buffer is the middle of a larger allocation whose two guard zones
hold a sentinel word; after the call both zones must be unchanged, so a write
past either end of a documented output (ragged channel tails, packed words,
pooled edges, grid tails, the network's workspace) is caught even where it
would not fault.  Shapes are ragged on purpose."""
import numpy as np
import pytest
import torch

import paper_2003_04296_amd as q
from paper_2003_04296_amd import synth
from paper_2003_04296_amd.nets import build_convnet

pytestmark = pytest.mark.gpu

SENT = 0x7FBADBAD  # a NaN pattern no kernel writes
GUARD = 16384      # words on each side (64 KB)


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    q.lib()
    return torch.device("cuda:0")


class Guarded:
    """words int32 words with guard zones; .view(dtype, shape) is the output."""

    def __init__(self, words, dev):
        self.n = int(words)
        self.buf = torch.full((self.n + 2 * GUARD,), SENT, dtype=torch.int32, device=dev)

    def view(self, dtype=torch.int32, shape=None):
        v = self.buf[GUARD:GUARD + self.n].view(dtype)
        return v.view(shape) if shape is not None else v

    def check(self, what):
        torch.cuda.synchronize()
        b = self.buf.cpu().numpy()
        lo, hi = b[:GUARD], b[GUARD + self.n:]
        assert (lo == SENT).all(), f"{what}: write before the output ({int((lo != SENT).sum())} words)"
        assert (hi == SENT).all(), f"{what}: write past the output ({int((hi != SENT).sum())} words)"


def _x(seed, shape):
    return synth.normal(synth.generator(seed), shape, 1.0)


def _w(seed, shape):
    fan = int(np.prod(shape[1:]))
    return synth.normal(synth.generator(seed), shape, 2.0 / fan)


@pytest.mark.parametrize("bits", [1, 2, 3, 16])
@pytest.mark.parametrize("shape", [(3, 40, 9, 7), (1, 1, 1, 1), (2, 100, 5, 3)])
def test_pack_act(dev, bits, shape):
    n, c, h, w = shape
    g = Guarded(q.packed_act_words(n, c, h, w, bits), dev)
    q.pack_act(_x(1, shape).to(dev), bits, out=g.view())
    g.check(f"pack_act bits {bits} {shape}")


@pytest.mark.parametrize("bits", [1, 2, 3])
@pytest.mark.parametrize("shape", [(70, 40, 3, 3), (1, 1, 1, 1), (130, 33, 1, 1)])
def test_pack_weight(dev, bits, shape):
    cout, cin, kh, kw = shape
    g = Guarded(q.packed_weight_words(cout, cin, kh, kw, bits), dev)
    gs = Guarded(cout, dev)
    w = _w(2, shape).to(dev)
    rc = q.lib().qconv_pack_weight(q._ptr(w), cout, cin, kh, kw, bits, None, q._ptr(g.view()),
                                   q._ptr(gs.view(torch.float32)), None)
    assert rc == 0
    g.check(f"pack_weight {bits} {shape}")
    gs.check(f"pack_weight scale {bits} {shape}")


CONV = [
    # n, cin, h, w, cout, k, stride, pad, a_bits, w_bits
    (3, 40, 9, 7, 70, 3, 1, 1, 2, 1),
    (2, 64, 13, 13, 96, 3, 2, 1, 3, 3),
    (1, 33, 7, 7, 40, 1, 2, 0, 1, 2),
    (128, 64, 28, 28, 64, 3, 1, 1, 2, 1),  # selects the store-overlapped kernel
    (2, 40, 9, 7, 70, 3, 1, 1, 16, 2),     # 16-bit inputs
    (2, 96, 30, 30, 64, 3, 2, 1, 16, 1),   # 16-bit inputs, wide staging when pooled
]
ALGOS = {"auto": q.ALGO_AUTO, "bitplane": q.ALGO_BITPLANE, "i8": q.ALGO_MFMA_I8, "fp4": q.ALGO_MFMA_FP4}


# 16-bit inputs have one algorithm (AUTO resolves to it)
CONV_ALGO = [(c, a) for c in CONV for a in ALGOS if c[8] != 16 or a == "auto"]


@pytest.mark.parametrize("case,algo", CONV_ALGO)
def test_conv_outputs(dev, case, algo):
    n, cin, h, w, cout, k, s, p, ab, wb = case
    x = _x(3, (n, cin, h, w)).to(dev)
    wq, scale = q.pack_weight(_w(4, (cout, cin, k, k)).to(dev), wb)
    act = q.pack_act(x, ab)
    kk = torch.full((cout,), 0.01, device=dev)
    bb = torch.zeros(cout, device=dev)
    ho, wo = q.out_size(h, k, s, p), q.out_size(w, k, s, p)
    a = ALGOS[algo]
    try:
        q.resolve_algo(n, cin, h, w, cout, k, s, p, ab, wb, q.EPI_BN_F32, 0, 0, a)
    except q.QconvError as e:
        assert e.status == q.QCONV_EUNSUPPORTED
        pytest.skip("configuration not supported by this algorithm")
    # unpacked fp32 output (int32 for quantized inputs as well)
    if ab != 16:
        g = Guarded(n * cout * ho * wo, dev)
        q.conv(act, wq, n, cin, h, w, cout, k, s, p, ab, wb, out=g.view(torch.int32, (n, cout, ho, wo)), algo=a)
        g.check(f"int32 {case} {algo}")
    g = Guarded(n * cout * ho * wo, dev)
    q.conv(act, wq, n, cin, h, w, cout, k, s, p, ab, wb, mode=q.EPI_BN_F32, bn_k=kk, bn_b=bb,
           out=g.view(torch.float32, (n, cout, ho, wo)), algo=a)
    g.check(f"bn f32 {case} {algo}")
    # packed output, with and without 2x2 pooling
    for pool in (False, True):
        if pool and (ho < 2 or wo < 2):
            continue
        hp, wp = (ho // 2, wo // 2) if pool else (ho, wo)
        flags = q.EPI_POOL2 if pool else 0
        try:
            q.resolve_algo(n, cin, h, w, cout, k, s, p, ab, wb, q.EPI_BN_PACK, flags, 2, a)
        except q.QconvError:
            continue
        gp = Guarded(q.packed_act_words(n, cout, hp, wp, 2), dev)
        q.conv(act, wq, n, cin, h, w, cout, k, s, p, ab, wb, mode=q.EPI_BN_PACK, flags=flags, bn_k=kk, bn_b=bb,
               out_bits=2, out_packed=gp.view(), algo=a)
        gp.check(f"packed pool={pool} {case} {algo}")


def test_network_workspace_and_logits(dev):
    """A small ConvNet: the workspace and the logits are both guarded."""
    params = synth.convnet_params(seed=9, batch=3, width=0.25, fc_width=0.25)
    net = build_convnet(params, dev)
    n = params["x"].shape[0]
    ws_bytes = net.net.workspace_bytes(n)
    gw = Guarded((ws_bytes + 3) // 4, dev)
    gl = Guarded(n * net.out_features, dev)
    net.net.forward(params["x"].to(dev), gl.view(torch.float32, (n, net.out_features)),
                    gw.view().view(torch.uint8)[:ws_bytes])
    gw.check("qnet workspace")
    gl.check("qnet logits")


@pytest.mark.parametrize("nvals", [1, 7, 4099])
def test_aqe_outputs(dev, nvals):
    x = _x(5, (nvals,)).to(dev)
    g = Guarded(nvals, dev)
    q.aqe_forward(x, 2, 0.5, out=g.view(torch.float32))
    g.check("aqe_forward")
    g = Guarded(nvals, dev)
    q.aqe_backward(x, x, 0.5, out=g.view(torch.float32))
    g.check("aqe_backward")
    g = Guarded(nvals, dev)
    wv = g.view(torch.float32)
    wv.copy_(x.clamp(-1, 1))
    q.aqe_sgd_clip(wv, x, 0.1)
    g.check("aqe_sgd_clip")
