"""The fp32 first convolution on the fp32 matrix cores (run with -m gpu):
conv -> BN -> ReLU, with the 3x3 / 2 max pooling and the next layer's
quantize fused into its epilogue, against the oracle.

The matrix cores sum each output's K = cin * k * k products in their own
order, so the fp32 results are compared with the exact (float64) value of
the oracle's layer within the standard bound of recursive summation in any
order, |err| <= gamma_K * sum |x w| (gamma_K = K u / (1 - K u), u = 2^-24),
carried through the BN scale, plus two ulps of the result for BN's and the
final rounding.  The bf16x6 algorithm splits x and w exactly into three bf16
parts each and drops the products x1 w2, x2 w1 and x2 w2, together below
2^-20 |x w|; its five kept small products sum in their own accumulator
(at most 5K terms, together below 2^-5.9 |x w|, so their rounding stays
below gamma_5K 2^-5.9 sum |x w| < 2^-20.4 sum |x w| for K <= 147) and one
more rounding adds them to the main sum: its bound gains
(2^-19 + u) sum |x w|.  Pooling takes maxima, so a pooled output is within the
largest bound of its window.  A quantized copy may differ from the oracle's
level only where that bound straddles a threshold.  Networks built this way
are checked as the readings for fp32 first layers say: the fp32 layer within
its bound, flips only near thresholds (counted), every later layer exact
given its input (the chained-fmaf networks of test_gpu_parity.py), and the
logits within 1e-3 relative."""
import numpy as np
import pytest
import torch

import oracle
import paper_2003_04296_amd as q
from paper_2003_04296_amd import synth
from helpers import unpack_act

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    oracle.lib()
    q.lib()
    return torch.device("cuda:0")


def _ref(x, w, k, b, s, p, relu, x6=False):
    """(exact conv -> BN -> ReLU in float64, error bound of an fp32 sum in any
    order; x6: plus the bf16x6 split's share)."""
    acc = oracle.conv_f64(x, w, s, p)
    mag = oracle.conv_f64(np.abs(x), np.abs(w), s, p)
    K = w.shape[1] * w.shape[2] * w.shape[3]
    u = 2.0 ** -24
    gamma = K * u / (1 - K * u)
    if x6:
        assert K <= 147
        gamma += 2.0 ** -19 + u
    kk = k.astype(np.float64)[None, :, None, None]
    z = kk * acc + b.astype(np.float64)[None, :, None, None]
    bound = np.abs(kk) * gamma * mag + 4 * u * np.abs(z) + 1e-37
    if relu:
        z = np.maximum(z, 0.0)
    return z, bound


def _pool(v):
    """3x3 / 2 max pooling with pad 1 (padding never wins) of a float64 array."""
    n, c, h, w = v.shape
    ho, wo = (h - 1) // 2 + 1, (w - 1) // 2 + 1
    pad = np.full((n, c, h + 2, w + 2), -np.inf)
    pad[:, :, 1:-1, 1:-1] = v
    out = np.full((n, c, ho, wo), -np.inf)
    for dy in range(3):
        for dx in range(3):
            out = np.maximum(out, pad[:, :, dy:dy + 2 * ho:2, dx:dx + 2 * wo:2])
    return out


def _codes_within(got, z, bound, bits):
    """Every code lies between those of z - bound and z + bound (Q(HardTanh(.))
    is monotone); returns the number that differ from the code of z."""
    lo = oracle.quantize(oracle.hardtanh(np.nextafter((z - bound).astype(np.float32), np.float32(-np.inf))), bits)
    hi = oracle.quantize(oracle.hardtanh(np.nextafter((z + bound).astype(np.float32), np.float32(np.inf))), bits)
    mid = oracle.quantize(oracle.hardtanh(z.astype(np.float32)), bits)
    g = got.astype(np.int32)
    assert ((lo <= g) & (g <= hi)).all(), int((~((lo <= g) & (g <= hi))).sum())
    return int((got != mid).sum())


def _inputs(seed, n, cin, h, w, cout, k):
    g = synth.generator(seed)
    x = synth.normal(g, (n, cin, h, w), 1.0)
    wt = synth.normal(g, (cout, cin, k, k), 2.0 / (cin * k * k))
    kk = synth.uniform(g, (cout,), 0.5, 1.5)
    bb = synth.normal(g, (cout,), 0.1)
    return x, wt, kk, bb


def _view(ws, net, tid, n):
    c, h, w, bits, off = net.tensor_info(tid, n)
    if bits == 0:
        return ws[off:off + 4 * n * c * h * w].view(torch.float32).view(n, c, h, w).cpu().numpy()
    words = n * h * w * ((c + 31) // 32) * {1: 1, 2: 2, 3: 4}[bits]
    return unpack_act(ws[off:off + 4 * words].view(torch.int32).cpu().numpy(), n, c, h, w, bits)


POOLED = [
    # n, cin, h, w, cout, k, stride, pad
    (2, 3, 224, 224, 64, 7, 2, 3),   # the ResNet-18 stem
    (3, 3, 37, 41, 40, 7, 2, 3),     # ragged pooled tiles, a ragged channel tile
    (2, 5, 30, 30, 33, 5, 1, 2),     # stride 1, 15 x 15 pooled outputs
    (2, 1, 29, 31, 36, 7, 2, 3),     # one input channel: an odd count of tap rows
    (2, 2, 40, 33, 64, 7, 2, 2),     # two input channels: an even count
]


def _kernel_name(algo, cin, k, s, pool, ob):
    x6 = algo == q.F32_BF16X6 and pool and k == 7 and s == 2 and cin <= 3
    return f"conv_f32_{'bf16x6' if x6 else 'mfma'}_kernel<{k}, {s}, {pool}, {ob}>"


@pytest.mark.parametrize("algo", [q.F32_MFMA, q.F32_BF16X6])
@pytest.mark.parametrize("case", POOLED)
@pytest.mark.parametrize("bits", [1, 2, 3])
def test_stem_conv_pool_quantize(dev, case, bits, algo):
    n, cin, h, w, cout, k, s, p = case
    x, wt, kk, bb = _inputs(70 + sum(case), n, cin, h, w, cout, k)
    net = q.Net(cin, h, w, algo)
    t1 = net.conv_f32(0, wt.to(dev), kk.to(dev), bb.to(dev), stride=s, pad=p, relu=True)
    t2 = net.maxpool_f32(t1, 3, 2, 1)
    t3 = net.quantize(t2, bits)
    t4 = net.avgpool(t2)
    fw = synth.normal(synth.generator(71), (5, cout), 1.0 / cout)
    net.fc_f32(t4, fw.to(dev))
    assert net.layers[1]["fused_into"] == 0 and net.layers[2]["fused_into"] == 0
    assert net.layer_kernel(0, n) == _kernel_name(algo, cin, k, s, 1, bits), net.layer_kernel(0, n)
    assert net.layer_kernel(1, n) == "" and net.layer_kernel(2, n) == ""
    ws = torch.empty(net.workspace_bytes(n), dtype=torch.uint8, device=dev)
    logits = torch.empty((n, 5), dtype=torch.float32, device=dev)
    net.forward(x.to(dev), logits, ws)
    torch.cuda.synchronize()
    x6 = "bf16x6" in net.layer_kernel(0, n)
    z, bound = _ref(x.numpy(), wt.numpy(), kk.numpy(), bb.numpy(), s, p, True, x6)
    zp, bp = _pool(z), _pool(bound)
    got = _view(ws, net, t2, n)
    assert np.all(np.abs(got.astype(np.float64) - zp) <= bp), float(np.max(np.abs(got - zp) - bp))
    flips = _codes_within(_view(ws, net, t3, n), zp, bp, bits)
    assert flips <= max(1, got.size // 100000), flips


PLAIN = [
    # n, cin, h, w, cout, k, stride, pad, relu, out_bits
    (4, 3, 32, 32, 128, 3, 1, 1, False, 1),   # the ConvNet first layer: BN -> sign, packed
    (2, 3, 20, 36, 70, 3, 1, 1, True, 0),     # fp32 output (+ a fused 2-bit quantize)
    (2, 4, 17, 9, 32, 3, 1, 0, False, 3),     # ragged rows and columns, 3-bit levels
    (3, 5, 40, 21, 40, 5, 1, 2, True, 2),     # 5 x 5 taps, ragged channel tile
    (2, 3, 24, 40, 150, 3, 1, 1, True, 2),    # five channel tiles: a block of four and one of one
    (1, 2, 12, 70, 160, 5, 1, 2, False, 1),   # five full channel tiles, 5 x 5 taps, wide rows
]


@pytest.mark.parametrize("case", PLAIN)
def test_first_conv_matrix_cores(dev, case):
    n, cin, h, w, cout, k, s, p, relu, ob = case
    x, wt, kk, bb = _inputs(80 + sum(case[:8]), n, cin, h, w, cout, k)
    net = q.Net(cin, h, w, q.F32_MFMA)
    t1 = net.conv_f32(0, wt.to(dev), kk.to(dev), bb.to(dev), stride=s, pad=p, relu=relu, out_bits=ob)
    t2 = None
    if ob == 0:
        t2 = net.quantize(t1, 2)
        assert net.layers[1]["fused_into"] == 0
    assert net.layer_kernel(0, n) == f"conv_f32_mfma_kernel<{k}, {s}, 0, {ob or 2}>", net.layer_kernel(0, n)
    # the network's fp32 end: a head over the input image itself
    net.fc_f32(net.avgpool(0), torch.ones((2, cin)).to(dev))
    ws = torch.empty(net.workspace_bytes(n), dtype=torch.uint8, device=dev)
    logits = torch.empty((n, 2), dtype=torch.float32, device=dev)
    net.forward(x.to(dev), logits, ws)
    torch.cuda.synchronize()
    z, bound = _ref(x.numpy(), wt.numpy(), kk.numpy(), bb.numpy(), s, p, relu)
    if ob == 0:
        got = _view(ws, net, t1, n)
        assert np.all(np.abs(got.astype(np.float64) - z) <= bound)
        _codes_within(_view(ws, net, t2, n), z, bound, 2)
    else:
        flips = _codes_within(_view(ws, net, t1, n), z, bound, ob)
        assert flips <= max(1, z.size // 100000), flips


def test_wide_window_falls_back_to_the_chain(dev):
    """A layer whose input window does not fit the matrix-core kernel's LDS
    (here an unpooled stride-2 conv: 8 rows x 32 columns need a 17 x 65
    window per channel) runs the fmaf chain, bit for bit as the oracle."""
    n, cin, h, w, cout, k, s, p = 2, 4, 17, 9, 32, 3, 2, 0
    x, wt, kk, bb = _inputs(90, n, cin, h, w, cout, k)
    net = q.Net(cin, h, w, q.F32_MFMA)
    t1 = net.conv_f32(0, wt.to(dev), kk.to(dev), bb.to(dev), stride=s, pad=p, relu=False, out_bits=0)
    assert net.layer_kernel(0, n).startswith("conv_f32_kernel<"), net.layer_kernel(0, n)
    net.fc_f32(net.avgpool(0), torch.ones((2, cin)).to(dev))
    ws = torch.empty(net.workspace_bytes(n), dtype=torch.uint8, device=dev)
    net.forward(x.to(dev), torch.empty((n, 2), dtype=torch.float32, device=dev), ws)
    torch.cuda.synchronize()
    want = oracle.bn_f32(oracle.conv_f32(x.numpy(), wt.numpy(), s, p), kk.numpy(), bb.numpy())
    np.testing.assert_array_equal(_view(ws, net, t1, n), want)


@pytest.mark.parametrize("algo", [q.F32_MFMA, q.F32_BF16X6])
def test_resnet18_matrix_core_stem(dev, algo):
    """ResNet-18 2W2A (batch 2) with the fused matrix-core stem (fp32 or
    bf16x6 matrix cores): the stem's pooled output within its bound and the
    logits within 1e-3 relative."""
    from paper_2003_04296_amd.nets import build_resnet18

    p = synth.resnet18_params(seed=1004, batch=2)
    qn = build_resnet18(p, dev, f32_algo=algo)
    assert qn.net.layer_kernel(0, 2) == _kernel_name(algo, 3, 7, 2, 1, 2), qn.net.layer_kernel(0, 2)
    logits = qn.forward(p["x"].to(dev)).cpu().numpy()
    st = p["stem"]
    ko, bo = oracle.bn_fold({kk: (v.numpy() if hasattr(v, "numpy") else v) for kk, v in st["bn"].items()})
    z, bound = _ref(p["x"].numpy(), st["w"].numpy(), ko, bo, 2, 3, True, algo == q.F32_BF16X6)
    zp, bp = _pool(z), _pool(bound)
    got, _ = qn.tensor(qn.ids["stem"], 2)
    got = got.cpu().numpy()
    assert np.all(np.abs(got.astype(np.float64) - zp) <= bp)
    want = oracle.resnet18_forward(p, 2, 2)
    err = np.max(np.abs(logits.astype(np.float64) - want)) / np.max(np.abs(want))
    assert err <= 1e-3, err


def test_convnet_matrix_core_first_layer(dev):
    """ConvNet (batch 16) with the matrix-core first layer: its sign levels
    differ from the oracle's only where z lies within the fp32 bound of 0;
    every image without such a flip has logits bit-identical to the oracle's
    (everything after the first layer is exact given its input)."""
    from paper_2003_04296_amd.nets import build_convnet

    p = synth.convnet_params(seed=1003, batch=16)
    qn = build_convnet(p, dev)
    assert qn.net.layer_kernel(0, 16) == "conv_f32_mfma_kernel<3, 1, 0, 1>", qn.net.layer_kernel(0, 16)
    logits = qn.forward(p["x"].to(dev)).cpu().numpy()
    c1 = p["convs"][0]
    ko, bo = oracle.bn_fold({kk: (v.numpy() if hasattr(v, "numpy") else v) for kk, v in c1["bn"].items()})
    z, bound = _ref(p["x"].numpy(), c1["w"].numpy(), ko, bo, 1, 1, False)
    words, bits = qn.tensor(qn.ids["conv1"], 16)
    lv = unpack_act(words.cpu().numpy(), 16, 128, 32, 32, bits)
    _codes_within(lv, z, bound, 1)
    want, levels = oracle.convnet_forward(p, return_levels=True)
    same = np.all((lv == levels[0]).reshape(16, -1), axis=1)
    assert same.sum() >= 8, int(same.sum())
    np.testing.assert_array_equal(logits[same], want[same])
    print(f"first-layer sign flips: {int((lv != levels[0]).sum())} in {16 - int(same.sum())} of 16 images")


@pytest.mark.parametrize("algo", [q.F32_MFMA, q.F32_BF16X6])
def test_stem_wide_exponent_range(dev, algo):
    """Inputs and weights spread over 2^-40 .. 2^40 (every element a full
    24-bit significand at its own scale): the three-way splits stay exact
    at any exponent, so the pooled output still lies within its bound."""
    n, cin, h, w, cout, k, s, p = 2, 3, 45, 47, 40, 7, 2, 3
    x, wt, kk, bb = _inputs(96, n, cin, h, w, cout, k)
    ex = torch.from_numpy(np.random.default_rng(98).integers(-40, 41, x.shape).astype(np.float32))
    ew = torch.from_numpy(np.random.default_rng(99).integers(-20, 21, wt.shape).astype(np.float32))
    x = (x * torch.pow(2.0, ex)).contiguous()
    wt = (wt * torch.pow(2.0, ew)).contiguous()
    net = q.Net(cin, h, w, algo)
    t1 = net.conv_f32(0, wt.to(dev), kk.to(dev), bb.to(dev), stride=s, pad=p, relu=True)
    t2 = net.maxpool_f32(t1, 3, 2, 1)
    net.fc_f32(net.avgpool(t2), torch.ones((2, cout)).to(dev))
    assert net.layer_kernel(0, n) == _kernel_name(algo, cin, k, s, 1, 0), net.layer_kernel(0, n)
    ws = torch.empty(net.workspace_bytes(n), dtype=torch.uint8, device=dev)
    net.forward(x.to(dev), torch.empty((n, 2), dtype=torch.float32, device=dev), ws)
    torch.cuda.synchronize()
    z, bound = _ref(x.numpy(), wt.numpy(), kk.numpy(), bb.numpy(), s, p, True, algo == q.F32_BF16X6)
    zp, bp = _pool(z), _pool(bound)
    got = _view(ws, net, t2, n).astype(np.float64)
    assert np.all(np.isfinite(got))
    assert np.all(np.abs(got - zp) <= bp), float(np.max(np.abs(got - zp) - bp))
