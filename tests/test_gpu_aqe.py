"""GPU parity of the AQE training steps (aqe_forward / aqe_backward /
aqe_sgd_clip) against the CPU oracle, bit for bit: every step is a fixed
sequence of single-rounding fp32 operations on both sides.  Run with -m gpu."""
import numpy as np
import pytest
import torch

import oracle
import paper_2003_04296_amd as q
from helpers import unpack_weight

pytestmark = pytest.mark.gpu

SPECIAL = np.array([0.0, -0.0, 0.5, -0.5, 0.125, 0.375, 0.75, -0.75, 1.0, -1.0, 1.0000001, -1.0000001,
                    3.0, -7.5, 1e-30, -1e-30, np.inf, -np.inf, np.nan], dtype=np.float32)


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    oracle.lib()
    q.lib()
    return torch.device("cuda:0")


def _x(seed, n, scale=1.0):
    rng = np.random.default_rng(seed)
    x = (rng.normal(0.0, 1.0, n) * scale).astype(np.float32)
    m = min(n, SPECIAL.size)
    x[:m] = SPECIAL[:m]
    return x


def _dev(a, dev, off):
    """Device copy of a, starting `off` floats into a buffer (unaligned for off % 4 != 0)."""
    buf = torch.zeros(a.size + off, dtype=torch.float32, device=dev)
    buf[off:] = torch.from_numpy(a).to(dev)
    return buf[off:]


SIZES = [(1, 0), (7, 0), (4096, 0), (1000003, 1), (257, 3), (65536, 2)]


@pytest.mark.parametrize("alpha", [0.0, 0.25, 0.5, 0.7, 1.0])
@pytest.mark.parametrize("bits", [1, 2, 3])
@pytest.mark.parametrize("n,off", SIZES)
def test_aqe_forward_activations(dev, bits, alpha, n, off):
    x = _x(100 + n + bits, n)
    y = q.aqe_forward(_dev(x, dev, off), bits, alpha)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(y.cpu().numpy(), oracle.aqe_forward(x, bits, alpha))


@pytest.mark.parametrize("alpha", [0.3, 1.0])
@pytest.mark.parametrize("bits", [1, 2, 3])
@pytest.mark.parametrize("shape", [(64, 32, 3, 3), (33, 17, 1, 1), (5, 3, 7, 7)])
def test_aqe_forward_weights(dev, bits, alpha, shape):
    """Weights: thresholds scaled per output channel by the s_c that
    qconv_pack_weight computes; at alpha = 1 the result is exactly the levels
    the inference path packs."""
    rng = np.random.default_rng(200 + bits + shape[0])
    w = rng.normal(0.0, 0.2, shape).astype(np.float32)
    w.reshape(-1)[:SPECIAL.size - 3] = SPECIAL[:SPECIAL.size - 3]  # finite specials only
    wd = torch.from_numpy(w).to(dev)
    wq, scale = q.pack_weight(wd, bits)
    k = int(np.prod(shape[1:]))
    y = q.aqe_forward(wd, bits, alpha, scale=scale, group_size=k)
    torch.cuda.synchronize()
    s = scale.cpu().numpy()
    np.testing.assert_array_equal(y.cpu().numpy(), oracle.aqe_forward_weights(w, bits, alpha, s))
    if alpha == 1.0:
        lv = unpack_weight(wq.cpu().numpy(), *shape, bits)
        np.testing.assert_array_equal(y.cpu().numpy(), oracle.levels_f32(lv, bits))


@pytest.mark.parametrize("alpha", [0.5, 0.3, 1.0, 0.0])
@pytest.mark.parametrize("n,off", SIZES)
def test_aqe_backward(dev, alpha, n, off):
    x = _x(300 + n, n, 0.8)
    g = _x(301 + n, n, 2.0)
    gx = q.aqe_backward(_dev(x, dev, off), _dev(g, dev, off), alpha)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(gx.cpu().numpy(), oracle.aqe_backward(x, g, alpha))


def test_aqe_backward_in_place(dev):
    x = _x(310, 100000, 0.8)
    g = _x(311, 100000)
    gd = torch.from_numpy(g).to(dev)
    q.aqe_backward(torch.from_numpy(x).to(dev), gd, 0.5, out=gd)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(gd.cpu().numpy(), oracle.ste_backward(x, g))


@pytest.mark.parametrize("lr", [0.01, 0.5, 3.0])
@pytest.mark.parametrize("n,off", SIZES)
def test_aqe_sgd_clip(dev, lr, n, off):
    w = np.random.default_rng(400 + n).uniform(-1.0, 1.0, n).astype(np.float32)
    g = _x(401 + n, n)
    wd = _dev(w, dev, off)
    q.aqe_sgd_clip(wd, _dev(g, dev, off), lr)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(wd.cpu().numpy(), oracle.sgd_clip(w, g, lr))


def test_aqe_empty_and_invalid(dev):
    e = torch.empty(0, dtype=torch.float32, device=dev)
    q.aqe_forward(e, 2, 0.5)
    q.aqe_backward(e, e, 0.5)
    q.aqe_sgd_clip(e, e, 0.1)
    x = torch.zeros(10, dtype=torch.float32, device=dev)
    for bad in (lambda: q.aqe_forward(x, 2, 1.5), lambda: q.aqe_forward(x, 4, 0.5),
                lambda: q.aqe_forward(x, 2, 0.5, scale=torch.ones(3, device=dev), group_size=3),
                lambda: q.aqe_backward(x, x, -0.1), lambda: q.aqe_sgd_clip(x, x, float("nan"))):
        with pytest.raises(q.QconvError) as ei:
            bad()
        assert ei.value.status == q.QCONV_EINVAL


def _mlp_loop_gpu(dev, x, t, w1, w2, alpha, lr, steps):
    x, t = torch.from_numpy(x).to(dev), torch.from_numpy(t).to(dev)
    w1, w2 = torch.from_numpy(w1).to(dev), torch.from_numpy(w2).to(dev)
    for _ in range(steps):
        _, s1 = q.pack_weight(w1.view(*w1.shape, 1, 1), 2)
        _, s2 = q.pack_weight(w2.view(*w2.shape, 1, 1), 2)
        wh1 = q.aqe_forward(w1, 2, alpha, scale=s1, group_size=w1.shape[1])
        wh2 = q.aqe_forward(w2, 2, alpha, scale=s2, group_size=w2.shape[1])
        z1 = x @ wh1.T
        a1 = q.aqe_forward(z1, 2, alpha)
        z2 = a1 @ wh2.T
        gz2 = (z2 - t) / x.shape[0]
        gwh2 = gz2.T @ a1
        ga1 = gz2 @ wh2
        gz1 = q.aqe_backward(z1, ga1, alpha)
        gwh1 = gz1.T @ x
        q.aqe_sgd_clip(w1, q.aqe_backward(w1, gwh1, alpha), lr)
        q.aqe_sgd_clip(w2, q.aqe_backward(w2, gwh2, alpha), lr)
    torch.cuda.synchronize()
    return w1.cpu().numpy(), w2.cpu().numpy()


def _mlp_loop_oracle(x, t, w1, w2, alpha, lr, steps, backward):
    f = lambda a: a.astype(np.float32)  # noqa: E731
    for _ in range(steps):
        wh1 = oracle.aqe_forward_weights(w1[:, :, None, None], 2, alpha, oracle.weight_scale(w1[:, :, None, None]))[:, :, 0, 0]
        wh2 = oracle.aqe_forward_weights(w2[:, :, None, None], 2, alpha, oracle.weight_scale(w2[:, :, None, None]))[:, :, 0, 0]
        z1 = f(x.astype(np.float64) @ wh1.T.astype(np.float64))
        a1 = oracle.aqe_forward(z1, 2, alpha)
        z2 = f(a1.astype(np.float64) @ wh2.T.astype(np.float64))
        gz2 = f((z2.astype(np.float64) - t) / x.shape[0])
        gwh2 = f(gz2.T.astype(np.float64) @ a1)
        ga1 = f(gz2.astype(np.float64) @ wh2)
        gz1 = backward(z1, ga1)
        gwh1 = f(gz1.T.astype(np.float64) @ x)
        w1 = oracle.sgd_clip(w1, backward(w1, gwh1), lr)
        w2 = oracle.sgd_clip(w2, backward(w2, gwh2), lr)
    return w1, w2


@pytest.mark.parametrize("alpha", [0.5, 0.8])
def test_training_loop_algorithm1(dev, alpha):
    """Algorithm 1, training branch, on a two-layer perceptron with 2-bit
    weights and activations, six SGD steps: AQE forward on weights and
    activations, AQE gradients, update + clip.  The GEMMs run in fp32 on the
    GPU (torch) and in fp64 in the oracle loop, so the weights are compared
    within a tolerance; they stay in [-1, 1].  At alpha = 1/2 the oracle loop
    uses the straight-through estimator of Sec. II-B (Theorem 1)."""
    rng = np.random.default_rng(500)
    x = rng.normal(0, 1, (64, 32)).astype(np.float32)
    t = rng.normal(0, 1, (64, 10)).astype(np.float32)
    w1 = rng.uniform(-0.5, 0.5, (48, 32)).astype(np.float32)
    w2 = rng.uniform(-0.5, 0.5, (10, 48)).astype(np.float32)
    g1, g2 = _mlp_loop_gpu(dev, x, t, w1, w2, alpha, 0.05, 6)
    if alpha == 0.5:
        bwd = oracle.ste_backward
    else:
        def bwd(v, g):
            return oracle.aqe_backward(v, g, alpha)
    o1, o2 = _mlp_loop_oracle(x, t, w1, w2, alpha, 0.05, 6, bwd)
    for g, o, w0 in ((g1, o1, w1), (g2, o2, w2)):
        assert np.abs(g).max() <= 1.0
        assert not np.array_equal(g, w0)  # the weights moved
        np.testing.assert_allclose(g, o, rtol=0, atol=2e-5)
