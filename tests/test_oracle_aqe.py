"""CPU pins of the oracle's AQE training steps (Sec. III-B..D; Eqs. ours,
activation, weight; Theorems 1 and 3; Algorithm 1, training branch)."""
import numpy as np
import pytest

import oracle

SPECIAL = np.array([0.0, -0.0, 0.5, -0.5, 0.125, 0.375, 0.75, -0.75, 1.0, -1.0, 1.0000001, -1.0000001,
                    3.0, -7.5, 1e-30, -1e-30, np.inf, -np.inf, np.nan], dtype=np.float32)


def _x(seed, n=4096):
    rng = np.random.default_rng(seed)
    x = rng.normal(0.0, 1.0, n).astype(np.float32)
    x[:SPECIAL.size] = SPECIAL
    return x


@pytest.mark.parametrize("bits", [1, 2, 3])
def test_alpha_one_is_the_quantizer(bits):
    """alpha = 1: the neuron output is h(x) itself (the binary/low-bit neuron)
    for every finite x (0 * inf is NaN in the formula, as in any float form of it)."""
    x = _x(bits)
    want = oracle.levels_f32(oracle.quantize(x, bits), bits)
    fin = np.isfinite(x)
    np.testing.assert_array_equal(oracle.aqe_forward(x, bits, 1.0)[fin], want[fin])
    # the levels are the paper's level sets (Sec. IV-C)
    allowed = {1: {-1.0, 1.0}, 2: {-1.0, 0.0, 1.0}, 3: {0.0, 0.25, 0.5, 1.0, -0.25, -0.5, -1.0}}[bits]
    assert set(np.unique(want).tolist()) <= allowed


@pytest.mark.parametrize("bits", [1, 2, 3])
def test_alpha_zero_is_the_identity(bits):
    """alpha = 0: the full-precision neuron, y = x (NaN stays NaN)."""
    x = _x(10 + bits)
    y = oracle.aqe_forward(x, bits, 0.0)
    fin = np.isfinite(x)
    np.testing.assert_array_equal(y[fin], x[fin])
    assert np.isnan(y[~np.isfinite(x) & np.isnan(x)]).all()


@pytest.mark.parametrize("alpha", [0.1, 0.5, 0.9])
@pytest.mark.parametrize("a1", [0.3, -0.7, 1.0, -0.05])
def test_theorem3_series_closed_form(alpha, a1):
    """Iterating a(n+1) = alpha sign(a(n)) + (1 - alpha) a(n) from a(1) keeps
    the sign and gives a(n+1) = s (1 - (1 - alpha)^n) + (1 - alpha)^n a(1)
    (the series summed in the proof of Theorem 3), which tends to sign(a(1))."""
    s = 1.0 if a1 > 0 else -1.0
    a = np.array([a1], dtype=np.float32)
    for n in range(1, 41):
        a = oracle.aqe_forward(a, 1, alpha)
        closed = s * (1.0 - (1.0 - alpha) ** n) + (1.0 - alpha) ** n * a1
        assert abs(float(a[0]) - closed) <= 2e-6 * n
    assert abs(float(a[0]) - s) < 1e-3 or alpha < 0.2


def test_alpha_half_backward_is_the_ste():
    """Theorem 1: with alpha = 1/2 the AQE gradient is the straight-through
    estimator g 1{|a| <= 1} of Sec. II-B, bit for bit."""
    x = _x(20)
    g = np.random.default_rng(21).normal(0, 1, x.size).astype(np.float32)
    np.testing.assert_array_equal(oracle.aqe_backward(x, g, 0.5), oracle.ste_backward(x, g))


@pytest.mark.parametrize("alpha", [0.0, 0.3, 1.0])
def test_backward_support_and_scale(alpha):
    """The gradient vanishes outside |x| <= 1 (and for NaN inputs) and is
    proportional to 2 alpha inside; at alpha = 0 it is zero everywhere."""
    x = _x(30)
    g = np.ones(x.size, dtype=np.float32)
    gx = oracle.aqe_backward(x, g, alpha)
    inside = np.abs(x) <= 1
    assert (gx[~inside] == 0).all()
    assert np.allclose(gx[inside], 2.0 * alpha)


def test_sgd_clip_invariants():
    rng = np.random.default_rng(40)
    w = rng.uniform(-1, 1, 10000).astype(np.float32)
    g = rng.normal(0, 10, 10000).astype(np.float32)
    v = oracle.sgd_clip(w, g, 0.05)
    assert (v >= -1).all() and (v <= 1).all()
    # a step that stays inside [-1, 1] is the plain step; zero gradient keeps w
    free = np.abs(w.astype(np.float64) - 0.05 * g.astype(np.float64)) < 0.999
    np.testing.assert_allclose(v[free], (w.astype(np.float64) - 0.05 * g.astype(np.float64))[free], rtol=0,
                               atol=1e-6)
    np.testing.assert_array_equal(oracle.sgd_clip(w, np.zeros_like(g), 0.05), w)
    # clipping is idempotent and saturates
    np.testing.assert_array_equal(oracle.sgd_clip(v, np.zeros_like(g), 0.05), v)
    big = oracle.sgd_clip(np.array([0.9, -0.9], np.float32), np.array([-100, 100], np.float32), 1.0)
    np.testing.assert_array_equal(big, np.array([1.0, -1.0], np.float32))


@pytest.mark.parametrize("bits", [2, 3])
def test_weight_forward_uses_the_inference_thresholds(bits):
    """alpha = 1 on weights gives the levels the inference quantizer gives with
    s_c = mean|W_c| (Eq. 20 with thresholds scaled by s_c)."""
    rng = np.random.default_rng(50 + bits)
    w = rng.normal(0, 0.1, (6, 5, 3, 3)).astype(np.float32)
    lv, s = oracle.quantize_weights(w, bits)
    np.testing.assert_array_equal(oracle.aqe_forward_weights(w, bits, 1.0, s), oracle.levels_f32(lv, bits))
