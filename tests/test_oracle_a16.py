"""CPU pins of the oracle's 16-bit-input product (Table I rows with 16-bit
inputs and 1..3-bit weights; Table IV, reduced weights): the IEEE binary16
rounding of the inputs, the exact fp64 sum and the layer epilogue."""
from fractions import Fraction

import numpy as np
import pytest

import oracle


def _bits(x16):
    return np.asarray(x16, np.float16).view(np.uint16)


# IEEE 754 binary16: 1 sign, 5 exponent (bias 15), 10 fraction bits; round to
# nearest, ties to the even significand; overflow past 65504 + half an ulp.
F16_CASES = [
    (1.0, 0x3C00),
    (-2.0, 0xC000),
    (0.5, 0x3800),
    (65504.0, 0x7BFF),                     # largest finite
    (65519.99609375, 0x7BFF),              # just below the overflow midpoint
    (65520.0, 0x7C00),                     # the midpoint rounds to even: +inf
    (-1e6, 0xFC00),
    (2.0 ** -14, 0x0400),                  # smallest normal
    (2.0 ** -24, 0x0001),                  # smallest subnormal
    (2.0 ** -25, 0x0000),                  # tie between 0 and 2^-24: even 0
    (2.0 ** -25 + 2.0 ** -40, 0x0001),     # just above that tie
    (3 * 2.0 ** -25, 0x0002),              # tie between 1 and 2 ulps: even 2
    (1.0 + 2.0 ** -11, 0x3C00),            # tie: even 1.0
    (1.0 + 3 * 2.0 ** -11, 0x3C02),        # tie between 0x3C01 and 0x3C02: even
    (1.0 + 2.0 ** -10, 0x3C01),
    (-0.0, 0x8000),
    (0.1, 0x2E66),                         # 0.0999755859375 is the nearest
    (1.0 / 3.0, 0x3555),                   # 0.333251953125 is the nearest
    (np.inf, 0x7C00),
    (1e-30, 0x0000),
]


@pytest.mark.parametrize("x,want", F16_CASES)
def test_to_f16_is_ieee_binary16(x, want):
    got = int(_bits(oracle.to_f16(np.array([x], np.float32)))[0])
    assert got == want, (x, hex(got), hex(want))


def test_to_f16_nan_and_value_of_bits():
    y = oracle.to_f16(np.array([np.nan], np.float32))
    b = int(_bits(y)[0])
    assert (b & 0x7C00) == 0x7C00 and (b & 0x03FF) != 0
    # decoding the bits by the format's definition gives back the value
    for x, want in F16_CASES:
        e, f, s = (want >> 10) & 0x1F, want & 0x3FF, -1.0 if want >> 15 else 1.0
        if e == 0x1F:
            continue
        v = s * (f * 2.0 ** -24 if e == 0 else (1 + f / 1024) * 2.0 ** (e - 15))
        assert float(oracle.to_f16(np.array([x], np.float32))[0]) == v


def _brute(x16, w, stride, pad):
    """Exact rational sums, by loops (tiny inputs only)."""
    n, cin, h, wd = x16.shape
    cout, _, kh, kw = w.shape
    ho, wo = (h + 2 * pad - kh) // stride + 1, (wd + 2 * pad - kw) // stride + 1
    out = np.empty((n, cout, ho, wo), dtype=object)
    for b in range(n):
        for co in range(cout):
            for oy in range(ho):
                for ox in range(wo):
                    acc = Fraction(0)
                    for ci in range(cin):
                        for ky in range(kh):
                            for kx in range(kw):
                                iy, ix = oy * stride - pad + ky, ox * stride - pad + kx
                                if 0 <= iy < h and 0 <= ix < wd:
                                    acc += Fraction(float(x16[b, ci, iy, ix])) * int(w[co, ci, ky, kx])
                    out[b, co, oy, ox] = acc
    return out


def _levels(rng, shape, bits):
    pool = {1: [-1, 1], 2: [-1, 0, 1], 3: [0, 1, -1, 2, -2, 4, -4]}[bits]
    return rng.choice(pool, size=shape).astype(np.int8)


@pytest.mark.parametrize("bits", [1, 2, 3])
@pytest.mark.parametrize("stride,pad", [(1, 1), (2, 1), (1, 0), (2, 2)])
def test_conv16_acc_is_the_exact_sum(bits, stride, pad):
    rng = np.random.default_rng(7 + bits + 10 * stride + pad)
    x16 = oracle.to_f16(rng.normal(0, 3, (2, 5, 6, 7)).astype(np.float32))
    x16.reshape(-1)[:4] = np.array([2.0 ** -24, -(2.0 ** -20), 60000.0, -0.0], np.float16)
    w = _levels(rng, (3, 5, 3, 3), bits)
    got = oracle.conv16_acc(x16, w, stride, pad)
    want = _brute(x16, w, stride, pad)
    assert got.shape == want.shape
    assert all(Fraction(float(g)) == v for g, v in zip(got.reshape(-1), want.reshape(-1)))
    idx = np.arange(got.size)[::3]
    np.testing.assert_array_equal(oracle.conv16_acc_at(x16, w, idx, stride, pad), got.reshape(-1)[idx])


@pytest.mark.parametrize("bits", [1, 2, 3])
def test_integer_inputs_reduce_to_the_level_product(bits):
    """Integer-valued 16-bit inputs in the code range: the same sum as the
    integer product of the quantized path (zero padding: level 0)."""
    rng = np.random.default_rng(30 + bits)
    a = rng.integers(-4, 5, (2, 37, 9, 8)).astype(np.int8)
    w = _levels(rng, (11, 37, 3, 3), bits)
    got = oracle.conv16_acc(a.astype(np.float16), w, 1, 1)
    np.testing.assert_array_equal(got, oracle.conv_levels(a, w, 1, 1, 0).astype(np.float64))


def test_one_by_one_is_a_matrix_product():
    rng = np.random.default_rng(40)
    x16 = oracle.to_f16(rng.normal(0, 1, (3, 64, 5, 4)).astype(np.float32))
    w = _levels(rng, (10, 64, 1, 1), 3)
    got = oracle.conv16_acc(x16, w)
    want = np.einsum("oc,nchw->nohw", w[:, :, 0, 0].astype(np.float64), x16.astype(np.float64))
    np.testing.assert_array_equal(got, want)  # both exact


def test_linearity_and_constant_border():
    rng = np.random.default_rng(41)
    x16 = oracle.to_f16(rng.normal(0, 1, (1, 8, 6, 6)).astype(np.float32))
    w = _levels(rng, (4, 8, 3, 3), 2)
    y = oracle.conv16_acc(x16, w, 1, 1)
    np.testing.assert_array_equal(oracle.conv16_acc(-x16, w, 1, 1), -y)
    np.testing.assert_array_equal(oracle.conv16_acc((2 * x16.astype(np.float32)).astype(np.float16), w, 1, 1), 2 * y)
    # a constant input c: an output sees c times the sum of its in-image taps
    c = np.float16(0.75)
    yc = oracle.conv16_acc(np.full((1, 8, 6, 6), c, np.float16), w, 1, 1)
    ws = w.astype(np.float64)
    assert yc[0, 2, 0, 0] == float(c) * ws[2, :, 1:, 1:].sum()      # corner: 2x2 taps
    assert yc[0, 1, 0, 3] == float(c) * ws[1, :, 1:, :].sum()       # top edge: 2x3 taps
    assert yc[0, 3, 3, 3] == float(c) * ws[3].sum()                 # interior: all taps


def test_layer_epilogue_on_integer_inputs_is_the_quantized_epilogue():
    """With integer inputs the fp32 accumulator is exact, and the 16-bit
    layer's epilogue is the one of the quantized layers on that integer."""
    rng = np.random.default_rng(50)
    a = rng.integers(-3, 4, (2, 20, 6, 6)).astype(np.int8)
    w = _levels(rng, (9, 20, 3, 3), 3)
    acc = oracle.conv_levels(a, w, 1, 1, 0)
    k = rng.uniform(0.01, 0.1, 9).astype(np.float32)
    b = rng.normal(0, 0.1, 9).astype(np.float32)
    s = rng.uniform(0.01, 0.1, 9).astype(np.float32)
    x16 = a.astype(np.float16)
    z, _ = oracle.qconv16_layer(x16, w, 3, 1, 1, "scale", s=s)
    np.testing.assert_array_equal(z, oracle.epi_scale(acc, s, 2))
    z, lv = oracle.qconv16_layer(x16, w, 3, 1, 1, "bn", k=k, b=b, out_bits=2)
    np.testing.assert_array_equal(z, oracle.epi_bn(acc, k, b, 2))
    np.testing.assert_array_equal(lv, oracle.quantize(oracle.hardtanh(oracle.epi_bn(acc, k, b, 2)), 2))
    z, _ = oracle.qconv16_layer(x16, w, 3, 1, 1, "bn", k=k, b=b, pool=True)
    np.testing.assert_array_equal(z, oracle.epi_bn(oracle.maxpool2_int(acc), k, b, 2))
    r = rng.normal(0, 1, z.shape).astype(np.float32)
    z2, _ = oracle.qconv16_layer(x16, w, 3, 1, 1, "bn", k=k, b=b, pool=True, residual=r)
    np.testing.assert_array_equal(z2, oracle.add(z, r))


# ---------------------------------------------------------------------------
# 1..3-bit inputs with 16-bit weights (Table I rows M x 16)
# ---------------------------------------------------------------------------

def _brute_w16(a, w16, a_bits, stride, pad):
    """Exact rational sums with padding taps at Q(0) (-1 for 1 bit), by loops."""
    n, cin, h, wd = a.shape
    cout, _, kh, kw = w16.shape
    pl = oracle.pad_level(a_bits)
    ho, wo = (h + 2 * pad - kh) // stride + 1, (wd + 2 * pad - kw) // stride + 1
    out = np.empty((n, cout, ho, wo), dtype=object)
    for b in range(n):
        for co in range(cout):
            for oy in range(ho):
                for ox in range(wo):
                    acc = Fraction(0)
                    for ci in range(cin):
                        for ky in range(kh):
                            for kx in range(kw):
                                iy, ix = oy * stride - pad + ky, ox * stride - pad + kx
                                lv = int(a[b, ci, iy, ix]) if 0 <= iy < h and 0 <= ix < wd else pl
                                acc += lv * Fraction(float(w16[co, ci, ky, kx]))
                    out[b, co, oy, ox] = acc
    return out


@pytest.mark.parametrize("a_bits", [1, 2, 3])
@pytest.mark.parametrize("stride,pad", [(1, 1), (2, 1), (1, 0)])
def test_conv16w_acc_is_the_exact_sum(a_bits, stride, pad):
    rng = np.random.default_rng(60 + a_bits + 10 * stride + pad)
    a = _levels(rng, (2, 5, 6, 7), a_bits)
    w16 = oracle.to_f16(rng.normal(0, 0.3, (3, 5, 3, 3)).astype(np.float32))
    w16.reshape(-1)[:3] = np.array([2.0 ** -24, -60000.0, -0.0], np.float16)
    got = oracle.conv16w_acc(a, w16, a_bits, stride, pad)
    want = _brute_w16(a, w16, a_bits, stride, pad)
    assert all(Fraction(float(g)) == v for g, v in zip(got.reshape(-1), want.reshape(-1)))


@pytest.mark.parametrize("a_bits", [1, 2, 3])
def test_integer_weights_reduce_to_the_level_product(a_bits):
    """Integer-valued 16-bit weights in the code range: the integer product
    of the quantized path, padding included."""
    rng = np.random.default_rng(70 + a_bits)
    a = _levels(rng, (2, 37, 9, 8), a_bits)
    w = rng.integers(-4, 5, (11, 37, 3, 3)).astype(np.int8)
    got = oracle.conv16w_acc(a, w.astype(np.float16), a_bits, 1, 1)
    np.testing.assert_array_equal(got, oracle.conv_levels(a, w, 1, 1, oracle.pad_level(a_bits)).astype(np.float64))
