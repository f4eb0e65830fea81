"""The arithmetic behind the bf16x6 fp32 convolution (QNET_F32_BF16X6 in
include/qconv.h), checked on the CPU in exact rational arithmetic: every
finite fp32 value of normal range is the exact sum of three bf16 parts made
by cutting to the leading 8 significant bits twice, and the six partial
products x_i w_j with i + j <= 2 miss x w by less than 2^-20 |x w|.  This
pins the error term that the GPU tests add to the fp32 summation bound."""
from fractions import Fraction

import numpy as np


def _cut(v):
    """v (float32) cut to its top 16 bits: a bf16 value, no larger in magnitude."""
    return (np.asarray(v, np.float32).view(np.uint32) & np.uint32(0xFFFF0000)).view(np.float32)


def _split(x):
    x = np.asarray(x, np.float32)
    p0 = _cut(x)
    r1 = (x - p0).astype(np.float32)
    p1 = _cut(r1)
    p2 = (r1 - p1).astype(np.float32)
    return p0, p1, p2


def _values(seed, n):
    g = np.random.default_rng(seed)
    mant = g.integers(1 << 23, 1 << 24, n)  # full 24-bit significands
    exp = g.integers(-100, 100, n)
    sign = g.choice([-1.0, 1.0], n)
    return (sign * np.ldexp(mant.astype(np.float64), exp - 23)).astype(np.float32)


def test_split_is_exact_and_each_part_is_bf16():
    x = np.concatenate([_values(1, 20000), np.float32([1.0, -3.0, 0.1, 65504.0, 3.0e38, -1.1754944e-38, 0.0])])
    p0, p1, p2 = _split(x)
    for p in (p0, p1, p2):
        assert np.all(p.view(np.uint32) & np.uint32(0xFFFF) == 0)  # representable in bf16
        assert np.all(np.abs(p) <= np.abs(x))
    s = p0.astype(np.float64) + p1.astype(np.float64) + p2.astype(np.float64)
    np.testing.assert_array_equal(s, x.astype(np.float64))
    # the parts shrink by 2^-7 per cut
    nz = x != 0
    assert np.all(np.abs(p1[nz]) < np.abs(x[nz]).astype(np.float64) * 2.0 ** -7)
    assert np.all(np.abs(p2[nz]) < np.abs(x[nz]).astype(np.float64) * 2.0 ** -14)


def test_six_partial_products_miss_by_less_than_2_to_the_minus_20():
    x = _values(2, 3000)
    w = _values(3, 3000)
    xs, ws = _split(x), _split(w)
    worst = Fraction(0)
    for i in range(len(x)):
        xi = [Fraction(float(v[i])) for v in xs]
        wi = [Fraction(float(v[i])) for v in ws]
        exact = Fraction(float(x[i])) * Fraction(float(w[i]))
        six = sum(xi[a] * wi[b] for a in range(3) for b in range(3) if a + b <= 2)
        worst = max(worst, abs(exact - six) / abs(exact))
    assert worst < Fraction(1, 2 ** 20), float(worst)
    assert worst > Fraction(1, 2 ** 30)  # the dropped products are not all zero
