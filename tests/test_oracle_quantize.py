"""Pins for the oracle's quantizers (Sec. III-C, Eqs. 4, 20-22) -- CPU only.

Each check is fixed by the paper or by mathematics, not by re-running the
oracle's own formula: the printed level sets, the sign tie rule, the "<="
ties, nearest-level rounding by brute force, odd symmetry and scale
invariance of the weight thresholds."""
import math
import os
from fractions import Fraction

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "levels.txt")


def _golden_levels():
    out = {}
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        bits, vals = line.split(":")
        out[int(bits)] = sorted(Fraction(v) for v in vals.split())
    return out


def _sweep():
    xs = np.linspace(-3, 3, 20001, dtype=np.float32)
    special = np.array([0.0, -0.0, 1e-45, -1e-45, 0.125, 0.375, 0.5, 0.75, 1.0, -1.0, 3e38, -3e38,
                        np.inf, -np.inf], np.float32)
    return np.concatenate([xs, special])


@pytest.mark.parametrize("bits", [1, 2, 3])
def test_level_sets_match_paper(oracle_mod, bits):
    gold = _golden_levels()[bits]
    codes = oracle_mod.quantize(_sweep(), bits)
    scale = 4 if bits == 3 else 1
    got = sorted({Fraction(int(c), scale) for c in np.unique(codes)})
    assert got == gold


def test_sign_tie_rule(oracle_mod):
    # Sec. II-A: +1 only for a positive input, -1 otherwise.
    x = np.array([0.0, -0.0, np.nan, 1e-45, -1e-45, np.inf, -np.inf], np.float32)
    assert oracle_mod.quantize(x, 1).tolist() == [-1, -1, -1, 1, -1, 1, -1]


def test_ternary_threshold_is_inclusive(oracle_mod):
    d = np.float32(0.5)
    up = np.nextafter(d, np.float32(np.inf))
    x = np.array([d, -d, up, -up, 0.0], np.float32)
    assert oracle_mod.quantize(x, 2).tolist() == [0, 0, 1, -1, 0]


def _nearest_level_code(x: float) -> int:
    """Brute force: nearest of {0, +-1/4, +-1/2, +-1}, ties to the smaller
    magnitude, everything beyond 1 saturates; returned as 4x code."""
    levels = [Fraction(0), Fraction(1, 4), Fraction(1, 2), Fraction(1)]
    ax = Fraction(abs(float(x)))
    best = min(levels, key=lambda L: (abs(ax - L), L))
    code = int(best * 4)
    return code if x > 0 else -code


def test_pow2_quantizer_rounds_to_nearest_level(oracle_mod):
    grid = np.concatenate([np.linspace(-1.5, 1.5, 6001, dtype=np.float32),
                           np.array([0.125, 0.375, 0.75, -0.125, -0.375, -0.75], np.float32)])
    for m in (0.125, 0.375, 0.75):
        f = np.float32(m)
        grid = np.concatenate([grid, [np.nextafter(f, np.float32(0)), np.nextafter(f, np.float32(2))]])
    got = oracle_mod.quantize(grid.astype(np.float32), 3)
    want = np.array([_nearest_level_code(v) for v in grid], np.int8)
    np.testing.assert_array_equal(got, want)


@pytest.mark.parametrize("bits", [2, 3])
def test_odd_symmetry(oracle_mod, bits):
    x = _sweep()
    x = x[np.isfinite(x)]
    np.testing.assert_array_equal(oracle_mod.quantize(-x, bits), -oracle_mod.quantize(x, bits))


def test_sign_odd_symmetry_away_from_zero(oracle_mod):
    x = _sweep()
    x = x[np.isfinite(x) & (x != 0)]
    np.testing.assert_array_equal(oracle_mod.quantize(-x, 1), -oracle_mod.quantize(x, 1))


@pytest.mark.parametrize("bits", [1, 2, 3])
def test_hardtanh_before_quantizer_is_identity(oracle_mod, bits):
    # Every threshold is < 1, so Q(HardTanh(z)) == Q(z) (Sec. III-E order).
    z = _sweep()
    np.testing.assert_array_equal(oracle_mod.quantize(oracle_mod.hardtanh(z), bits),
                                  oracle_mod.quantize(z, bits))


def test_weight_scale_is_mean_abs(oracle_mod):
    rng = np.random.default_rng(0)
    w = rng.standard_normal((16, 8, 3, 3)).astype(np.float32)
    s = oracle_mod.weight_scale(w)
    exact = [float(sum(Fraction(float(v)) for v in np.abs(w[c]).ravel()) / w[c].size) for c in range(16)]
    for c in range(16):
        # double accumulation then one rounding to float: within 1 float ulp of the exact mean
        assert abs(float(s[c]) - exact[c]) <= np.spacing(np.float32(exact[c]))


def test_weight_scale_counts_every_weight(oracle_mod):
    # Integer-valued weights: every partial sum and the total are exact in
    # double, so s_c is the exact mean, rounded by the one division and the
    # one conversion to float.  K = 37 * 3 * 3 = 333 is not a multiple of the
    # 256 partial sums (a dropped or doubled tail element changes the mean);
    # an all-zero channel and a channel of one large weight close the set.
    rng = np.random.default_rng(3)
    w = rng.integers(-1000, 1001, size=(6, 37, 3, 3)).astype(np.float32)
    w[2] = 0.0
    w[3] = 0.0
    w[3, 36, 2, 2] = -(2.0 ** 40)
    s = oracle_mod.weight_scale(w)
    for c in range(6):
        total = int(np.abs(w[c]).astype(np.float64).sum())  # exact: integers far below 2^53
        mean = Fraction(total, w[c].size)
        assert s[c] == np.float32(float(mean)), (c, s[c], float(mean))


@pytest.mark.parametrize("bits", [2, 3])
def test_weight_thresholds_scale_with_channel(oracle_mod, bits):
    # Thresholds are relative to s_c: scaling a channel by 2^k leaves its levels unchanged.
    rng = np.random.default_rng(1)
    w = rng.standard_normal((8, 4, 3, 3)).astype(np.float32)
    scaled = w.copy()
    for c in range(8):
        scaled[c] *= np.float32(2.0 ** (c - 4))
    a, s1 = oracle_mod.quantize_weights(w, bits)
    b, s2 = oracle_mod.quantize_weights(scaled, bits)
    np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(s2, s1 * (2.0 ** (np.arange(8) - 4)).astype(np.float32))


def test_weight_ternary_threshold_is_07_mean_abs(oracle_mod):
    # A channel of values {+-a, +-b} with mean |w| = 1: |w| <= 0.7 -> 0, else sign.
    w = np.array([[0.7, -0.7, 1.3, -1.3, 0.69, 1.31, -0.71, -1.29]], np.float32).reshape(1, 8, 1, 1)
    w[0, :, 0, 0] *= np.float32(1.0)
    lv, s = oracle_mod.quantize_weights(w, 2)
    mean = float(np.abs(w).astype(np.float64).mean())
    thr = 0.7 * mean
    want = [0 if abs(float(v)) <= np.float32(thr) else int(math.copysign(1, v)) for v in w.ravel()]
    assert lv.ravel().tolist() == want
    assert lv.ravel().tolist().count(0) >= 2


def test_pad_levels(oracle_mod):
    # The padding tap holds Q(0): -1 for the sign quantizer, 0 otherwise.
    assert [oracle_mod.pad_level(b) for b in (1, 2, 3)] == [-1, 0, 0]


def test_hardtanh_clamps_to_unit_interval(oracle_mod):
    """HardTanh (Sec. III-E) is max(-1, min(1, x)): evaluated here with Python's
    own float min/max on a sweep through +-1, one ulp either side of +-1, the
    extremes, infinities and signed zeros; NaN passes through."""
    one = np.float32(1)
    pts = [0.0, -0.0, 0.5, -0.5, 1.0, -1.0, 2.0, -2.0, 1e-45, -1e-45, 3e38, -3e38, np.inf, -np.inf,
           np.nextafter(one, np.float32(2)), np.nextafter(one, np.float32(0)),
           np.nextafter(-one, np.float32(-2)), np.nextafter(-one, np.float32(0))]
    x = np.concatenate([np.array(pts, np.float32), np.linspace(-4, 4, 4001, dtype=np.float32)])
    got = oracle_mod.hardtanh(x)
    want = np.array([max(-1.0, min(1.0, float(v))) for v in x], np.float32)
    np.testing.assert_array_equal(got, want)
    # signed zeros are kept (no clamp applies to them)
    assert np.signbit(oracle_mod.hardtanh(np.array([-0.0], np.float32))[0])
    assert not np.signbit(oracle_mod.hardtanh(np.array([0.0], np.float32))[0])
    # values inside [-1, 1] are returned unchanged, values outside land exactly on the bound
    inside = x[np.abs(x) <= 1]
    np.testing.assert_array_equal(oracle_mod.hardtanh(inside), inside)
    assert set(np.unique(got[np.abs(x) > 1]).tolist()) == {-1.0, 1.0}
    nan = oracle_mod.hardtanh(np.array([np.nan], np.float32))
    assert np.isnan(nan[0])


def _pow2_channel(scale_exp: int, rng):
    """One output channel of 3-bit test weights whose mean |w| is exactly
    2^scale_exp: a dyadic grid over [-1.5, 1.5] (in units of the scale, so it
    holds the midpoints 1/8, 3/8, 3/4 of adjacent levels exactly), the
    neighbours one ulp either side of each midpoint in pairs whose |sum| is
    exact, and one balancing weight that makes sum |w| = K * 2^scale_exp."""
    s = 2.0 ** scale_exp
    grid = [i / 64 for i in range(-96, 97)]
    pts = []
    for m in (0.125, 0.375, 0.75):
        mf = np.float32(m)
        up = float(np.nextafter(mf, np.float32(2))) - m
        dn = m - float(np.nextafter(mf, np.float32(0)))
        # m + up and k copies of m - dn with up == k * dn sum to an exact dyadic value
        k = int(round(up / dn))
        pts += [m + up] + [m - dn] * k
        pts += [-(m + up)] + [-(m - dn)] * k
    units = grid + pts
    rng.shuffle(units)
    total = sum(abs(Fraction(u)) for u in units)
    kk = len(units) + 1
    bal = Fraction(kk) - total
    assert bal >= 0
    units.append(float(bal))
    w = np.array([u * s for u in units], np.float32)
    assert sum(abs(Fraction(float(v))) for v in w) == Fraction(kk) * Fraction(s)
    return w


def test_pow2_weight_thresholds_round_to_nearest_scaled_level(oracle_mod):
    """3-bit weights (Eq. 22 with thresholds t * s_c): brute force in exact
    rationals, each weight goes to the nearest of {0, +-s/4, +-s/2, +-s}
    (s = mean |W_c|), ties to the smaller magnitude, saturating at s.  With s a
    power of two every threshold t * s is exact in fp32, so the oracle must
    agree on every weight, the exact midpoints and their fp32 neighbours
    included.  A wrong base threshold (any value other than 1/8, 3/8, 3/4)
    moves a grid point to another level."""
    rng = np.random.default_rng(7)
    chans = [_pow2_channel(e, rng) for e in (-5, -1, 0, 3)]
    kk = chans[0].size
    w = np.stack(chans).reshape(len(chans), kk, 1, 1)
    lv, s = oracle_mod.quantize_weights(w, 3)
    for c, e in enumerate((-5, -1, 0, 3)):
        assert float(s[c]) == 2.0 ** e
        sc = Fraction(2) ** e
        levels = [Fraction(0), sc / 4, sc / 2, sc]
        for i in range(kk):
            v = float(w[c, i, 0, 0])
            a = abs(Fraction(v))
            best = min(levels, key=lambda L: (abs(a - L), L))
            code = int(best / sc * 4)
            want = code if v > 0 else -code
            assert int(lv[c, i, 0, 0]) == want, (c, v)
