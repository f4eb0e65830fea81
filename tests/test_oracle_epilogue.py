"""Pins for the oracle's epilogue steps and fp32 support layers -- CPU only.

Rounding is pinned against exact rational arithmetic (Python ``Fraction`` ->
float rounds to nearest-even), pooling against library routines on exact
integers, fp32 layers against float64 within the fp32 chain's error bound."""
from fractions import Fraction

import numpy as np
import pytest
import torch
import torch.nn.functional as F


def _round_f32(fr: Fraction) -> np.float32:
    # float(Fraction) rounds to nearest double; to get a single rounding to
    # float32 we round the exact rational to float32 directly.
    d = float(fr)
    f = np.float32(d)
    # correct a possible double-rounding by checking neighbours exactly
    cands = [np.nextafter(f, np.float32(-np.inf)), f, np.nextafter(f, np.float32(np.inf))]
    best = min(cands, key=lambda c: (abs(Fraction(float(c)) - fr),
                                     int(np.frombuffer(np.float32(c).tobytes(), np.uint32)[0]) & 1))
    return np.float32(best)


def test_bn_epilogue_is_one_rounding(oracle_mod):
    rng = np.random.default_rng(0)
    acc = rng.integers(-4608, 4608, size=(2, 5, 3, 3)).astype(np.int32)
    k = rng.uniform(0.01, 2, 5).astype(np.float32)
    b = rng.normal(0, 1, 5).astype(np.float32)
    for shift in (0, 2, 4):
        z = oracle_mod.epi_bn(acc, k, b, shift)
        for idx in np.ndindex(acc.shape):
            c = idx[1]
            exact = Fraction(float(k[c])) * Fraction(int(acc[idx]), 2 ** shift) + Fraction(float(b[c]))
            assert z[idx] == _round_f32(exact), (idx, shift)


def test_scale_epilogue_is_one_rounding(oracle_mod):
    rng = np.random.default_rng(1)
    acc = rng.integers(-1152, 1152, size=(1, 4, 4, 4)).astype(np.int32)
    s = rng.uniform(0.3, 0.7, 4).astype(np.float32)
    y = oracle_mod.epi_scale(acc, s)
    for idx in np.ndindex(acc.shape):
        exact = Fraction(float(s[idx[1]])) * int(acc[idx])
        assert y[idx] == _round_f32(exact)


def test_bn_fold(oracle_mod):
    rng = np.random.default_rng(2)
    c = 7
    bn = {"gamma": rng.uniform(0.5, 1.5, c).astype(np.float32),
          "beta": rng.normal(0, 0.3, c).astype(np.float32),
          "mean": rng.normal(0, 1, c).astype(np.float32),
          "var": rng.uniform(1, 100, c).astype(np.float32), "eps": 1e-5}
    k, b = oracle_mod.bn_fold(bn)
    kd = bn["gamma"].astype(np.float64) / np.sqrt(bn["var"].astype(np.float64) + 1e-5)
    np.testing.assert_array_equal(k, kd.astype(np.float32))
    np.testing.assert_array_equal(b, (bn["beta"].astype(np.float64) - kd * bn["mean"]).astype(np.float32))


def test_maxpool2_int_matches_library(oracle_mod):
    rng = np.random.default_rng(3)
    acc = rng.integers(-1000, 1000, size=(2, 3, 7, 6)).astype(np.int32)
    want = F.max_pool2d(torch.from_numpy(acc.astype(np.float64)), 2).numpy().astype(np.int32)
    np.testing.assert_array_equal(oracle_mod.maxpool2_int(acc), want)


@pytest.mark.parametrize("bits", [1, 2, 3])
def test_pool_before_bn_commutes_with_monotone_bn(oracle_mod, bits):
    # With k_c > 0, BN then Q is monotone non-decreasing in acc, so pooling
    # the accumulator first equals pooling the quantized levels (Sec. III-E order).
    rng = np.random.default_rng(4)
    acc = rng.integers(-300, 300, size=(2, 4, 6, 6)).astype(np.int32)
    k = rng.uniform(0.001, 0.02, 4).astype(np.float32)
    b = rng.normal(0, 0.5, 4).astype(np.float32)
    q_then_pool = F.max_pool2d(torch.from_numpy(
        oracle_mod.quantize(oracle_mod.epi_bn(acc, k, b), bits).astype(np.float64)), 2).numpy()
    pool_then_q = oracle_mod.quantize(oracle_mod.epi_bn(oracle_mod.maxpool2_int(acc), k, b), bits)
    np.testing.assert_array_equal(pool_then_q, q_then_pool.astype(np.int8))


def test_residual_add_and_relu(oracle_mod):
    rng = np.random.default_rng(5)
    x = rng.normal(0, 1, 1000).astype(np.float32)
    r = rng.normal(0, 1, 1000).astype(np.float32)
    y = oracle_mod.add(x, r)
    for i in range(0, 1000, 37):
        assert y[i] == _round_f32(Fraction(float(x[i])) + Fraction(float(r[i])))
    np.testing.assert_array_equal(oracle_mod.relu(x), np.where(x > 0, x, 0).astype(np.float32))


@pytest.mark.parametrize("case", [(2, 3, 9, 9, 8, 3, 1, 1), (1, 3, 20, 20, 4, 7, 2, 3), (1, 5, 6, 6, 3, 1, 1, 0)])
def test_conv_f32_within_chain_bound_of_float64(oracle_mod, case):
    n, cin, h, w, cout, k, s, p = case
    rng = np.random.default_rng(6)
    x = rng.normal(0, 1, (n, cin, h, w)).astype(np.float32)
    wt = rng.normal(0, 0.3, (cout, cin, k, k)).astype(np.float32)
    ref = F.conv2d(torch.from_numpy(x.astype(np.float64)), torch.from_numpy(wt.astype(np.float64)),
                   stride=s, padding=p).numpy()
    np.testing.assert_allclose(oracle_mod.conv_f64(x, wt, s, p), ref, rtol=1e-12, atol=1e-12)
    y = oracle_mod.conv_f32(x, wt, s, p)
    # |fl(chain) - exact| <= K * u * sum |x||w|   (u = 2^-24, K taps)
    K = cin * k * k
    absref = F.conv2d(torch.from_numpy(np.abs(x).astype(np.float64)),
                      torch.from_numpy(np.abs(wt).astype(np.float64)), stride=s, padding=p).numpy()
    assert np.all(np.abs(y - ref) <= K * 2.0 ** -24 * absref + 1e-30)


def test_fc_f32(oracle_mod):
    rng = np.random.default_rng(7)
    x = rng.normal(0, 1, (3, 50)).astype(np.float32)
    w = rng.normal(0, 0.2, (6, 50)).astype(np.float32)
    b = rng.normal(0, 1, 6).astype(np.float32)
    ref = x.astype(np.float64) @ w.astype(np.float64).T + b
    y = oracle_mod.fc_f32(x, w, b)
    bound = 51 * 2.0 ** -24 * (np.abs(x).astype(np.float64) @ np.abs(w).astype(np.float64).T + np.abs(b))
    assert np.all(np.abs(y - ref) <= bound)


def test_maxpool_f32_and_avgpool(oracle_mod):
    rng = np.random.default_rng(8)
    x = rng.normal(0, 1, (2, 3, 11, 10)).astype(np.float32)
    want = F.max_pool2d(torch.from_numpy(x), 3, 2, 1).numpy()
    np.testing.assert_array_equal(oracle_mod.maxpool_f32(x, 3, 2, 1), want)
    avg = oracle_mod.avgpool_f32(x)
    np.testing.assert_allclose(avg, x.astype(np.float64).mean(axis=(2, 3)), rtol=0, atol=2e-6)
