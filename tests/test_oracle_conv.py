"""Pins for the oracle's quantized product (Algorithm 1, inference branch) --
CPU only.

The integer accumulator has a plain definition (a direct convolution over
level codes); it is pinned by a float64 library convolution (exact for these
integers), closed forms, brute force of the XNOR-popcount identity, the
bitplane (shift) decomposition, symmetry and linearity."""
import itertools

import numpy as np
import pytest
import torch
import torch.nn.functional as F

LEVELS = {1: np.array([-1, 1]), 2: np.array([-1, 0, 1]), 3: np.array([0, 1, 2, 4, -1, -2, -4])}


def _rand_levels(rng, shape, bits):
    return rng.choice(LEVELS[bits], size=shape).astype(np.int8)


def _torch_conv(a, w, stride, pad, pad_value):
    x = torch.from_numpy(a.astype(np.float64))
    if pad:
        x = F.pad(x, (pad, pad, pad, pad), value=float(pad_value))
    return F.conv2d(x, torch.from_numpy(w.astype(np.float64)), stride=stride).numpy()


CASES = [
    # n, cin, h, w, cout, k, stride, pad
    (2, 3, 7, 5, 4, 3, 1, 1),
    (1, 33, 6, 6, 5, 3, 2, 1),
    (2, 8, 9, 9, 3, 1, 2, 0),
    (1, 5, 8, 8, 2, 7, 2, 3),
    (3, 16, 4, 4, 6, 4, 1, 0),
    (1, 64, 3, 3, 2, 3, 1, 1),
]


@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("bits", [(1, 1), (2, 1), (2, 2), (3, 3), (1, 3), (3, 2)])
def test_conv_levels_matches_float64_library_conv(oracle_mod, case, bits):
    n, cin, h, w, cout, k, s, p = case
    ab, wb = bits
    rng = np.random.default_rng(hash((case, bits)) % 2**32)
    a = _rand_levels(rng, (n, cin, h, w), ab)
    wt = _rand_levels(rng, (cout, cin, k, k), wb)
    pl = oracle_mod.pad_level(ab)
    got = oracle_mod.qconv_acc(a, wt, ab, s, p)
    want = _torch_conv(a, wt, s, p, pl)
    np.testing.assert_array_equal(got, want.astype(np.int32))


def test_all_ones_closed_form(oracle_mod):
    # All +1 inputs and weights, 3x3 pad 1 with pad level -1:
    # interior K, edges K - 6 Cin, corners K - 10 Cin.
    cin, h = 5, 6
    a = np.ones((1, cin, h, h), np.int8)
    w = np.ones((1, cin, 3, 3), np.int8)
    acc = oracle_mod.qconv_acc(a, w, 1, 1, 1)[0, 0]
    K = 9 * cin
    assert acc[2, 2] == K
    assert acc[0, 2] == acc[2, 0] == acc[h - 1, 3] == acc[3, h - 1] == K - 6 * cin
    assert acc[0, 0] == acc[0, h - 1] == acc[h - 1, 0] == acc[h - 1, h - 1] == K - 10 * cin


def test_xnor_popcount_identity_brute_force(oracle_mod):
    # Every 1-bit 3x3 input (2^9) against every 1-bit 3x3 kernel (2^9), pad 1
    # with pad level -1.  For +-1 vectors: dot = 2 * popcount(xnor) - K.
    pats = np.array(list(itertools.product([0, 1], repeat=9)), np.int8)  # bit 1 <-> +1
    lv = (2 * pats - 1).astype(np.int8)
    a = lv.reshape(512, 1, 3, 3)
    w = lv.reshape(512, 1, 3, 3)
    acc = oracle_mod.qconv_acc(a, w, 1, 1, 1)  # [512 inputs, 512 kernels, 3, 3]
    # bit form of the padded input: padding is bit 0 (level -1)
    padded = np.zeros((512, 5, 5), np.int8)
    padded[:, 1:4, 1:4] = pats.reshape(512, 3, 3)
    wbits = pats.reshape(512, 9)
    for oh in range(3):
        for ow in range(3):
            win = padded[:, oh:oh + 3, ow:ow + 3].reshape(512, 9)
            xnor = 1 - (win[:, None, :] ^ wbits[None, :, :])
            want = 2 * xnor.sum(-1) - 9
            np.testing.assert_array_equal(acc[:, :, oh, ow], want)


def _planes(levels, bits):
    """Bitplanes of the method: sign bit S (1 <-> level > 0) and magnitude
    planes E_j with exponent e_j, so level = (2S - 1) * sum_j 2^e_j E_j."""
    S = (levels > 0).astype(np.int64)
    mag = np.abs(levels.astype(np.int64))
    if bits == 1:
        return S, [(0, np.ones_like(mag))]
    if bits == 2:
        return S, [(0, (mag == 1).astype(np.int64))]
    return S, [(2, (mag == 4).astype(np.int64)), (1, (mag == 2).astype(np.int64)),
               (0, (mag == 1).astype(np.int64))]


@pytest.mark.parametrize("bits", [(1, 1), (2, 1), (1, 2), (2, 2), (3, 3), (3, 1), (2, 3)])
def test_bitplane_shift_decomposition(oracle_mod, bits):
    # Each output is sum_{j,r} 2^(e_j + e_r) * [pc(M) - 2 pc(M & (S_a xor S_w))]
    # with M = E_j^a & E_r^w, counted bit by bit over the receptive field
    # (no padding here).  This is the XNOR/SHIFT form of the product.
    ab, wb = bits
    rng = np.random.default_rng(7)
    a = _rand_levels(rng, (2, 6, 5, 5), ab)
    w = _rand_levels(rng, (3, 6, 3, 3), wb)
    Sa, pa = _planes(a, ab)
    Sw, pw = _planes(w, wb)
    win = lambda t: np.lib.stride_tricks.sliding_window_view(t, (3, 3), axis=(2, 3))  # n,c,oh,ow,3,3
    Sa_w = win(Sa)
    want = np.zeros((2, 3, 3, 3), np.int64)
    for (ea, Ea), (ew, Ew) in itertools.product(pa, pw):
        Ea_w = win(Ea)
        for co in range(3):
            M = Ea_w * Ew[co][None, :, None, None, :, :]
            X = Sa_w ^ Sw[co][None, :, None, None, :, :]
            term = M.sum(axis=(1, 4, 5)) - 2 * (M * X).sum(axis=(1, 4, 5))
            want[:, co] += (1 << (ea + ew)) * term
    np.testing.assert_array_equal(oracle_mod.conv_levels(a, w, 1, 0, 0), want)


@pytest.mark.parametrize("bits", [1, 2, 3])
def test_negating_weights_negates_output(oracle_mod, bits):
    rng = np.random.default_rng(bits)
    a = _rand_levels(rng, (2, 7, 6, 6), bits)
    w = _rand_levels(rng, (4, 7, 3, 3), bits)
    pos = oracle_mod.qconv_acc(a, w, bits, 1, 1)
    neg = oracle_mod.qconv_acc(a, (-w).astype(np.int8), bits, 1, 1)
    np.testing.assert_array_equal(neg, -pos)


@pytest.mark.parametrize("bits", [2, 3])
def test_negating_input_negates_output_zero_pad(oracle_mod, bits):
    rng = np.random.default_rng(10 + bits)
    a = _rand_levels(rng, (2, 7, 6, 6), bits)
    w = _rand_levels(rng, (4, 7, 3, 3), bits)
    np.testing.assert_array_equal(oracle_mod.qconv_acc((-a).astype(np.int8), w, bits, 1, 1),
                                  -oracle_mod.qconv_acc(a, w, bits, 1, 1))


def test_negating_input_with_minus_one_padding(oracle_mod):
    # 1 bit, pad -1: conv(x) + conv(-x) = -2 * (sum of weights over padded taps).
    rng = np.random.default_rng(3)
    a = _rand_levels(rng, (1, 4, 5, 5), 1)
    w = _rand_levels(rng, (3, 4, 3, 3), 1)
    s = oracle_mod.qconv_acc(a, w, 1, 1, 1) + oracle_mod.qconv_acc((-a).astype(np.int8), w, 1, 1, 1)
    pad_mask = np.ones((1, 4, 7, 7))
    pad_mask[:, :, 1:6, 1:6] = 0
    want = -2 * F.conv2d(torch.from_numpy(pad_mask), torch.from_numpy(w.astype(np.float64))).numpy()
    np.testing.assert_array_equal(s, want.astype(np.int32))


def test_linearity_in_input(oracle_mod):
    rng = np.random.default_rng(4)
    x = _rand_levels(rng, (2, 5, 6, 6), 3)
    y = _rand_levels(rng, (2, 5, 6, 6), 3)
    w = _rand_levels(rng, (3, 5, 3, 3), 3)
    lhs = oracle_mod.conv_levels((x + y).astype(np.int8), w, 2, 1, 0)
    rhs = oracle_mod.conv_levels(x, w, 2, 1, 0) + oracle_mod.conv_levels(y, w, 2, 1, 0)
    np.testing.assert_array_equal(lhs, rhs)


def test_sampled_outputs_match_full(oracle_mod):
    rng = np.random.default_rng(5)
    a = _rand_levels(rng, (3, 9, 7, 7), 2)
    w = _rand_levels(rng, (5, 9, 3, 3), 1)
    full = oracle_mod.conv_levels(a, w, 2, 1, 0)
    idx = rng.choice(full.size, 50, replace=False)
    np.testing.assert_array_equal(oracle_mod.conv_levels_at(a, w, idx, 2, 1, 0), full.ravel()[idx])


def test_int32_overflow_is_reported(oracle_mod):
    # 127 * 127 * 133200 > 2^31 - 1: the oracle refuses instead of wrapping.
    cin = 133200
    a = np.full((1, cin, 1, 1), 127, np.int8)
    w = np.full((1, cin, 1, 1), 127, np.int8)
    with pytest.raises(OverflowError):
        oracle_mod.conv_levels(a, w, 1, 0, 0)
