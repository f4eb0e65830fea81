"""GPU parity of the HIP path against the CPU oracle (run with -m gpu).

Integer results (packed levels, accumulators) must match bit for bit.  The
fp32 epilogues are single-rounding fmaf / multiply / add in both
implementations and must match bit for bit as well (the 1e-3 relative bar is
the floor; exact equality is what is asserted).  Inputs come from the seeded
generators; the oracle quantizes them itself and never sees GPU output."""
import numpy as np
import pytest
import torch

import oracle
import paper_2003_04296_amd as q
from paper_2003_04296_amd import synth
from helpers import tail_bits_zero, unpack_act, unpack_weight, weight_copies

pytestmark = pytest.mark.gpu

BIT_PAIRS = [(1, 1), (2, 1), (1, 2), (2, 2), (3, 3), (3, 1), (1, 3), (3, 2), (2, 3)]  # (a_bits, w_bits)


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    oracle.lib()
    q.lib()
    return torch.device("cuda:0")


def _inputs(seed, n, cin, h, w, cout, k, special=True):
    g = synth.generator(seed)
    x = synth.normal(g, (n, cin, h, w), 1.0)
    wt = synth.normal(g, (cout, cin, k, k), 2.0 / (cin * k * k))
    if special and x.numel() > 16:
        flat = x.view(-1)
        vals = torch.tensor([0.0, -0.0, float("nan"), 0.5, -0.5, 0.125, 0.375, 0.75, -0.75, 1e-40, -1e-40, 3.0])
        flat[:vals.numel()] = vals
    return x, wt


def _bn(seed, cout):
    g = synth.generator(seed + 7)
    k = synth.uniform(g, (cout,), 0.001, 0.05)
    b = synth.normal(g, (cout,), 0.1)
    return k, b


# ---------------------------------------------------------------------------
# quantize + pack
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("bits", [1, 2, 3])
@pytest.mark.parametrize("shape", [(1, 1, 1, 1), (2, 40, 9, 7), (3, 64, 5, 5), (2, 100, 3, 3), (1, 32, 17, 31)])
def test_pack_act_matches_oracle_levels(dev, bits, shape):
    n, c, h, w = shape
    x, _ = _inputs(11, n, c, h, w, 1, 1)
    words = q.pack_act(x.to(dev), bits)
    torch.cuda.synchronize()
    got = unpack_act(words.cpu().numpy(), n, c, h, w, bits)
    np.testing.assert_array_equal(got, oracle.quantize(x.numpy(), bits))
    assert tail_bits_zero(words.cpu().numpy(), c, bits)


@pytest.mark.parametrize("bits", [1, 2, 3])
@pytest.mark.parametrize("shape", [(1, 1, 1, 1), (70, 40, 3, 3), (128, 128, 3, 3), (33, 64, 1, 1), (16, 512, 4, 4)])
def test_pack_weight_matches_oracle(dev, bits, shape):
    cout, cin, kh, kw = shape
    _, w = _inputs(12, 1, cin, 1, 1, cout, kh, special=False)
    words, scale = q.pack_weight(w.to(dev), bits)
    torch.cuda.synchronize()
    lv, s = oracle.quantize_weights(w.numpy(), bits)
    np.testing.assert_array_equal(scale.cpu().numpy(), s)
    np.testing.assert_array_equal(unpack_weight(words.cpu().numpy(), cout, cin, kh, kw, bits), lv)
    # padding rows of the weight layout are zero
    cop = (cout + 127) // 128 * 128
    P = {1: 1, 2: 2, 3: 4}[bits]
    wd = words.cpu().numpy().view(np.uint32)[:kh * kw * ((cin + 31) // 32) * cop * P]
    wd = wd.reshape(kh, kw, (cin + 31) // 32, cop, P)
    assert np.all(wd[:, :, :, cout:, :] == 0)
    # the matrix-core operand copies hold the same levels (0 past cin)
    lv8, lv4 = weight_copies(words.cpu().numpy(), cout, cin, kh, kw, bits)
    np.testing.assert_array_equal(lv8, lv)
    np.testing.assert_array_equal(lv4, lv)
    # ... and 0 in the rows of padding output channels
    raw = words.cpu().numpy().view(np.uint8)
    cw = (cin + 31) // 32
    off = kh * kw * cw * cop * P * 4
    i8 = raw[off:off + kh * kw * cw * cop * 32].reshape(kh, kw, cw, cop, 32)
    f4 = raw[off + i8.size:off + i8.size + kh * kw * ((cw + 1) // 2) * cop * 32].reshape(kh, kw, -1, cop, 32)
    assert np.all(i8[:, :, :, cout:, :] == 0) and np.all(f4[:, :, :, cout:, :] == 0)


# ---------------------------------------------------------------------------
# the quantized product, element by element
# ---------------------------------------------------------------------------

CONV_CASES = [
    # n, cin, h, w, cout, k, stride, pad
    (2, 32, 8, 8, 32, 3, 1, 1),
    (3, 40, 9, 7, 70, 3, 1, 1),     # ragged cin and cout
    (2, 64, 13, 13, 96, 3, 2, 1),   # stride 2
    (1, 33, 7, 7, 40, 1, 2, 0),     # 1x1 stride 2 (ResNet shortcut)
    (2, 96, 6, 6, 33, 4, 1, 0),     # kernel covering a 4x4 map (FC as conv)
    (1, 7, 11, 11, 17, 7, 2, 3),    # 7x7 / 2 pad 3
    (2, 31, 20, 20, 64, 3, 1, 1),   # 800 pixels: several 256-pixel blocks + ragged tail
    (1, 160, 1, 1, 100, 1, 1, 0),   # 1x1 map (FC)
    # shapes aimed at the matrix-core tiling
    (3, 64, 7, 7, 64, 3, 1, 1),     # several whole images per block, ho*wo % 4 != 0
    (6, 256, 14, 14, 130, 3, 1, 1), # two channel chunks, cout padded to 256
    (2, 96, 30, 30, 64, 3, 2, 1),   # stride 2, odd output size
    (2, 64, 56, 56, 64, 3, 1, 1),   # image spans many blocks, blocks span rows
]

ALGOS = {"bitplane": q.ALGO_BITPLANE, "mfma_i8": q.ALGO_MFMA_I8, "mfma_fp4": q.ALGO_MFMA_FP4}


def _run_or_skip(fn):
    try:
        return fn()
    except q.QconvError as e:
        if e.status == q.QCONV_EUNSUPPORTED:
            pytest.skip("configuration not supported by this algorithm")
        raise


def _gpu_conv(dev, x, w, a_bits, w_bits, stride, pad, algo=q.ALGO_AUTO, **epi):
    n, cin, h, ww = x.shape
    cout, _, k, _ = w.shape
    act = q.pack_act(x.to(dev), a_bits)
    wq, scale = q.pack_weight(w.to(dev), w_bits)
    out, outp = q.conv(act, wq, n, cin, h, ww, cout, k, stride, pad, a_bits, w_bits, algo=algo, **epi)
    torch.cuda.synchronize()
    return out, outp, scale


def _oracle_acc(x, w, a_bits, w_bits, stride, pad):
    la = oracle.quantize(x.numpy(), a_bits)
    lw, s = oracle.quantize_weights(w.numpy(), w_bits)
    return oracle.qconv_acc(la, lw, a_bits, stride, pad), s


@pytest.mark.parametrize("algo", list(ALGOS))
@pytest.mark.parametrize("bits", BIT_PAIRS)
@pytest.mark.parametrize("case", CONV_CASES)
def test_conv_int32_bit_exact(dev, bits, case, algo):
    n, cin, h, w, cout, k, s, p = case
    ab, wb = bits
    x, wt = _inputs(100 + sum(case), n, cin, h, w, cout, k)
    out, _, _ = _run_or_skip(lambda: _gpu_conv(dev, x, wt, ab, wb, s, p, algo=ALGOS[algo]))
    want, _ = _oracle_acc(x, wt, ab, wb, s, p)
    np.testing.assert_array_equal(out.cpu().numpy(), want)


def _scale_epi_conv(dev, x, wt, ab, wb, algo):
    n, cin, h, w = x.shape
    cout, _, k, _ = wt.shape
    act = q.pack_act(x.to(dev), ab)
    wq, scale = q.pack_weight(wt.to(dev), wb)
    out, _ = q.conv(act, wq, n, cin, h, w, cout, k, 1, 1, ab, wb, mode=q.EPI_SCALE_F32, scale=scale, algo=algo)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("algo", list(ALGOS))
@pytest.mark.parametrize("bits", [(1, 1), (3, 3)])
def test_scale_epilogue_uses_mean_abs_weight(dev, bits, algo):
    ab, wb = bits
    x, wt = _inputs(6, 2, 40, 9, 9, 70, 3)
    out = _run_or_skip(lambda: _scale_epi_conv(dev, x, wt, ab, wb, ALGOS[algo]))
    acc, s = _oracle_acc(x, wt, ab, wb, 1, 1)
    shift = oracle.level_shift(ab) + oracle.level_shift(wb)
    np.testing.assert_array_equal(out.cpu().numpy(), oracle.epi_scale(acc, s, shift))


@pytest.mark.parametrize("algo", list(ALGOS))
@pytest.mark.parametrize("bits", BIT_PAIRS)
@pytest.mark.parametrize("pool", [False, True])
@pytest.mark.parametrize("out_bits", [0, 1, 2, 3])
def test_bn_epilogues(dev, bits, pool, out_bits, algo):
    """{QConv-[pool]-BN-HardTanh} -> fp32 output, or requantized + packed output."""
    ab, wb = bits
    n, cin, h, w, cout = 2, 40, 10, 9, 70
    x, wt = _inputs(7, n, cin, h, w, cout, 3)
    k, b = _bn(7, cout)
    flags = q.EPI_POOL2 if pool else 0
    mode = q.EPI_BN_PACK if out_bits else q.EPI_BN_F32
    out, outp, _ = _run_or_skip(lambda: _gpu_conv(dev, x, wt, ab, wb, 1, 1, algo=ALGOS[algo], mode=mode, flags=flags,
                                                  bn_k=k.to(dev), bn_b=b.to(dev), out_bits=out_bits))
    acc, _ = _oracle_acc(x, wt, ab, wb, 1, 1)
    if pool:
        acc = oracle.maxpool2_int(acc)
    shift = oracle.level_shift(ab) + oracle.level_shift(wb)
    z = oracle.epi_bn(acc, k.numpy(), b.numpy(), shift)
    if out_bits == 0:
        np.testing.assert_array_equal(out.cpu().numpy(), z)
    else:
        want = oracle.quantize(oracle.hardtanh(z), out_bits)
        got = unpack_act(outp.cpu().numpy(), n, cout, acc.shape[2], acc.shape[3], out_bits)
        np.testing.assert_array_equal(got, want)
        assert tail_bits_zero(outp.cpu().numpy(), cout, out_bits)


@pytest.mark.parametrize("algo", list(ALGOS))
@pytest.mark.parametrize("bits", [(2, 2), (1, 1), (3, 3)])
@pytest.mark.parametrize("hw", [8, 7])
def test_bn_residual_and_repack(dev, bits, algo, hw):
    ab, wb = bits
    n, cin, h, w, cout = 3, 64, hw, hw, 64
    x, wt = _inputs(8, n, cin, h, w, cout, 3)
    k, b = _bn(8, cout)
    g = synth.generator(99)
    res = synth.normal(g, (n, cout, h, w), 1.0)
    act = q.pack_act(x.to(dev), ab)
    wq, _ = q.pack_weight(wt.to(dev), wb)
    outp = torch.empty(q.packed_act_words(n, cout, h, w, ab), dtype=torch.int32, device=dev)
    out, _ = _run_or_skip(lambda: q.conv(act, wq, n, cin, h, w, cout, 3, 1, 1, ab, wb, mode=q.EPI_BN_F32,
                                         flags=q.EPI_RESIDUAL, bn_k=k.to(dev), bn_b=b.to(dev), residual=res.to(dev),
                                         out_bits=ab, out_packed=outp, algo=ALGOS[algo]))
    torch.cuda.synchronize()
    acc, _ = _oracle_acc(x, wt, ab, wb, 1, 1)
    shift = oracle.level_shift(ab) + oracle.level_shift(wb)
    zz = oracle.add(oracle.epi_bn(acc, k.numpy(), b.numpy(), shift), res.numpy())
    np.testing.assert_array_equal(out.cpu().numpy(), zz)
    np.testing.assert_array_equal(unpack_act(outp.cpu().numpy(), n, cout, h, w, ab),
                                  oracle.quantize(oracle.hardtanh(zz), ab))


# ---------------------------------------------------------------------------
# the LDS-tiled XNOR kernel: 1- and 2-bit operands, 1x1 / 3x3, stride 1 / 2,
# unpacked outputs; its K split across 1, 2 or 4 lanes follows the layer size
# ---------------------------------------------------------------------------

XNOR_CASES = [
    # n, cin, h, w, cout, k, stride, pad
    (64, 64, 56, 56, 128, 1, 2, 0),   # ResNet-18 shortcut shape: 1024 blocks
    (16, 128, 32, 32, 128, 3, 1, 1),  # 512 blocks of 64 channels
    (4, 128, 32, 32, 128, 3, 1, 1),   # the 1W1A workload's shape: 256 blocks of 32 channels
    (3, 520, 9, 11, 70, 3, 1, 1),     # several staged chunks of words, ragged tiles and channels
    (2, 33, 30, 30, 40, 3, 2, 1),     # stride 2 with odd halo columns, ragged last word
    (5, 96, 7, 7, 300, 1, 1, 0),      # 1x1 stride 1, three channel tiles
    (3, 70, 27, 27, 50, 1, 2, 0),     # 1x1 stride 2 on 4 x 16 tiles (14 x 14 output), ragged words and channels
    (2, 40, 4, 60, 36, 1, 1, 0),      # 1x1 on 2 x 32 tiles, a ragged last column tile
]


def _xnor_tiles(k, ho, wo):
    """Output tiles of the XNOR kernel: 8 x 8 for 3x3 layers; for 1x1 layers
    the one of 2 x 32, 4 x 16, 8 x 8 with the fewest tiles (widest on ties)."""
    if k != 1:
        return -(-ho // 8) * -(-wo // 8)
    best = None
    for tw in (32, 16, 8):
        t = -(-wo // tw) * -(-ho // (64 // tw))
        if best is None or t < best:
            best = t
    return best


def _expected_ks(case):
    n, cin, h, w, cout, k, s, p = case
    ho, wo = (h + 2 * p - k) // s + 1, (w + 2 * p - k) // s + 1
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    for ks in (1, 2, 4):
        if n * _xnor_tiles(k, ho, wo) * -(-cout // (128 // ks)) >= 2 * cus:
            return ks
    return 4


@pytest.mark.parametrize("bits", [(1, 1), (2, 1), (1, 2), (2, 2)])
@pytest.mark.parametrize("case", XNOR_CASES)
def test_xnor_kernel(dev, case, bits):
    n, cin, h, w, cout, k, s, p = case
    ab, wb = bits
    name = q.kernel_name(n, cin, h, w, cout, k, s, p, ab, wb, algo=q.ALGO_BITPLANE)
    assert name == f"conv_xnor_kernel<{ab}, {wb}, {_expected_ks(case)}>", name
    x, wt = _inputs(900 + sum(case) + ab, n, cin, h, w, cout, k)
    kk, bb = _bn(900 + cin, cout)
    ho, wo = q.out_size(h, k, s, p), q.out_size(w, k, s, p)
    res = synth.normal(synth.generator(901), (n, cout, ho, wo), 1.0)
    act = q.pack_act(x.to(dev), ab)
    wq, scale = q.pack_weight(wt.to(dev), wb)
    conv = lambda **kw: q.conv(act, wq, n, cin, h, w, cout, k, s, p, ab, wb, algo=q.ALGO_BITPLANE, **kw)[0]
    acc = conv()
    sc = conv(mode=q.EPI_SCALE_F32, scale=scale)
    z = conv(mode=q.EPI_BN_F32, bn_k=kk.to(dev), bn_b=bb.to(dev))
    zr = conv(mode=q.EPI_BN_F32, flags=q.EPI_RESIDUAL, bn_k=kk.to(dev), bn_b=bb.to(dev), residual=res.to(dev))
    torch.cuda.synchronize()
    want, s_c = _oracle_acc(x, wt, ab, wb, s, p)
    np.testing.assert_array_equal(acc.cpu().numpy(), want)
    np.testing.assert_array_equal(sc.cpu().numpy(), oracle.epi_scale(want, s_c))
    zw = oracle.epi_bn(want, kk.numpy(), bb.numpy())
    np.testing.assert_array_equal(z.cpu().numpy(), zw)
    np.testing.assert_array_equal(zr.cpu().numpy(), oracle.add(zw, res.numpy()))
    # the matrix cores give the same bits
    other, _ = _run_or_skip(lambda: q.conv(act, wq, n, cin, h, w, cout, k, s, p, ab, wb, algo=q.ALGO_MFMA_FP4))
    assert torch.equal(other, acc)


# ---------------------------------------------------------------------------
# 256-row x 64-channel blocks on layers whose 128-channel blocks would leave
# compute units idle while the 64-channel ones give every CU one
# ---------------------------------------------------------------------------

HALF_CASES = [
    # n, cin, h, w, cout
    (32, 70, 14, 14, 500),  # one 196-pixel image per item, ragged cin and cout
    (130, 64, 7, 7, 640),   # five whole 7x7 images per item, ragged last item
]


@pytest.mark.parametrize("bits", [(2, 2), (3, 3), (1, 1)])
@pytest.mark.parametrize("case", HALF_CASES)
def test_half_width_blocks(dev, bits, case):
    ab, wb = bits
    n, cin, h, w, cout = case
    name = q.kernel_name(n, cin, h, w, cout, 3, 1, 1, ab, wb)
    assert name.startswith("conv_mfma_kernel<") and name.split(", ")[2] == "1", name
    x, wt = _inputs(31, n, cin, h, w, cout, 3)
    k, b = _bn(31, cout)
    act = q.pack_act(x.to(dev), ab)
    wq, _ = q.pack_weight(wt.to(dev), wb)
    acc, _ = q.conv(act, wq, n, cin, h, w, cout, 3, 1, 1, ab, wb)
    outp = torch.empty(q.packed_act_words(n, cout, h, w, ab), dtype=torch.int32, device=dev)
    z, _ = q.conv(act, wq, n, cin, h, w, cout, 3, 1, 1, ab, wb, mode=q.EPI_BN_F32, bn_k=k.to(dev),
                  bn_b=b.to(dev), out_bits=ab, out_packed=outp)
    torch.cuda.synchronize()
    want, _ = _oracle_acc(x, wt, ab, wb, 1, 1)
    np.testing.assert_array_equal(acc.cpu().numpy(), want)
    shift = oracle.level_shift(ab) + oracle.level_shift(wb)
    zz = oracle.epi_bn(want, k.numpy(), b.numpy(), shift)
    np.testing.assert_array_equal(z.cpu().numpy(), zz)
    np.testing.assert_array_equal(unpack_act(outp.cpu().numpy(), n, cout, h, w, ab),
                                  oracle.quantize(oracle.hardtanh(zz), ab))


# ---------------------------------------------------------------------------
# the store-overlapped kernel: two wave groups per block alternate between
# the MFMAs of one item and the stores of the previous one; chosen for
# unpacked, unpooled outputs with at least two items per compute unit
# ---------------------------------------------------------------------------

PP_CASES = [
    # n, cin, h, w, cout, k, stride, pad
    (128, 128, 32, 32, 128, 3, 1, 1),  # 512 items of 256 pixels x 128 channels
    (128, 64, 28, 28, 64, 3, 1, 1),    # 784-pixel images: ragged last item; 64-channel blocks
    (64, 96, 32, 32, 256, 3, 1, 1),    # two channel tiles; cin padded to a whole k-step
    (1023, 64, 16, 16, 128, 3, 2, 1),  # stride 2, two whole images per item, odd batch
]


def _kernel(case, ab, wb, algo, mode=q.EPI_INT32, flags=0):
    n, cin, h, w, cout, k, s, p = case
    return q.kernel_name(n, cin, h, w, cout, k, s, p, ab, wb, mode=mode, flags=flags, algo=algo)


@pytest.mark.parametrize("bits", [(2, 1), (1, 1), (3, 3), (1, 2)])
@pytest.mark.parametrize("case", PP_CASES)
def test_pp_kernel_int32_bit_exact(dev, case, bits):
    n, cin, h, w, cout, k, s, p = case
    ab, wb = bits
    name = _kernel(case, ab, wb, q.ALGO_MFMA_FP4)
    assert name.startswith("conv_mfma_pp_kernel<1,"), name
    x, wt = _inputs(300 + sum(case), n, cin, h, w, cout, k)
    out, _, _ = _gpu_conv(dev, x, wt, ab, wb, s, p, algo=q.ALGO_MFMA_FP4)
    want, _ = _oracle_acc(x, wt, ab, wb, s, p)
    np.testing.assert_array_equal(out.cpu().numpy(), want)


def test_pp_kernel_int8_operands(dev):
    case = PP_CASES[1]
    n, cin, h, w, cout, k, s, p = case
    name = _kernel(case, 2, 2, q.ALGO_MFMA_I8)
    assert name.startswith("conv_mfma_pp_kernel<0,"), name
    x, wt = _inputs(310, n, cin, h, w, cout, k)
    out, _, _ = _gpu_conv(dev, x, wt, 2, 2, s, p, algo=q.ALGO_MFMA_I8)
    want, _ = _oracle_acc(x, wt, 2, 2, s, p)
    np.testing.assert_array_equal(out.cpu().numpy(), want)


@pytest.mark.parametrize("epi", ["scale", "bn", "bn_residual"])
@pytest.mark.parametrize("ci", [1, 2])
def test_pp_kernel_epilogues(dev, ci, epi):
    case = PP_CASES[ci]
    n, cin, h, w, cout, k, s, p = case
    ab, wb = 2, 1
    mode = q.EPI_SCALE_F32 if epi == "scale" else q.EPI_BN_F32
    flags = q.EPI_RESIDUAL if epi == "bn_residual" else 0
    name = _kernel(case, ab, wb, q.ALGO_AUTO, mode=mode, flags=flags)
    assert name.startswith("conv_mfma_pp_kernel<1,"), name
    x, wt = _inputs(320 + ci, n, cin, h, w, cout, k)
    kk, bb = _bn(320 + ci, cout)
    ho, wo = q.out_size(h, k, s, p), q.out_size(w, k, s, p)
    res = synth.normal(synth.generator(321 + ci), (n, cout, ho, wo), 1.0)
    act = q.pack_act(x.to(dev), ab)
    wq, scale = q.pack_weight(wt.to(dev), wb)
    kw = dict(mode=mode, flags=flags)
    if epi == "scale":
        kw["scale"] = scale
    else:
        kw.update(bn_k=kk.to(dev), bn_b=bb.to(dev))
    if flags:
        kw["residual"] = res.to(dev)
    out, _ = q.conv(act, wq, n, cin, h, w, cout, k, s, p, ab, wb, **kw)
    torch.cuda.synchronize()
    acc, sc = _oracle_acc(x, wt, ab, wb, s, p)
    shift = oracle.level_shift(ab) + oracle.level_shift(wb)
    if epi == "scale":
        want = oracle.epi_scale(acc, sc, shift)
    else:
        want = oracle.epi_bn(acc, kk.numpy(), bb.numpy(), shift)
        if flags:
            want = oracle.add(want, res.numpy())
    np.testing.assert_array_equal(out.cpu().numpy(), want)


@pytest.mark.parametrize("bits", [(2, 1), (1, 1), (3, 3), (2, 2)])
@pytest.mark.parametrize("ci", [0, 1, 3])
@pytest.mark.parametrize("resid", [False, True])
def test_pp_kernel_packed_copy(dev, ci, bits, resid):
    """BN (+ residual) fp32 output with the packed Q(HardTanh(z)) of the next
    layer from the same store phase (a network's residual block output and
    the next block's quantized input)."""
    case = PP_CASES[ci]
    n, cin, h, w, cout, k, s, p = case
    ab, wb = bits
    flags = q.EPI_RESIDUAL if resid else 0
    name = q.kernel_name(n, cin, h, w, cout, k, s, p, ab, wb, mode=q.EPI_BN_F32, flags=flags, out_bits=ab,
                         packed_out=True)
    assert name.startswith("conv_mfma_pp_kernel<1,") and name.endswith(f", {ab}>"), name
    x, wt = _inputs(340 + ci + ab, n, cin, h, w, cout, k)
    kk, bb = _bn(340 + ci, cout)
    ho, wo = q.out_size(h, k, s, p), q.out_size(w, k, s, p)
    res = synth.normal(synth.generator(341 + ci), (n, cout, ho, wo), 1.0)
    act = q.pack_act(x.to(dev), ab)
    wq, _ = q.pack_weight(wt.to(dev), wb)
    outp = torch.empty(q.packed_act_words(n, cout, ho, wo, ab), dtype=torch.int32, device=dev)
    out, _ = q.conv(act, wq, n, cin, h, w, cout, k, s, p, ab, wb, mode=q.EPI_BN_F32, flags=flags,
                    bn_k=kk.to(dev), bn_b=bb.to(dev), residual=res.to(dev) if resid else None, out_bits=ab,
                    out_packed=outp)
    torch.cuda.synchronize()
    acc, _ = _oracle_acc(x, wt, ab, wb, s, p)
    z = oracle.epi_bn(acc, kk.numpy(), bb.numpy(), oracle.level_shift(ab) + oracle.level_shift(wb))
    if resid:
        z = oracle.add(z, res.numpy())
    np.testing.assert_array_equal(out.cpu().numpy(), z)
    np.testing.assert_array_equal(unpack_act(outp.cpu().numpy(), n, cout, ho, wo, ab),
                                  oracle.quantize(oracle.hardtanh(z), ab))
    assert tail_bits_zero(outp.cpu().numpy(), cout, ab)


PP_PACK_CASES = [
    # n, cin, h, w, cout, k, stride, pad: stride-2 layers whose base-kernel
    # items are fewer than two per CU, so that a packed output alone takes the
    # store-overlapped kernel (on 64-channel items; stride-1 layers of that
    # size take the base kernel's 64-channel items, three blocks per CU)
    (64, 64, 56, 56, 128, 3, 2, 1),    # ResNet-18's 64 -> 128 stride-2 layer
    (64, 64, 54, 60, 100, 3, 2, 1),    # ragged channels, a 27 x 30 output: ragged last items
    (66, 64, 56, 58, 120, 3, 2, 1),    # odd batch, ragged channels and rows
]


@pytest.mark.parametrize("bits", [(2, 1), (1, 1), (3, 3), (2, 2)])
@pytest.mark.parametrize("ci", [0, 1, 2])
def test_pp_kernel_packed_output(dev, ci, bits):
    """BN -> Q(HardTanh(z)) packed output alone (a network layer feeding only
    the next quantized conv) on the store-overlapped kernel."""
    case = PP_PACK_CASES[ci]
    n, cin, h, w, cout, k, s, p = case
    ab, wb = bits
    name = q.kernel_name(n, cin, h, w, cout, k, s, p, ab, wb, mode=q.EPI_BN_PACK, out_bits=ab, packed_out=True)
    assert name.startswith("conv_mfma_pp_kernel<1,") and name.endswith(f", {ab}>"), name
    x, wt = _inputs(360 + ci + ab, n, cin, h, w, cout, k)
    kk, bb = _bn(360 + ci, cout)
    ho, wo = q.out_size(h, k, s, p), q.out_size(w, k, s, p)
    act = q.pack_act(x.to(dev), ab)
    wq, _ = q.pack_weight(wt.to(dev), wb)
    _, outp = q.conv(act, wq, n, cin, h, w, cout, k, s, p, ab, wb, mode=q.EPI_BN_PACK, bn_k=kk.to(dev),
                     bn_b=bb.to(dev), out_bits=ab)
    torch.cuda.synchronize()
    acc, _ = _oracle_acc(x, wt, ab, wb, s, p)
    z = oracle.epi_bn(acc, kk.numpy(), bb.numpy(), oracle.level_shift(ab) + oracle.level_shift(wb))
    np.testing.assert_array_equal(unpack_act(outp.cpu().numpy(), n, cout, ho, wo, ab),
                                  oracle.quantize(oracle.hardtanh(z), ab))
    assert tail_bits_zero(outp.cpu().numpy(), cout, ab)


STRIDE2_WIDE_CASES = [
    # n, cin, h, w, cout, k, stride, pad: ResNet-18's stride-2 3x3 layers at
    # batch 64, whose 256-row input tiles (twice the input rows of a stride-1
    # tile) are staged in the wide halo buffer
    (64, 64, 56, 56, 128, 3, 2, 1),
    (64, 128, 28, 28, 256, 3, 2, 1),
]


@pytest.mark.parametrize("ci", [0, 1])
def test_stride2_layers_on_256_row_tiles(dev, ci):
    """BN -> packed 2-bit output of the stride-2 layers on 256-row items
    (not the 64-row split-K shape), bit for bit against the oracle."""
    n, cin, h, w, cout, k, s, p = STRIDE2_WIDE_CASES[ci]
    name = q.kernel_name(n, cin, h, w, cout, k, s, p, 2, 2, mode=q.EPI_BN_PACK, out_bits=2, packed_out=True)
    cfg = int(name.split("<")[1].split(",")[2])
    assert cfg != 2, name
    x, wt = _inputs(380 + ci, n, cin, h, w, cout, k)
    kk, bb = _bn(380 + ci, cout)
    ho, wo = q.out_size(h, k, s, p), q.out_size(w, k, s, p)
    act = q.pack_act(x.to(dev), 2)
    wq, _ = q.pack_weight(wt.to(dev), 2)
    _, outp = q.conv(act, wq, n, cin, h, w, cout, k, s, p, 2, 2, mode=q.EPI_BN_PACK, bn_k=kk.to(dev),
                     bn_b=bb.to(dev), out_bits=2)
    torch.cuda.synchronize()
    acc, _ = _oracle_acc(x, wt, 2, 2, s, p)
    z = oracle.epi_bn(acc, kk.numpy(), bb.numpy(), oracle.level_shift(2) + oracle.level_shift(2))
    np.testing.assert_array_equal(unpack_act(outp.cpu().numpy(), n, cout, ho, wo, 2),
                                  oracle.quantize(oracle.hardtanh(z), 2))
    assert tail_bits_zero(outp.cpu().numpy(), cout, 2)


def test_128_channel_layer_takes_64_channel_items_when_128_are_too_few(dev):
    """A 128-channel stride-1 layer whose 256-row x 128-channel items are
    fewer than two per CU runs 256 x 64 items (three blocks per CU) on the
    base kernel, bit-exact; the same layer with stride 2 runs them on the
    store-overlapped kernel (PP_PACK_CASES)."""
    n, cin, h, w, cout = 64, 128, 28, 28, 128
    name = q.kernel_name(n, cin, h, w, cout, 3, 1, 1, 2, 2, mode=q.EPI_BN_PACK, out_bits=2, packed_out=True)
    assert name == "conv_mfma_kernel<1, 2, 1, 1>", name
    x, wt = _inputs(371, n, cin, h, w, cout, 3)
    kk, bb = _bn(371, cout)
    act = q.pack_act(x.to(dev), 2)
    wq, _ = q.pack_weight(wt.to(dev), 2)
    _, outp = q.conv(act, wq, n, cin, h, w, cout, 3, 1, 1, 2, 2, mode=q.EPI_BN_PACK, bn_k=kk.to(dev),
                     bn_b=bb.to(dev), out_bits=2)
    torch.cuda.synchronize()
    acc, _ = _oracle_acc(x, wt, 2, 2, 1, 1)
    z = oracle.epi_bn(acc, kk.numpy(), bb.numpy(), 0)
    np.testing.assert_array_equal(unpack_act(outp.cpu().numpy(), n, cout, h, w, 2),
                                  oracle.quantize(oracle.hardtanh(z), 2))


def test_pp_kernel_repeated_launches_agree(dev):
    """Back-to-back launches on one stream (the second overlapping the first's
    drained stores) give identical outputs, also after an unrelated launch."""
    case = PP_CASES[0]
    n, cin, h, w, cout, k, s, p = case
    x, wt = _inputs(330, n, cin, h, w, cout, k)
    act = q.pack_act(x.to(dev), 2)
    wq, _ = q.pack_weight(wt.to(dev), 1)
    outs = [q.conv(act, wq, n, cin, h, w, cout, k, s, p, 2, 1)[0] for _ in range(3)]
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1]) and torch.equal(outs[0], outs[2])


POOL_CASES = [
    # n, cin, h, w, cout, k, stride, pad -- conv output widths 8, 16, 32, 64
    (3, 40, 8, 8, 70, 3, 1, 1),     # wo 8, two whole images per block, last block half empty
    (1, 32, 9, 8, 33, 3, 1, 1),     # wo 8, odd conv rows: the last one has no pooled row
    (2, 32, 10, 8, 32, 3, 1, 1),    # wo 8, 80-pixel images (one block each)
    (2, 33, 4, 16, 40, 3, 1, 1),    # wo 16, 64-pixel images, two per block
    (2, 64, 16, 16, 96, 3, 1, 1),   # wo 16, two blocks per image
    (1, 64, 32, 32, 128, 3, 1, 1),  # wo 32
    (2, 32, 7, 32, 64, 3, 1, 1),    # wo 32, odd conv rows
    (3, 64, 2, 32, 64, 3, 1, 1),    # wo 32, 2-row images, two per block
    (2, 64, 64, 64, 64, 3, 2, 1),   # wo 32 after stride 2
    (1, 32, 6, 64, 33, 3, 1, 1),    # wo 64: interleaved M-tiles
    (2, 32, 7, 8, 32, 3, 1, 1),     # wo 8 with odd rows and two images per block: bit-serial only
    (2, 40, 10, 9, 70, 3, 1, 1),    # odd width: bit-serial only
]
POOL_ALGOS = dict(ALGOS, auto=q.ALGO_AUTO)


@pytest.mark.parametrize("algo", list(POOL_ALGOS))
@pytest.mark.parametrize("case", POOL_CASES)
def test_pooled_conv_int32(dev, case, algo):
    """2x2 max pooling of the integer accumulator, every pairing of the M-tiles."""
    n, cin, h, w, cout, k, s, p = case
    for ab, wb in [(1, 1), (2, 2), (3, 1)]:
        x, wt = _inputs(300 + sum(case) + ab, n, cin, h, w, cout, k)
        out, _, _ = _run_or_skip(lambda: _gpu_conv(dev, x, wt, ab, wb, s, p, algo=POOL_ALGOS[algo],
                                                   flags=q.EPI_POOL2))
        acc, _ = _oracle_acc(x, wt, ab, wb, s, p)
        np.testing.assert_array_equal(out.cpu().numpy(), oracle.maxpool2_int(acc), err_msg=str((ab, wb)))


@pytest.mark.parametrize("algo", list(POOL_ALGOS))
@pytest.mark.parametrize("case", POOL_CASES)
def test_pooled_conv_bn_pack_and_residual(dev, case, algo):
    """{QConv-pool-BN-HardTanh-quantize} packed; and pool-BN + residual -> fp32 + repack."""
    n, cin, h, w, cout, k, s, p = case
    ab, wb = 1, 2
    x, wt = _inputs(400 + sum(case), n, cin, h, w, cout, k)
    kk, bb = _bn(400 + sum(case), cout)
    acc, _ = _oracle_acc(x, wt, ab, wb, s, p)
    acc = oracle.maxpool2_int(acc)
    ho, wo = acc.shape[2], acc.shape[3]
    shift = oracle.level_shift(ab) + oracle.level_shift(wb)
    z = oracle.epi_bn(acc, kk.numpy(), bb.numpy(), shift)
    for out_bits in (1, 2):
        _, outp, _ = _run_or_skip(lambda: _gpu_conv(dev, x, wt, ab, wb, s, p, algo=POOL_ALGOS[algo],
                                                    mode=q.EPI_BN_PACK, flags=q.EPI_POOL2, bn_k=kk.to(dev),
                                                    bn_b=bb.to(dev), out_bits=out_bits))
        got = unpack_act(outp.cpu().numpy(), n, cout, ho, wo, out_bits)
        np.testing.assert_array_equal(got, oracle.quantize(oracle.hardtanh(z), out_bits))
        assert tail_bits_zero(outp.cpu().numpy(), cout, out_bits)
    res = synth.normal(synth.generator(401), (n, cout, ho, wo), 1.0)
    act = q.pack_act(x.to(dev), ab)
    wq, _ = q.pack_weight(wt.to(dev), wb)
    outp = torch.empty(q.packed_act_words(n, cout, ho, wo, 2), dtype=torch.int32, device=dev)
    out, _ = _run_or_skip(lambda: q.conv(act, wq, n, cin, h, w, cout, k, s, p, ab, wb, mode=q.EPI_BN_F32,
                                         flags=q.EPI_POOL2 | q.EPI_RESIDUAL, bn_k=kk.to(dev), bn_b=bb.to(dev),
                                         residual=res.to(dev), out_bits=2, out_packed=outp,
                                         algo=POOL_ALGOS[algo]))
    torch.cuda.synchronize()
    zz = oracle.add(z, res.numpy())
    np.testing.assert_array_equal(out.cpu().numpy(), zz)
    np.testing.assert_array_equal(unpack_act(outp.cpu().numpy(), n, cout, ho, wo, 2),
                                  oracle.quantize(oracle.hardtanh(zz), 2))


@pytest.mark.parametrize("algo", [q.ALGO_MFMA_FP4, q.ALGO_MFMA_I8])
def test_one_whole_image_per_item(dev, algo):
    """Images small enough for several per 256-row item (128 output pixels)
    whose input tile leaves room for only one: each item is one image, one
    block per image (this plan once produced an empty launch)."""
    n, cin, h, w, cout, k, s, p = 300, 64, 15, 31, 64, 3, 2, 1
    assert q.kernel_name(n, cin, h, w, cout, k, s, p, 2, 1, algo=algo).startswith("conv_mfma_kernel<")
    x, wt = _inputs(31, n, cin, h, w, cout, k)
    out, _, _ = _gpu_conv(dev, x, wt, 2, 1, s, p, algo=algo)
    want, _ = _oracle_acc(x, wt, 2, 1, s, p)
    np.testing.assert_array_equal(out.cpu().numpy(), want)


def test_empty_batch_is_a_no_op(dev):
    x = torch.zeros((0, 32, 4, 4), device=dev)
    act = q.pack_act(x, 1)
    wq, _ = q.pack_weight(torch.ones((32, 32, 3, 3), device=dev), 1)
    out, _ = q.conv(act, wq, 0, 32, 4, 4, 32, 3, 1, 1, 1, 1)
    torch.cuda.synchronize()
    assert out.numel() == 0


def test_deterministic_rerun(dev):
    x, wt = _inputs(9, 4, 128, 16, 16, 128, 3)
    a1, _, _ = _gpu_conv(dev, x, wt, 2, 1, 1, 1)
    a2, _, _ = _gpu_conv(dev, x, wt, 2, 1, 1, 1)
    assert torch.equal(a1, a2)


# ---------------------------------------------------------------------------
# full-size workloads: every output against the oracle
# ---------------------------------------------------------------------------

def test_workload1_full(dev):
    """1W1A, batch 4 x 128 x 32 x 32, 128 out, pad -1: int32 and s_c * acc, every output."""
    case = synth.workload1()
    n, c, h, w = case.x.shape
    act = q.pack_act(case.x.to(dev), 1)
    wq, scale = q.pack_weight(case.w.to(dev), 1)
    acc, _ = q.conv(act, wq, n, c, h, w, 128, 3, 1, 1, 1, 1)
    y, _ = q.conv(act, wq, n, c, h, w, 128, 3, 1, 1, 1, 1, mode=q.EPI_SCALE_F32, scale=scale)
    torch.cuda.synchronize()
    want, s = _oracle_acc(case.x, case.w, 1, 1, 1, 1)
    np.testing.assert_array_equal(acc.cpu().numpy(), want)
    np.testing.assert_array_equal(y.cpu().numpy(), oracle.epi_scale(want, s))


def test_workload2_full(dev):
    """1W2A, batch 256 x 128 x 32 x 32, BN epilogue, in the launch the benchmark
    times: every int32 accumulator and every BN output against the oracle's
    direct convolution of the whole layer."""
    case = synth.workload2()
    n, c, h, w = case.x.shape
    xd = case.x.to(dev)
    act = q.pack_act(xd, 2)
    wq, _ = q.pack_weight(case.w.to(dev), 1)
    k, b = q.fold_bn(*(case.bn[kk].numpy() for kk in ("gamma", "beta", "mean", "var")), case.bn["eps"])
    kd, bd = torch.from_numpy(k).to(dev), torch.from_numpy(b).to(dev)
    z, _ = q.conv(act, wq, n, c, h, w, 128, 3, 1, 1, 2, 1, mode=q.EPI_BN_F32, bn_k=kd, bn_b=bd)
    acc, _ = q.conv(act, wq, n, c, h, w, 128, 3, 1, 1, 2, 1)
    torch.cuda.synchronize()
    la = oracle.quantize(case.x.numpy(), 2)
    lw, _ = oracle.quantize_weights(case.w.numpy(), 1)
    want = oracle.qconv_acc(la, lw, 2, 1, 1)
    np.testing.assert_array_equal(acc.cpu().numpy(), want)
    ok, ob = oracle.bn_fold({kk: (v.numpy() if hasattr(v, "numpy") else v) for kk, v in case.bn.items()})
    np.testing.assert_array_equal(z.cpu().numpy(), oracle.epi_bn(want, ok, ob))
    for algo in (q.ALGO_BITPLANE, q.ALGO_MFMA_I8):
        other, _ = q.conv(act, wq, n, c, h, w, 128, 3, 1, 1, 2, 1, algo=algo)
        assert torch.equal(other, acc), algo
    assert int(acc.abs().max()) <= c * 9


@pytest.mark.parametrize("layer", [0, 1, 2, 3])
def test_workload5_full(dev, layer):
    """3W3A ResNet-18 3x3 layers at batch 256: every int32 accumulator (16 x
    the real dot) against the oracle's direct convolution, and the same bits
    from the other two algorithms."""
    case = synth.workload5(layer)
    n, c, h, w = case.x.shape
    act = q.pack_act(case.x.to(dev), 3)
    wq, _ = q.pack_weight(case.w.to(dev), 3)
    acc, _ = q.conv(act, wq, n, c, h, w, c, 3, 1, 1, 3, 3)
    torch.cuda.synchronize()
    la = oracle.quantize(case.x.numpy(), 3)
    lw, _ = oracle.quantize_weights(case.w.numpy(), 3)
    np.testing.assert_array_equal(acc.cpu().numpy(), oracle.qconv_acc(la, lw, 3, 1, 1))
    for algo in (q.ALGO_BITPLANE, q.ALGO_MFMA_I8):
        other, _ = q.conv(act, wq, n, c, h, w, c, 3, 1, 1, 3, 3, algo=algo)
        assert torch.equal(other, acc), algo
    assert int(acc.abs().max()) <= c * 9 * 16


def test_int8_exact_past_fp32_integer_range(dev):
    """A 3W3A product whose accumulators exceed 2^24 (K = 2^20 + 1): fp4 is
    refused there; the int8 matrix cores (split-K, pooled, int32 output) and
    the bitplane kernel return the exact integers, 2^24 + 1 included."""
    cin, cout = (1 << 20) + 1, 32
    assert q.resolve_algo(1, cin, 2, 2, cout, 1, 1, 0, 3, 3) != q.ALGO_MFMA_FP4
    x = torch.ones((1, cin, 2, 2), dtype=torch.float32)
    x[0, 0] = 0.2  # level 1/4 (code 1) in channel 0
    x[0, 1, 1, 1] = -1.0  # one negative code in the second window position
    wt = torch.ones((cout, cin, 1, 1), dtype=torch.float32)
    wt[:, 0] = 0.2  # code 1
    wt[1::2, 2] = -1.0
    la = oracle.quantize(x.numpy(), 3)
    lw, _ = oracle.quantize_weights(wt.numpy(), 3)
    want = oracle.qconv_acc(la, lw, 3, 1, 0)
    assert int(np.abs(want).max()) > (1 << 24) and (want % 2 == 1).any()
    act = q.pack_act(x.to(dev), 3)
    wq, _ = q.pack_weight(wt.to(dev), 3)
    for algo in (q.ALGO_MFMA_I8, q.ALGO_BITPLANE, q.ALGO_AUTO):
        out, _ = q.conv(act, wq, 1, cin, 2, 2, cout, 1, 1, 0, 3, 3, algo=algo)
        pooled, _ = q.conv(act, wq, 1, cin, 2, 2, cout, 1, 1, 0, 3, 3, flags=q.EPI_POOL2, algo=algo)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(out.cpu().numpy(), want, err_msg=str(algo))
        np.testing.assert_array_equal(pooled.cpu().numpy(), oracle.maxpool2_int(want), err_msg=str(algo))
    del wq, act


# ---------------------------------------------------------------------------
# networks
# ---------------------------------------------------------------------------

def _levels_of(words, shape, bits):
    n, c, h, w = shape
    return unpack_act(words.cpu().numpy(), n, c, h, w, bits)


def test_convnet_layers_and_logits(dev):
    """ConvNet (Model A widths), batch 4: every binary layer's packed output and the
    logits equal the oracle's."""
    from paper_2003_04296_amd.nets import build_convnet

    p = synth.convnet_params(seed=1003, batch=4)
    net = build_convnet(p, dev, f32_algo=q.F32_FMAF_CHAIN)
    logits = net.forward(p["x"].to(dev))
    torch.cuda.synchronize()
    want, levels = oracle.convnet_forward(p, return_levels=True)
    names = ["conv1", "conv2", "conv3", "conv4", "conv5", "conv6", "fc1", "fc2"]
    for name, lv in zip(names, levels):
        tid = net.ids[name]
        words, bits = net.tensor(tid, 4)
        shape = lv.shape if lv.ndim == 4 else (lv.shape[0], lv.shape[1], 1, 1)
        np.testing.assert_array_equal(_levels_of(words, shape, bits).reshape(lv.shape), lv, err_msg=name)
    np.testing.assert_array_equal(logits.cpu().numpy(), want)


def test_convnet_full_batch(dev):
    """Batch 256 on the GPU: every row of the logits equals the oracle's
    network, bit for bit (the fp32 layers follow one fixed fmaf order)."""
    from paper_2003_04296_amd.nets import build_convnet

    p = synth.convnet_params(seed=1003, batch=256)
    net = build_convnet(p, dev, f32_algo=q.F32_FMAF_CHAIN)
    logits = net.forward(p["x"].to(dev)).cpu().numpy()
    want = oracle.convnet_forward(p)
    np.testing.assert_array_equal(logits, want)


def test_resnet18_blocks_and_logits(dev):
    """ResNet-18 2W2A at 224x224, batch 2: the fp32 residual stream after the stem
    and every block, and the logits, equal the oracle's."""
    from paper_2003_04296_amd.nets import build_resnet18

    p = synth.resnet18_params(seed=1004, batch=2)
    net = build_resnet18(p, dev, f32_algo=q.F32_FMAF_CHAIN)
    logits = net.forward(p["x"].to(dev))
    torch.cuda.synchronize()
    want, acts = oracle.resnet18_forward(p, 2, 2, return_acts=True)
    got_stem, _ = net.tensor(net.ids["stem"], 2)
    np.testing.assert_array_equal(got_stem.cpu().numpy(), acts[0])
    for i in range(8):
        if net.ids[f"block{i}"] == net.ids["logits"]:
            continue
        got, _ = net.tensor(net.ids[f"block{i}"], 2)
        np.testing.assert_array_equal(got.cpu().numpy(), acts[i + 1], err_msg=f"block{i}")
    np.testing.assert_array_equal(logits.cpu().numpy(), want)


def test_resnet18_full_batch(dev):
    """Batch 64 at 224 x 224: every row of the logits equals the oracle's."""
    from paper_2003_04296_amd.nets import build_resnet18

    p = synth.resnet18_params(seed=1004, batch=64)
    net = build_resnet18(p, dev, f32_algo=q.F32_FMAF_CHAIN)
    logits = net.forward(p["x"].to(dev)).cpu().numpy()
    want = oracle.resnet18_forward(p, 2, 2)
    np.testing.assert_array_equal(logits, want)


# ---------------------------------------------------------------------------
# fp32 support layers through small qnet graphs
# ---------------------------------------------------------------------------

def _run_net(dev, net, x, out_features):
    ws = torch.empty(max(net.workspace_bytes(x.shape[0]), 1), dtype=torch.uint8, device=dev)
    logits = torch.empty((x.shape[0], out_features), dtype=torch.float32, device=dev)
    net.forward(x.to(dev), logits, ws)
    torch.cuda.synchronize()
    return logits.cpu().numpy()


@pytest.mark.parametrize("n,c,h,w,out,bias", [
    (1, 5, 1, 1, 1, True),        # single image, tiny
    (3, 7, 3, 3, 10, False),      # in = 63 (not a multiple of 4), no bias
    (70, 512, 1, 1, 1000, True),  # ResNet head: two image groups, ragged last group
    (65, 200, 1, 1, 13, True),    # in spans two chunks with a ragged one
    (2, 100, 2, 2, 5, True),      # in = 400: two full chunks + 16
])
def test_fc_f32_fp32_input(dev, n, c, h, w, out, bias):
    g = synth.generator(500 + n + c + out)
    x = synth.normal(g, (n, c, h, w), 1.0)
    wt = synth.normal(g, (out, c * h * w), 2.0 / (c * h * w))
    b = synth.normal(g, (out,), 0.1) if bias else None
    net = q.Net(c, h, w, q.F32_FMAF_CHAIN)
    net.fc_f32(0, wt.to(dev), b.to(dev) if bias else None)
    got = _run_net(dev, net, x, out)
    want = oracle.fc_f32(x.numpy().reshape(n, -1), wt.numpy(), b.numpy() if bias else None)
    np.testing.assert_array_equal(got, want)


@pytest.mark.parametrize("n,c,out", [(256, 1024, 10), (3, 33, 7), (64, 2049, 5), (1, 32, 1), (130, 64, 9)])
def test_fc_f32_binary_input(dev, n, c, out):
    """FC over a packed {-1,+1} vector (ConvNet head); inputs span whole and ragged words and chunks."""
    g = synth.generator(600 + n + c + out)
    x = synth.normal(g, (n, c, 1, 1), 1.0)
    wt = synth.normal(g, (out, c), 2.0 / c)
    b = synth.normal(g, (out,), 0.1)
    net = q.Net(c, 1, 1)
    t = net.quantize(0, 1)
    net.fc_f32(t, wt.to(dev), b.to(dev))
    got = _run_net(dev, net, x, out)
    lv = oracle.quantize(x.numpy(), 1).astype(np.float32).reshape(n, c)
    np.testing.assert_array_equal(got, oracle.fc_f32(lv, wt.numpy(), b.numpy()))


@pytest.mark.parametrize("n,c,h,w", [(3, 300, 7, 7), (2, 129, 1, 1), (5, 100, 6, 10), (2, 70, 61, 1), (1, 257, 8, 8)])
def test_avgpool_head(dev, n, c, h, w):
    """Average pool -> FC, bit-exact: planes of up to 60 values are summed
    from LDS (a ragged last block of planes), larger ones from memory."""
    g = synth.generator(720 + n + c + h * w)
    x = synth.normal(g, (n, c, h, w), 1.0)
    fw = synth.normal(g, (7, c), 2.0 / c)
    net = q.Net(c, h, w, q.F32_FMAF_CHAIN)
    t = net.avgpool(0)
    net.fc_f32(t, fw.to(dev))
    assert net.layer_kernel(0, n) == ("avgpool_lds_kernel" if h * w <= 60 else "avgpool_f32_kernel"), net.layer_kernel(0, n)
    ws = torch.empty(max(net.workspace_bytes(n), 1), dtype=torch.uint8, device=dev)
    logits = torch.empty((n, 7), dtype=torch.float32, device=dev)
    net.forward(x.to(dev), logits, ws)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(logits.cpu().numpy(), oracle.fc_f32(oracle.avgpool_f32(x.numpy()), fw.numpy()))


@pytest.mark.parametrize("pk,ps,pp", [(3, 2, 1), (2, 2, 0), (4, 3, 1)])
@pytest.mark.parametrize("n,cin,hw,cout,k,s,p", [(2, 3, 32, 128, 3, 1, 1), (1, 3, 37, 64, 7, 2, 3), (3, 5, 9, 40, 3, 2, 0),
                                                 (1, 3, 64, 96, 7, 2, 3), (2, 40, 18, 33, 5, 1, 2)])
def test_conv_f32_pools_and_head(dev, n, cin, hw, cout, k, s, p, pk, ps, pp):
    """fp32 conv -> BN -> ReLU -> max pool -> avg pool -> FC, layer by layer
    (several 16 x 16 output tiles with ragged edges, two channel blocks, more
    input channels than one LDS chunk holds for k = 5; pool windows of 3, 2 and
    a generic 4)."""
    g = synth.generator(700 + hw + cout)
    x = synth.normal(g, (n, cin, hw, hw), 1.0)
    wt = synth.normal(g, (cout, cin, k, k), 2.0 / (cin * k * k))
    kk, bb = _bn(700 + hw, cout)
    fw = synth.normal(g, (11, cout), 2.0 / cout)
    net = q.Net(cin, hw, hw, q.F32_FMAF_CHAIN)
    t1 = net.conv_f32(0, wt.to(dev), kk.to(dev), bb.to(dev), stride=s, pad=p, relu=True)
    t2 = net.maxpool_f32(t1, pk, ps, pp)
    t3 = net.avgpool(t2)
    net.fc_f32(t3, fw.to(dev))
    ws = torch.empty(max(net.workspace_bytes(n), 1), dtype=torch.uint8, device=dev)
    logits = torch.empty((n, 11), dtype=torch.float32, device=dev)
    net.forward(x.to(dev), logits, ws)
    torch.cuda.synchronize()

    def view(tid):
        c, h, w, bits, off = net.tensor_info(tid, n)
        return ws[off:off + 4 * n * c * h * w].view(torch.float32).view(n, c, h, w).cpu().numpy()

    y = oracle.conv_f32(x.numpy(), wt.numpy(), s, p)
    z = oracle.relu(oracle.bn_f32(y, kk.numpy(), bb.numpy()))
    np.testing.assert_array_equal(view(t1), z)
    mp = oracle.maxpool_f32(z, pk, ps, pp)
    np.testing.assert_array_equal(view(t2), mp)
    ap = oracle.avgpool_f32(mp)
    np.testing.assert_array_equal(logits.cpu().numpy(), oracle.fc_f32(ap, fw.numpy()))
