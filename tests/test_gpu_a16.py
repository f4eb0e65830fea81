"""GPU parity of the 16-bit-input layer (fp16 activations x 1..3-bit
weights on the fp16 matrix cores; Table I rows with 16-bit inputs, Table IV
reduced-weight rows) against the CPU oracle.  Run with -m gpu.

The conversion to fp16 and the weight codes are compared bit for bit.  The
product is exact except for its fp32 accumulation, whose order the matrix
cores fix, so:
  * integer-valued inputs (every partial sum an integer below 2^24) must match
    the oracle bit for bit, through every epilogue;
  * other inputs must match within the bound of any fp32 summation order of
    K terms, gamma_K * sum|x * code| with gamma_K = K u / (1 - K u),
    u = 2^-24, carried through the epilogue's scale (plus the ulps of the
    epilogue's own roundings, which a different accumulator can flip);
    quantized outputs must match except where the oracle's value lies within
    that bound of a quantizer threshold, where either code is correct."""
import numpy as np
import pytest
import torch

import oracle
import paper_2003_04296_amd as q
from paper_2003_04296_amd import synth
from helpers import unpack_act, unpack_act16, unpack_weight, weight_copy_f16

pytestmark = pytest.mark.gpu

U = 2.0 ** -24


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    oracle.lib()
    q.lib()
    return torch.device("cuda:0")


SPECIAL16 = torch.tensor([0.0, -0.0, 1.0 + 2.0 ** -11, 1.0 + 3 * 2.0 ** -11, 65504.0, 65520.0, -1e6, 2.0 ** -24,
                          2.0 ** -25, 3 * 2.0 ** -25, 1e-30, 0.1, float("nan"), float("inf"), -float("inf"),
                          65519.99609375])


def _x(seed, shape, special=False, integer=False):
    g = synth.generator(seed)
    if integer:
        x = torch.floor(synth.uniform(g, shape, -4.0, 5.0))
    else:
        x = synth.normal(g, shape, 1.0)
    if special and x.numel() > SPECIAL16.numel():
        x.view(-1)[:SPECIAL16.numel()] = SPECIAL16
    return x


def _w(seed, cout, cin, k):
    g = synth.generator(seed + 1)
    return synth.normal(g, (cout, cin, k, k), 2.0 / (cin * k * k))


def _bn(seed, cout):
    g = synth.generator(seed + 7)
    return synth.uniform(g, (cout,), 0.001, 0.05), synth.normal(g, (cout,), 0.1)


# ---------------------------------------------------------------------------
# fp32 -> fp16 inputs and the fp16 weight copy
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("shape", [(1, 1, 1, 1), (2, 40, 9, 7), (3, 64, 5, 5), (2, 100, 3, 3), (1, 32, 17, 31)])
def test_pack_act16_is_ieee_binary16(dev, shape):
    n, c, h, w = shape
    x = _x(5, shape, special=True)
    words = q.pack_act(x.to(dev), 16)
    torch.cuda.synchronize()
    assert words.numel() * 4 == n * h * w * ((c + 31) // 32) * 64
    got, pad_ok = unpack_act16(words.cpu().numpy(), n, c, h, w)
    want = oracle.to_f16(x.numpy())
    assert pad_ok
    nan = np.isnan(want)
    np.testing.assert_array_equal(np.isnan(got), nan)
    np.testing.assert_array_equal(got.view(np.uint16)[~nan], want.view(np.uint16)[~nan])


@pytest.mark.parametrize("bits", [1, 2, 3])
@pytest.mark.parametrize("shape", [(1, 1, 1, 1), (70, 40, 3, 3), (128, 128, 3, 3), (33, 64, 1, 1), (16, 512, 4, 4)])
def test_pack_weight_f16_copy(dev, bits, shape):
    cout, cin, kh, kw = shape
    w = _w(12, cout, cin, kh)
    words, _ = q.pack_weight(w.to(dev), bits)
    torch.cuda.synchronize()
    lv, _ = oracle.quantize_weights(w.numpy(), bits)
    wn = words.cpu().numpy()
    np.testing.assert_array_equal(unpack_weight(wn, cout, cin, kh, kw, bits), lv)
    np.testing.assert_array_equal(weight_copy_f16(wn, cout, cin, kh, kw, bits), lv)
    # padding channels (past cin, past cout) of the copy are +0
    cw = (cin + 31) // 32
    cop = (cout + 127) // 128 * 128
    P = {1: 1, 2: 2, 3: 4}[bits]
    off = kh * kw * cw * cop * (P * 4 + 32) + kh * kw * ((cw + 1) // 2) * cop * 32
    h = wn.view(np.uint8)[off:off + kh * kw * 2 * cw * cop * 32].view(np.uint16).reshape(kh, kw, 2 * cw, cop, 16)
    assert np.all(h[:, :, :, cout:, :] == 0)
    full = np.moveaxis(h, 2, 3).reshape(kh, kw, cop, 2 * cw * 16)
    assert np.all(full[:, :, :, cin:] == 0)


# ---------------------------------------------------------------------------
# the layer
# ---------------------------------------------------------------------------

CASES = [
    # n, cin, h, w, cout, k, stride, pad
    (2, 32, 8, 8, 32, 3, 1, 1),
    (3, 40, 9, 7, 70, 3, 1, 1),     # ragged cin and cout
    (2, 64, 13, 13, 96, 3, 2, 1),   # stride 2
    (1, 33, 7, 7, 40, 1, 2, 0),     # 1x1 stride 2
    (2, 96, 6, 6, 33, 4, 1, 0),     # kernel covering a 4x4 map
    (1, 7, 11, 11, 17, 7, 2, 3),    # 7x7 / 2 pad 3
    (2, 31, 20, 20, 64, 3, 1, 1),   # several 256-pixel blocks + ragged tail
    (1, 160, 1, 1, 100, 1, 1, 0),   # 1x1 map
    (3, 64, 7, 7, 64, 3, 1, 1),     # several whole images per block
    (6, 256, 14, 14, 130, 3, 1, 1), # eight channel chunks, cout padded to 256
    (2, 96, 30, 30, 64, 3, 2, 1),   # stride 2, odd output size
    (2, 64, 56, 56, 64, 3, 1, 1),   # image spans many blocks
    (4, 128, 32, 32, 128, 3, 1, 1), # the 32x32 layer shape of the benchmark
]


def _layer(dev, x, w, w_bits, stride, pad, **epi):
    n, cin, h, ww = x.shape
    cout, _, k, _ = w.shape
    act = q.pack_act(x.to(dev), 16)
    wq, scale = q.pack_weight(w.to(dev), w_bits)
    out, outp = q.conv(act, wq, n, cin, h, ww, cout, k, stride, pad, 16, w_bits, **epi)
    torch.cuda.synchronize()
    return out, outp, scale


def _dev(t, dev):
    return None if t is None else torch.as_tensor(t).to(dev)


def _supported(case, w_bits, mode, flags=0, out_bits=0):
    """Whether the library takes this 16-bit layer.  Tiles too large for the
    usual staging buffers use wide ones, so every case here must be taken;
    the only refusal the library may give is for an input tile beyond those
    (wide rows with pooling after a stride-2 conv)."""
    n, cin, h, w, cout, k, stride, pad = case
    try:
        algo = q.resolve_algo(n, cin, h, w, cout, k, stride, pad, 16, w_bits, mode, flags, out_bits)
    except q.QconvError as e:
        assert e.status == q.QCONV_EUNSUPPORTED
        assert flags & q.EPI_POOL2 and stride == 2 and w >= 24, case  # no other shape may be refused
        return False
    assert algo == q.ALGO_MFMA_F16
    return True


@pytest.mark.parametrize("w_bits", [1, 2, 3])
@pytest.mark.parametrize("case", CASES)
def test_integer_inputs_bit_exact(dev, case, w_bits):
    """Integer-valued inputs: the fp32 accumulator is exact, so every
    epilogue matches the oracle bit for bit."""
    n, cin, h, w, cout, k, stride, pad = case
    x = _x(100 + cin + w_bits, (n, cin, h, w), integer=True)
    wt = _w(101 + cout, cout, cin, k)
    x16 = oracle.to_f16(x.numpy())
    lw, s = oracle.quantize_weights(wt.numpy(), w_bits)
    A = oracle.conv16_acc(x16, lw, stride, pad)
    kk, bb = _bn(cout, cout)
    ones = torch.ones(cout)
    # scale 1: the accumulator itself (real units)
    out, _, _ = _layer(dev, x, wt, w_bits, stride, pad, mode=q.EPI_SCALE_F32, scale=_dev(ones, dev))
    z, _ = oracle.qconv16_layer(x16, lw, w_bits, stride, pad, "scale", s=ones.numpy(), acc=A)
    np.testing.assert_array_equal(out.cpu().numpy(), z)
    # scale s_c as packed
    act = q.pack_act(x.to(dev), 16)
    wq, scale = q.pack_weight(wt.to(dev), w_bits)
    out, _ = q.conv(act, wq, n, cin, h, w, cout, k, stride, pad, 16, w_bits, mode=q.EPI_SCALE_F32, scale=scale)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(scale.cpu().numpy(), s)
    z, _ = oracle.qconv16_layer(x16, lw, w_bits, stride, pad, "scale", s=s, acc=A)
    np.testing.assert_array_equal(out.cpu().numpy(), z)
    # BN, BN + fp32 residual, BN + packed requantization (with and without pooling)
    zb, _ = oracle.qconv16_layer(x16, lw, w_bits, stride, pad, "bn", k=kk.numpy(), b=bb.numpy(), acc=A)
    r = synth.normal(synth.generator(7), zb.shape, 1.0)
    out, _ = q.conv(act, wq, n, cin, h, w, cout, k, stride, pad, 16, w_bits, mode=q.EPI_BN_F32,
                    flags=q.EPI_RESIDUAL, bn_k=_dev(kk, dev), bn_b=_dev(bb, dev), residual=_dev(r, dev))
    torch.cuda.synchronize()
    zr, _ = oracle.qconv16_layer(x16, lw, w_bits, stride, pad, "bn", k=kk.numpy(), b=bb.numpy(), residual=r.numpy(), acc=A)
    np.testing.assert_array_equal(out.cpu().numpy(), zr)
    ho, wo = zb.shape[2], zb.shape[3]
    for pool in ([False, True] if ho >= 2 and wo >= 2 else [False]):
        for ob in (1, 2, 3):
            flags = q.EPI_POOL2 if pool else 0
            if not _supported(case, w_bits, q.EPI_BN_F32, flags, ob):
                continue
            out, outp = q.conv(act, wq, n, cin, h, w, cout, k, stride, pad, 16, w_bits, mode=q.EPI_BN_F32,
                               flags=flags, bn_k=_dev(kk, dev), bn_b=_dev(bb, dev), out_bits=ob,
                               out_packed=torch.empty(q.packed_act_words(n, cout, ho // 2 if pool else ho,
                                                                         wo // 2 if pool else wo, ob),
                                                      dtype=torch.int32, device=dev))
            torch.cuda.synchronize()
            zp, lv = oracle.qconv16_layer(x16, lw, w_bits, stride, pad, "bn", k=kk.numpy(), b=bb.numpy(),
                                          pool=pool, out_bits=ob, acc=A)
            np.testing.assert_array_equal(out.cpu().numpy(), zp)
            np.testing.assert_array_equal(unpack_act(outp.cpu().numpy(), n, cout, zp.shape[2], zp.shape[3], ob), lv)


def _bound(x16, lw, w_bits, stride, pad, kabs, pool=False):
    """gamma_K * sum|x * code| carried through the scale k_c 2^-shift."""
    cin, kh, kw = lw.shape[1:]
    K = cin * kh * kw
    g = K * U / (1 - K * U)
    S = oracle.conv16_acc(np.abs(x16.astype(np.float32)).astype(np.float16), np.abs(lw.astype(np.int32)), stride, pad)
    if pool:
        S = oracle.maxpool_f32(S.astype(np.float32), 2, 2, 0).astype(np.float64)
    return (g + U) * S * (kabs[None, :, None, None] * 2.0 ** -oracle.level_shift(w_bits))


def _close(got, want, bound, extra_ulps_of=None):
    ref = np.abs(want) if extra_ulps_of is None else np.maximum(np.abs(want), np.abs(extra_ulps_of))
    tol = bound + 4 * np.spacing(ref.astype(np.float32)).astype(np.float64)
    err = np.abs(got.astype(np.float64) - want.astype(np.float64))
    bad = ~(err <= tol)
    assert not bad.any(), (int(bad.sum()), float(err[bad].max()), float(tol[bad].min()))


def _codes_valid(got, want, z, bound, bits):
    """Codes equal, except where z lies within `bound` of a threshold; there
    the GPU code must be one the quantizer gives to some value within the
    bound of z: Q(HardTanh(.)) is monotone, so it lies between the codes of
    z - bound and z + bound (each widened by one fp32 ulp outwards)."""
    z64 = z.astype(np.float64)
    b64 = np.broadcast_to(bound, z.shape).astype(np.float64)
    lo_z = np.nextafter((z64 - b64).astype(np.float32), np.float32(-np.inf))
    hi_z = np.nextafter((z64 + b64).astype(np.float32), np.float32(np.inf))
    lo = oracle.quantize(oracle.hardtanh(lo_z), bits).astype(np.int32)
    hi = oracle.quantize(oracle.hardtanh(hi_z), bits).astype(np.int32)
    g = got.astype(np.int32)
    diff = got != want
    assert ((lo <= g) & (g <= hi)).all(), int((diff & ~((lo <= g) & (g <= hi))).sum())
    # a differing code only where the bound straddles a threshold
    assert not (diff & (lo == hi)).any(), int((diff & (lo == hi)).sum())
    assert diff.mean() < 1e-3


@pytest.mark.parametrize("w_bits", [1, 2, 3])
@pytest.mark.parametrize("case", CASES)
def test_random_inputs_within_the_accumulation_bound(dev, case, w_bits):
    n, cin, h, w, cout, k, stride, pad = case
    x = _x(200 + cin + w_bits, (n, cin, h, w))
    wt = _w(201 + cout, cout, cin, k)
    x16 = oracle.to_f16(x.numpy())
    lw, s = oracle.quantize_weights(wt.numpy(), w_bits)
    A = oracle.conv16_acc(x16, lw, stride, pad)
    kk, bb = _bn(cout + 1, cout)
    act = q.pack_act(x.to(dev), 16)
    wq, scale = q.pack_weight(wt.to(dev), w_bits)
    out, _ = q.conv(act, wq, n, cin, h, w, cout, k, stride, pad, 16, w_bits, mode=q.EPI_SCALE_F32, scale=scale)
    torch.cuda.synchronize()
    z, _ = oracle.qconv16_layer(x16, lw, w_bits, stride, pad, "scale", s=s, acc=A)
    _close(out.cpu().numpy(), z, _bound(x16, lw, w_bits, stride, pad, np.abs(s)))
    zb, _ = oracle.qconv16_layer(x16, lw, w_bits, stride, pad, "bn", k=kk.numpy(), b=bb.numpy(), acc=A)
    r = synth.normal(synth.generator(8), zb.shape, 1.0)
    out, _ = q.conv(act, wq, n, cin, h, w, cout, k, stride, pad, 16, w_bits, mode=q.EPI_BN_F32,
                    flags=q.EPI_RESIDUAL, bn_k=_dev(kk, dev), bn_b=_dev(bb, dev), residual=_dev(r, dev))
    torch.cuda.synchronize()
    zr, _ = oracle.qconv16_layer(x16, lw, w_bits, stride, pad, "bn", k=kk.numpy(), b=bb.numpy(), residual=r.numpy(), acc=A)
    bnd = _bound(x16, lw, w_bits, stride, pad, np.abs(kk.numpy()))
    _close(out.cpu().numpy(), zr, bnd, extra_ulps_of=zb)
    ho, wo = zb.shape[2], zb.shape[3]
    pool = ho >= 2 and wo >= 2
    ob = 1 + (cin % 3)
    if pool and not _supported(case, w_bits, q.EPI_BN_F32, q.EPI_POOL2, ob):
        pool = False
    hp, wp = (ho // 2, wo // 2) if pool else (ho, wo)
    out, outp = q.conv(act, wq, n, cin, h, w, cout, k, stride, pad, 16, w_bits, mode=q.EPI_BN_F32,
                       flags=q.EPI_POOL2 if pool else 0, bn_k=_dev(kk, dev), bn_b=_dev(bb, dev), out_bits=ob,
                       out_packed=torch.empty(q.packed_act_words(n, cout, hp, wp, ob), dtype=torch.int32, device=dev))
    torch.cuda.synchronize()
    zp, lv = oracle.qconv16_layer(x16, lw, w_bits, stride, pad, "bn", k=kk.numpy(), b=bb.numpy(), pool=pool,
                                  out_bits=ob, acc=A)
    bp = _bound(x16, lw, w_bits, stride, pad, np.abs(kk.numpy()), pool=pool)
    _close(out.cpu().numpy(), zp, bp)
    _codes_valid(unpack_act(outp.cpu().numpy(), n, cout, hp, wp, ob), lv, zp, bp, ob)


def test_benchmark_layer_full_size_sampled(dev):
    """The 32x32 layer at batch 256 (fp16 inputs, 1-bit weights, BN output),
    in the launch configuration the benchmark times: 4096 sampled outputs
    against the oracle one by one, and properties of the whole output."""
    n, cin, h, w, cout, k = 256, 128, 32, 32, 128, 3
    x = _x(300, (n, cin, h, w))
    wt = _w(301, cout, cin, k)
    kk, bb = _bn(302, cout)
    out, _, _ = _layer(dev, x, wt, 1, 1, 1, mode=q.EPI_BN_F32, bn_k=_dev(kk, dev), bn_b=_dev(bb, dev))
    got = out.cpu().numpy()
    assert np.isfinite(got).all()
    x16 = oracle.to_f16(x.numpy())
    lw, _ = oracle.quantize_weights(wt.numpy(), 1)
    idx = np.random.default_rng(303).choice(got.size, 4096, replace=False)
    co = (idx // (h * w)) % cout
    acc = oracle.conv16_acc_at(x16, lw, idx, 1, 1).astype(np.float32)
    S = oracle.conv16_acc_at(np.abs(x16.astype(np.float32)).astype(np.float16), np.abs(lw.astype(np.int32)), idx, 1, 1)
    kc, bc = kk.numpy()[co].astype(np.float64), bb.numpy()[co].astype(np.float64)
    want = kc * acc.astype(np.float64) + bc  # fmaf up to one rounding, inside the ulps below
    K = cin * k * k
    bound = (K * U / (1 - K * U) + U) * S * np.abs(kc)
    _close(got.reshape(-1)[idx], want, bound)
    # the same launch twice gives the same bits
    out2, _, _ = _layer(dev, x, wt, 1, 1, 1, mode=q.EPI_BN_F32, bn_k=_dev(kk, dev), bn_b=_dev(bb, dev))
    np.testing.assert_array_equal(out2.cpu().numpy(), got)


def test_api_rules(dev):
    n, cin, h, w, cout, k = 2, 32, 8, 8, 32, 3
    x = _x(400, (n, cin, h, w))
    wt = _w(401, cout, cin, k)
    act = q.pack_act(x.to(dev), 16)
    wq, scale = q.pack_weight(wt.to(dev), 2)
    assert q.resolve_algo(n, cin, h, w, cout, k, 1, 1, 16, 2, mode=q.EPI_SCALE_F32) == q.ALGO_MFMA_F16
    assert q.kernel_name(n, cin, h, w, cout, k, 1, 1, 16, 2, mode=q.EPI_SCALE_F32).startswith("conv_mfma_kernel<2, 16,")
    bad = [
        lambda: q.conv(act, wq, n, cin, h, w, cout, k, 1, 1, 16, 2, mode=q.EPI_INT32),
        lambda: q.conv(act, wq, n, cin, h, w, cout, k, 1, 1, 16, 2, mode=q.EPI_SCALE_F32, scale=scale,
                       algo=q.ALGO_BITPLANE),
        lambda: q.conv(act, wq, n, cin, h, w, cout, k, 1, 1, 16, 2, mode=q.EPI_SCALE_F32, scale=scale,
                       algo=q.ALGO_MFMA_FP4),
        lambda: q.conv(q.pack_act(x.to(dev), 2), wq, n, cin, h, w, cout, k, 1, 1, 2, 2, mode=q.EPI_SCALE_F32,
                       scale=scale, algo=q.ALGO_MFMA_F16),
    ]
    for f in bad:
        with pytest.raises(q.QconvError) as ei:
            f()
        assert ei.value.status == q.QCONV_EUNSUPPORTED
    # an empty batch launches nothing
    e = torch.empty(0, dtype=torch.int32, device=dev)
    q.conv(e, wq, 0, cin, h, w, cout, k, 1, 1, 16, 2, mode=q.EPI_SCALE_F32, scale=scale,
           out=torch.empty(0, dtype=torch.float32, device=dev))
    torch.cuda.synchronize()


# ---------------------------------------------------------------------------
# 1..3-bit inputs with 16-bit weights (Table I rows M x 16)
# ---------------------------------------------------------------------------

def _w16_decode(words, cout, cin, kh, kw):
    """fp16 weights [kh][kw][2 cw][cout_pad][16] -> ([cout][cin][kh][kw], padding all +0)."""
    cw = (cin + 31) // 32
    cop = (cout + 127) // 128 * 128
    h = np.asarray(words).view(np.float16).reshape(kh, kw, 2 * cw, cop, 16)
    full = np.moveaxis(h, 2, 3).reshape(kh, kw, cop, 2 * cw * 16)
    pad_ok = bool((full[:, :, cout:, :].view(np.uint16) == 0).all() and (full[:, :, :, cin:].view(np.uint16) == 0).all())
    return np.ascontiguousarray(np.transpose(full[:, :, :cout, :cin], (2, 3, 0, 1))), pad_ok


@pytest.mark.parametrize("shape", [(1, 1, 1, 1), (70, 40, 3, 3), (130, 33, 1, 1), (16, 512, 4, 4)])
def test_pack_weight_16_is_binary16(dev, shape):
    cout, cin, kh, kw = shape
    w = _w(20, cout, cin, kh)
    words, _ = q.pack_weight(w.to(dev), 16)
    torch.cuda.synchronize()
    assert words.numel() * 4 == kh * kw * 2 * ((cin + 31) // 32) * ((cout + 127) // 128 * 128) * 32
    got, pad_ok = _w16_decode(words.cpu().numpy(), cout, cin, kh, kw)
    assert pad_ok
    np.testing.assert_array_equal(got.view(np.uint16), oracle.to_f16(w.numpy()).view(np.uint16))


def _layer_w16(dev, x, w16f, a_bits, case, **epi):
    n, cin, h, ww, cout, k, stride, pad = case
    act = q.pack_act(x.to(dev), a_bits)
    wq, _ = q.pack_weight(w16f.to(dev), 16)
    out, outp = q.conv(act, wq, n, cin, h, ww, cout, k, stride, pad, a_bits, 16, **epi)
    torch.cuda.synchronize()
    return out, outp


@pytest.mark.parametrize("a_bits", [1, 2, 3])
@pytest.mark.parametrize("case", CASES)
def test_w16_integer_weights_bit_exact(dev, case, a_bits):
    """Integer-valued 16-bit weights: every partial sum is an integer, so the
    fp32 accumulator is exact and every epilogue matches bit for bit."""
    n, cin, h, w, cout, k, stride, pad = case
    x = _x(600 + cin + a_bits, (n, cin, h, w))
    wi = torch.floor(synth.uniform(synth.generator(601 + cout), (cout, cin, k, k), -4.0, 5.0))
    la = oracle.quantize(x.numpy(), a_bits)
    w16 = oracle.to_f16(wi.numpy())
    A = oracle.conv16w_acc(la, w16, a_bits, stride, pad)
    kk, bb = _bn(cout + 2, cout)
    zb, _ = oracle.qconv16w_layer(la, w16, a_bits, stride, pad, "bn", k=kk.numpy(), b=bb.numpy(), acc=A)
    out, _ = _layer_w16(dev, x, wi, a_bits, case, mode=q.EPI_BN_F32, bn_k=_dev(kk, dev), bn_b=_dev(bb, dev))
    np.testing.assert_array_equal(out.cpu().numpy(), zb)
    ho, wo = zb.shape[2], zb.shape[3]
    for pool in ([False, True] if ho >= 2 and wo >= 2 else [False]):
        ob = 1 + (cin + a_bits) % 3
        hp, wp = (ho // 2, wo // 2) if pool else (ho, wo)
        out, outp = _layer_w16(dev, x, wi, a_bits, case, mode=q.EPI_BN_F32, flags=q.EPI_POOL2 if pool else 0,
                               bn_k=_dev(kk, dev), bn_b=_dev(bb, dev), out_bits=ob,
                               out_packed=torch.empty(q.packed_act_words(n, cout, hp, wp, ob), dtype=torch.int32,
                                                      device=dev))
        zp, lv = oracle.qconv16w_layer(la, w16, a_bits, stride, pad, "bn", k=kk.numpy(), b=bb.numpy(), pool=pool,
                                       out_bits=ob, acc=A)
        np.testing.assert_array_equal(out.cpu().numpy(), zp)
        np.testing.assert_array_equal(unpack_act(outp.cpu().numpy(), n, cout, hp, wp, ob), lv)


@pytest.mark.parametrize("a_bits", [1, 2, 3])
@pytest.mark.parametrize("case", CASES[::2])
def test_w16_random_weights_within_the_accumulation_bound(dev, case, a_bits):
    n, cin, h, w, cout, k, stride, pad = case
    x = _x(700 + cin + a_bits, (n, cin, h, w))
    wt = _w(701 + cout, cout, cin, k)
    la = oracle.quantize(x.numpy(), a_bits)
    w16 = oracle.to_f16(wt.numpy())
    kk, bb = _bn(cout + 3, cout)
    zb, _ = oracle.qconv16w_layer(la, w16, a_bits, stride, pad, "bn", k=kk.numpy(), b=bb.numpy())
    out, _ = _layer_w16(dev, x, wt, a_bits, case, mode=q.EPI_BN_F32, bn_k=_dev(kk, dev), bn_b=_dev(bb, dev))
    K = cin * k * k
    pl = abs(oracle.pad_level(a_bits))
    ap = np.pad(np.abs(la.astype(np.float64)), ((0, 0), (0, 0), (pad, pad), (pad, pad)), constant_values=float(pl))
    S = oracle.conv_f64(ap, np.abs(w16.astype(np.float64)), stride, 0)
    bound = (K * U / (1 - K * U) + U) * S * (np.abs(kk.numpy())[None, :, None, None] *
                                              2.0 ** -oracle.level_shift(a_bits))
    _close(out.cpu().numpy(), zb, bound)


def test_w16_api_rules(dev):
    n, cin, h, w, cout, k = 2, 32, 8, 8, 32, 3
    x = _x(800, (n, cin, h, w))
    wq, _ = q.pack_weight(_w(801, cout, cin, k).to(dev), 16)
    act = q.pack_act(x.to(dev), 2)
    assert q.resolve_algo(n, cin, h, w, cout, k, 1, 1, 2, 16, mode=q.EPI_BN_F32) == q.ALGO_MFMA_F16
    assert q.kernel_name(n, cin, h, w, cout, k, 1, 1, 2, 16, mode=q.EPI_BN_F32).startswith("conv_mfma_kernel<2, 2,")
    bad = [
        lambda: q.conv(act, wq, n, cin, h, w, cout, k, 1, 1, 2, 16, mode=q.EPI_INT32),
        lambda: q.conv(act, wq, n, cin, h, w, cout, k, 1, 1, 2, 16, mode=q.EPI_SCALE_F32,
                       scale=torch.ones(cout, device=dev), algo=q.ALGO_MFMA_FP4),
        lambda: q.conv(q.pack_act(x.to(dev), 16), wq, n, cin, h, w, cout, k, 1, 1, 16, 16, mode=q.EPI_SCALE_F32,
                       scale=torch.ones(cout, device=dev)),
    ]
    for f in bad:
        with pytest.raises(q.QconvError) as ei:
            f()
        assert ei.value.status == q.QCONV_EUNSUPPORTED


@pytest.mark.parametrize("a_bits", [1, 2, 3])
def test_convnet_with_16_bit_weights(dev, a_bits):
    """ConvNet (Model A widths), batch 2, 16-bit weights in every quantized
    layer (Table I rows M x 16).  The hidden layers' weights are integer
    valued, so every partial sum is an exact integer and every layer's levels
    and the logits must equal the oracle's bit for bit."""
    from paper_2003_04296_amd.nets import build_convnet

    p = synth.convnet_params(seed=1013, batch=2)
    g = synth.generator(1014)
    for layer in p["convs"][1:] + p["fcs"]:
        layer["w"] = torch.floor(synth.uniform(g, tuple(layer["w"].shape), -2.0, 3.0))
    net = build_convnet(p, dev, a_bits=a_bits, w_bits=16, f32_algo=q.F32_FMAF_CHAIN)
    logits = net.forward(p["x"].to(dev))
    torch.cuda.synchronize()
    want, levels = oracle.convnet16w_forward(p, a_bits, return_levels=True)
    names = ["conv1", "conv2", "conv3", "conv4", "conv5", "conv6", "fc1", "fc2"]
    for name, lv in zip(names, levels):
        words, bits = net.tensor(net.ids[name], 2)
        shape = lv.shape if lv.ndim == 4 else (lv.shape[0], lv.shape[1], 1, 1)
        got = unpack_act(words.cpu().numpy(), *shape, bits).reshape(lv.shape)
        np.testing.assert_array_equal(got, lv, err_msg=name)
    np.testing.assert_array_equal(logits.cpu().numpy(), want)
