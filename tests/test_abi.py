"""Host-side tests of the C ABI (CPU only, no kernel is launched): the
library loads and exports every function include/qconv.h declares, status
strings, the inference-operation rule against Table I, size queries, BN
folding against the oracle, and argument validation that must reject bad
input before any launch."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2003_04296_amd as q

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "qconv.h")
GOLDEN = os.path.join(ROOT, "tests", "golden", "dispatch_table1.txt")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"\b((?:qconv|qnet|aqe)_[a-z0-9_]+)\s*\(", text)
    return sorted(set(names))


def test_library_exports_every_declared_function():
    L = q.lib()
    declared = _declared_functions()
    assert len(declared) >= 20
    missing = [n for n in declared if not hasattr(L, n)]
    assert not missing, missing
    assert set(declared) == set(q.EXPORTED)


def test_error_strings():
    L = q.lib()
    for code in (0, -1, -2, -3, -4, -5):
        s = L.qconv_error_string(code).decode()
        assert s and s != "unknown status"
    assert L.qconv_error_string(-99).decode() == "unknown status"


def test_inference_op_matches_table1():
    rows = [ln.split() for ln in open(GOLDEN) if ln.strip() and not ln.startswith("#")]
    assert len(rows) == 16
    for m, n, op, prec in rows:
        got_op, got_bits = q.inference_op(int(m), int(n))
        assert got_op == op, (m, n)
        want_bits = int(prec.split("-")[0])
        assert got_bits == want_bits, (m, n)


def test_inference_op_rejects_other_widths():
    op, prec = ctypes.c_int(), ctypes.c_int()
    assert q.lib().qconv_inference_op(4, 1, ctypes.byref(op), ctypes.byref(prec)) == q.QCONV_EINVAL


@pytest.mark.parametrize("n,c,h,w,bits", [(1, 1, 1, 1, 1), (2, 33, 5, 7, 2), (256, 128, 32, 32, 2), (3, 64, 4, 4, 3),
                                         (2, 33, 5, 7, 16), (256, 128, 32, 32, 16)])
def test_packed_act_size(n, c, h, w, bits):
    want = n * h * w * ((c + 31) // 32) * {1: 1, 2: 2, 3: 4, 16: 16}[bits] * 4
    assert q.lib().qconv_packed_act_bytes(n, c, h, w, bits) == want


@pytest.mark.parametrize("cout,cin,k,bits", [(128, 128, 3, 1), (10, 33, 1, 2), (512, 256, 3, 3)])
def test_packed_weight_size(cout, cin, k, bits):
    cw, cop = (cin + 31) // 32, (cout + 127) // 128 * 128
    planes = k * k * cw * cop * {1: 1, 2: 2, 3: 4}[bits] * 4
    i8 = k * k * cw * cop * 32
    fp4 = k * k * ((cw + 1) // 2) * cop * 32
    f16 = k * k * 2 * cw * cop * 32
    assert q.lib().qconv_packed_weight_bytes(cout, cin, k, k, bits) == planes + i8 + fp4 + f16


def test_size_queries_reject_bad_input():
    L = q.lib()
    assert L.qconv_packed_act_bytes(1, 0, 1, 1, 1) == 0
    assert L.qconv_packed_act_bytes(1, 1, 1, 1, 4) == 0
    assert L.qconv_packed_weight_bytes(0, 1, 1, 1, 1) == 0


def test_out_size():
    assert q.out_size(32, 3, 1, 1) == 32
    assert q.out_size(224, 7, 2, 3) == 112
    assert q.out_size(56, 1, 2, 0) == 28
    assert q.lib().qconv_out_size(2, 5, 1, 0) == q.QCONV_EINVAL


def test_fold_bn_matches_oracle(oracle_mod):
    rng = np.random.default_rng(0)
    c = 64
    bn = {"gamma": rng.uniform(0.5, 1.5, c).astype(np.float32), "beta": rng.normal(0, 0.3, c).astype(np.float32),
          "mean": rng.normal(0, 1, c).astype(np.float32), "var": rng.uniform(1, 2000, c).astype(np.float32),
          "eps": 1e-5}
    k, b = q.fold_bn(bn["gamma"], bn["beta"], bn["mean"], bn["var"], bn["eps"])
    ko, bo = oracle_mod.bn_fold(bn)
    np.testing.assert_array_equal(k, ko)
    np.testing.assert_array_equal(b, bo)


def test_pooled_resolution():
    """AUTO takes the matrix cores for pooled layers of any geometry (every 2x2
    window occupies four M rows of one lane) whose input tile fits the staging
    buffer; rows too wide for it fall back to the bitplane kernel."""
    fp4 = q.ALGO_MFMA_FP4
    assert q.resolve_algo(2, 128, 32, 32, 128, 3, 1, 1, 1, 1, flags=q.EPI_POOL2) == fp4
    assert q.resolve_algo(2, 128, 8, 8, 128, 3, 1, 1, 1, 1, flags=q.EPI_POOL2) == fp4
    assert q.resolve_algo(2, 128, 9, 9, 128, 3, 1, 1, 1, 1, flags=q.EPI_POOL2) == fp4
    assert q.resolve_algo(2, 128, 8, 64, 128, 3, 1, 1, 1, 1, flags=q.EPI_POOL2) == fp4
    assert q.resolve_algo(1, 128, 8, 4096, 128, 3, 1, 1, 1, 1, flags=q.EPI_POOL2) == q.ALGO_BITPLANE
    assert q.resolve_algo(1, 128, 8, 4096, 128, 3, 1, 1, 1, 1) == q.ALGO_BITPLANE


def test_auto_takes_the_bitplane_kernel_for_tiny_contractions():
    """AUTO: fp4 matrix cores for K = cin*kh*kw > 256, the bitplane kernel at
    or below (the ResNet-18 1x1 shortcut convolutions)."""
    for cin in (64, 128, 256):
        assert q.resolve_algo(64, cin, 28, 28, 2 * cin, 1, 2, 0, 2, 2, mode=q.EPI_BN_F32) == q.ALGO_BITPLANE
    assert q.resolve_algo(64, 257, 28, 28, 512, 1, 2, 0, 2, 2, mode=q.EPI_BN_F32) == q.ALGO_MFMA_FP4
    assert q.resolve_algo(64, 29, 28, 28, 64, 3, 1, 1, 2, 2, mode=q.EPI_BN_F32) == q.ALGO_MFMA_FP4  # K = 261
    # explicit requests are honoured
    assert q.resolve_algo(64, 64, 28, 28, 128, 1, 2, 0, 2, 2, algo=q.ALGO_MFMA_FP4) == q.ALGO_MFMA_FP4


def test_auto_keeps_small_contractions_the_xnor_kernel_cannot_take_on_the_matrix_cores():
    """K <= 256 goes to the bitplane algorithm only where its LDS-tiled XNOR
    form applies; packed or pooled outputs and 3-bit operands stay on the fp4
    matrix cores (the one-lane-per-pixel kernel is slower there)."""
    fp4 = q.ALGO_MFMA_FP4
    assert q.resolve_algo(64, 64, 56, 56, 64, 1, 1, 0, 2, 2, mode=q.EPI_BN_PACK, out_bits=2) == fp4
    assert q.resolve_algo(64, 128, 28, 28, 128, 1, 1, 0, 1, 1, mode=q.EPI_BN_PACK, out_bits=1) == fp4
    assert q.resolve_algo(64, 64, 28, 28, 128, 1, 2, 0, 3, 3, mode=q.EPI_BN_F32) == fp4
    assert q.resolve_algo(64, 16, 28, 28, 64, 3, 1, 1, 1, 1, mode=q.EPI_BN_F32, flags=q.EPI_POOL2) == fp4
    # the same shapes with an unpacked output and 1-2 bit operands keep the XNOR kernel
    assert q.resolve_algo(64, 64, 56, 56, 64, 1, 1, 0, 2, 2, mode=q.EPI_BN_F32) == q.ALGO_BITPLANE
    assert q.resolve_algo(64, 16, 28, 28, 64, 3, 1, 1, 1, 1, mode=q.EPI_BN_F32) == q.ALGO_BITPLANE


FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: every call below fails validation first


def _desc(**kw):
    base = dict(n=1, cin=32, h=8, w=8, cout=32, kh=3, kw=3, stride=1, pad=1, a_bits=1, w_bits=1, algo=0)
    base.update(kw)
    return q.qconv_desc(*[base[f] for f, _ in q.qconv_desc._fields_])


def _fwd(d, e, out=FAKE, out_packed=None):
    return q.lib().qconv_forward(ctypes.byref(d), FAKE, FAKE, ctypes.byref(e), out, out_packed, None)


@pytest.mark.parametrize("bad", [dict(a_bits=0), dict(w_bits=4), dict(cin=0), dict(kh=0), dict(stride=0),
                                 dict(pad=-1), dict(h=1, pad=0), dict(algo=7), dict(n=-1)])
def test_forward_rejects_bad_desc(bad):
    e = q.qconv_epilogue(q.EPI_INT32, 0, None, None, None, None, 0, None)
    assert _fwd(_desc(**bad), e) == q.QCONV_EINVAL


def test_sixteen_bit_input_rules():
    """16-bit inputs run on the fp16 matrix cores only, with an fp32 epilogue;
    the int32 overflow rule does not apply to them."""
    sc = q.qconv_epilogue(q.EPI_SCALE_F32, 0, FAKE, None, None, None, 0, None)
    assert q.resolve_algo(2, 128, 32, 32, 128, 3, 1, 1, 16, 1, mode=q.EPI_SCALE_F32) == q.ALGO_MFMA_F16
    assert q.resolve_algo(2, 128, 32, 32, 128, 3, 1, 1, 16, 3, mode=q.EPI_BN_F32, flags=q.EPI_POOL2) == q.ALGO_MFMA_F16
    assert q.lib().qconv_resolve_algo(ctypes.byref(_desc(a_bits=16, algo=q.ALGO_MFMA_F16)), ctypes.byref(sc)) == 4
    for algo in (q.ALGO_BITPLANE, q.ALGO_MFMA_I8, q.ALGO_MFMA_FP4):
        assert _fwd(_desc(a_bits=16, algo=algo), sc) == q.QCONV_EUNSUPPORTED
    assert _fwd(_desc(a_bits=2, algo=q.ALGO_MFMA_F16), sc) == q.QCONV_EUNSUPPORTED
    assert _fwd(_desc(a_bits=16, algo=5), sc) == q.QCONV_EINVAL
    assert _fwd(_desc(a_bits=8), sc) == q.QCONV_EINVAL
    e32 = q.qconv_epilogue(q.EPI_INT32, 0, None, None, None, None, 0, None)
    assert _fwd(_desc(a_bits=16), e32) == q.QCONV_EUNSUPPORTED
    assert _fwd(_desc(cin=134218000, kh=1, kw=1, pad=0, a_bits=16, w_bits=3), sc) != q.QCONV_EOVERFLOW
    assert q.kernel_name(2, 128, 32, 32, 128, 3, 1, 1, 16, 1, mode=q.EPI_BN_F32).startswith("conv_mfma_kernel<2, 16, ")


def test_sixteen_bit_weight_rules():
    """Table I's rows with 1..3-bit inputs and 16-bit weights: the packed
    weight buffer is the fp16 copy alone; the fp16 matrix cores only; 16 x 16
    is not a row of the tables."""
    cw, cop = (128 + 31) // 32, 256
    assert q.lib().qconv_packed_weight_bytes(130, 128, 3, 3, 16) == 9 * 2 * cw * cop * 32
    sc = q.qconv_epilogue(q.EPI_SCALE_F32, 0, FAKE, None, None, None, 0, None)
    for ab in (1, 2, 3):
        assert q.resolve_algo(2, 128, 32, 32, 128, 3, 1, 1, ab, 16, mode=q.EPI_BN_F32) == q.ALGO_MFMA_F16
        assert _fwd(_desc(a_bits=ab, w_bits=16, algo=q.ALGO_BITPLANE), sc) == q.QCONV_EUNSUPPORTED
    assert _fwd(_desc(a_bits=16, w_bits=16), sc) == q.QCONV_EUNSUPPORTED
    e32 = q.qconv_epilogue(q.EPI_INT32, 0, None, None, None, None, 0, None)
    assert _fwd(_desc(a_bits=2, w_bits=16), e32) == q.QCONV_EUNSUPPORTED
    assert _fwd(_desc(a_bits=2, w_bits=8), sc) == q.QCONV_EINVAL


def test_forward_rejects_overflowing_k():
    e = q.qconv_epilogue(q.EPI_INT32, 0, None, None, None, None, 0, None)
    # K = 134218000 * 1 * 1 with 3-bit codes (max 4*4) exceeds 2^31
    assert _fwd(_desc(cin=134218000, kh=1, kw=1, pad=0, a_bits=3, w_bits=3), e) == q.QCONV_EOVERFLOW


def test_forward_rejects_bad_epilogue():
    d = _desc()
    assert _fwd(d, q.qconv_epilogue(9, 0, None, None, None, None, 0, None)) == q.QCONV_EINVAL
    assert _fwd(d, q.qconv_epilogue(q.EPI_SCALE_F32, 0, None, None, None, None, 0, None)) == q.QCONV_EINVAL
    assert _fwd(d, q.qconv_epilogue(q.EPI_BN_F32, 0, None, FAKE, None, None, 0, None)) == q.QCONV_EINVAL
    assert _fwd(d, q.qconv_epilogue(q.EPI_BN_PACK, 0, None, FAKE, FAKE, None, 1, None), out_packed=None) == q.QCONV_EINVAL
    assert _fwd(d, q.qconv_epilogue(q.EPI_BN_PACK, 0, None, FAKE, FAKE, None, 5, None), out_packed=FAKE) == q.QCONV_EINVAL
    assert _fwd(d, q.qconv_epilogue(q.EPI_INT32, 0x10, None, None, None, None, 0, None)) == q.QCONV_EINVAL
    assert _fwd(d, q.qconv_epilogue(q.EPI_INT32, q.EPI_RESIDUAL, None, None, None, FAKE, 0, None)) == q.QCONV_EINVAL
    d1 = _desc(h=1, w=1, pad=0, kh=1, kw=1)
    assert _fwd(d1, q.qconv_epilogue(q.EPI_INT32, q.EPI_POOL2, None, None, None, None, 0, None)) == q.QCONV_EINVAL
    bad_thr = (ctypes.c_float * 3)(0.5, 0.25, 0.75)
    e = q.qconv_epilogue(q.EPI_BN_PACK, 0, None, FAKE, FAKE, None, 3, ctypes.cast(bad_thr, ctypes.c_void_p))
    assert _fwd(d, e, out_packed=FAKE) == q.QCONV_EINVAL


def test_pack_calls_reject_bad_input():
    L = q.lib()
    assert L.qconv_pack_act(FAKE, 1, 1, 1, 1, 0, None, FAKE, None) == q.QCONV_EINVAL
    assert L.qconv_pack_act(None, 1, 1, 1, 1, 1, None, FAKE, None) == q.QCONV_EINVAL
    neg = (ctypes.c_float * 1)(-0.5)
    assert L.qconv_pack_act(FAKE, 1, 1, 1, 1, 2, neg, FAKE, None) == q.QCONV_EINVAL
    assert L.qconv_pack_weight(FAKE, 1, 1, 1, 1, 2, None, FAKE, None, None) == q.QCONV_EINVAL
    dec = (ctypes.c_float * 3)(0.3, 0.2, 0.9)
    assert L.qconv_pack_weight(FAKE, 1, 1, 1, 1, 3, dec, FAKE, FAKE, None) == q.QCONV_EINVAL


def test_qnet_validation_and_workspace():
    L = q.lib()
    assert not L.qnet_create(0, 32, 32)
    net = q.Net(3, 32, 32)
    h = net._h
    assert L.qnet_add_qconv(h, 0, FAKE, 16, 3, 1, 1, 1, 0, FAKE, FAKE, -1, 1) == q.QCONV_EINVAL  # fp32 source
    assert L.qnet_add_conv_f32(h, 5, FAKE, 16, 3, 1, 1, FAKE, FAKE, 0, 1) == q.QCONV_EINVAL  # no tensor 5
    t1 = L.qnet_add_conv_f32(h, 0, FAKE, 16, 3, 1, 1, FAKE, FAKE, 0, 1)
    assert t1 == 1
    assert L.qnet_add_maxpool_f32(h, t1, 2, 2, 0) == q.QCONV_EINVAL  # packed source
    t2 = L.qnet_add_qconv(h, t1, FAKE, 16, 3, 1, 1, 1, 1, FAKE, FAKE, -1, 0)
    assert t2 == 2
    assert net.tensor_info(t2, 4)[:4] == (16, 16, 16, 0)
    t3 = L.qnet_add_avgpool(h, t2)
    t4 = L.qnet_add_fc_f32(h, t3, FAKE, None, 10)
    assert t4 == 4
    need = net.workspace_bytes(4)
    # packed conv1 output + fp32 conv2 output + avgpool + transposed conv1 weights
    assert need >= 4 * 32 * 32 * 4 + 4 * 16 * 16 * 16 * 4 + 4 * 16 * 4
    rc = L.qnet_forward(h, FAKE, 4, FAKE, FAKE, need - 1, None)
    assert rc == q.QCONV_EWORKSPACE
    assert L.qnet_forward(h, None, 4, FAKE, FAKE, need, None) == q.QCONV_EINVAL


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(q, "_lib", None)
    monkeypatch.setattr(q, "LIB_PATH", str(tmp_path / "absent.so"))
    with pytest.raises(RuntimeError, match="no CPU fallback"):
        q.lib()


def test_fp4_refused_past_exact_fp32_accumulation():
    """The fp4 matrix cores accumulate in fp32, exact only while every partial
    sum (at most K * max|a| * max|w|) stays below 2^24: an explicit fp4 request
    past that is refused, and AUTO takes the int8 matrix cores (exact int32)
    or the bitplane kernel instead."""
    bint = q.qconv_epilogue(q.EPI_INT32, 0, None, None, None, None, 0, None)
    L = q.lib()
    for ab, wb, mx in ((3, 3, 16), (1, 1, 1), (3, 1, 4)):
        k_lim = (1 << 24) // mx  # smallest K whose bound reaches 2^24
        for cin, ok in ((k_lim - 1, True), (k_lim, False), (k_lim + 1000, False)):
            d = _desc(n=1, cin=cin, h=2, w=2, kh=1, kw=1, pad=0, a_bits=ab, w_bits=wb, cout=32,
                      algo=q.ALGO_MFMA_FP4)
            rc = L.qconv_resolve_algo(ctypes.byref(d), ctypes.byref(bint))
            if ok:
                assert rc == q.ALGO_MFMA_FP4, (ab, wb, cin)
            else:
                assert rc == q.QCONV_EUNSUPPORTED, (ab, wb, cin)
                d.algo = q.ALGO_AUTO
                auto = L.qconv_resolve_algo(ctypes.byref(d), ctypes.byref(bint))
                assert auto in (q.ALGO_MFMA_I8, q.ALGO_BITPLANE), (ab, wb, cin, auto)
                d.algo = q.ALGO_MFMA_I8
                assert L.qconv_resolve_algo(ctypes.byref(d), ctypes.byref(bint)) in (q.ALGO_MFMA_I8,
                                                                                       q.QCONV_EUNSUPPORTED)
    # the 3x3 form of the 3W3A bound: K = 9 cin
    assert q.resolve_algo(1, 116508, 4, 4, 32, 3, 1, 1, 3, 3, algo=q.ALGO_AUTO) == q.ALGO_MFMA_FP4
    assert q.resolve_algo(1, 116509, 4, 4, 32, 3, 1, 1, 3, 3, algo=q.ALGO_AUTO) != q.ALGO_MFMA_FP4


@pytest.mark.parametrize("bits,vals", [(2, [0.5, 0.6]), (3, [0.1, 0.2]), (3, [0.1, 0.2, 0.3, 0.4]), (2, [])])
def test_binding_checks_threshold_counts(bits, vals):
    """The C side reads exactly one threshold for 2 bits and three for 3 bits
    from the host array; the binding refuses any other count before the call."""
    with pytest.raises(ValueError, match="thresholds take"):
        q._host_thr(vals, bits, "test")
    assert q._host_thr(None, bits, "test") is None
    assert q._host_thr(np.array([0.5] * {2: 1, 3: 3}[bits], np.float32), bits, "test") is not None
    # zero-valued thresholds are a real setting, not "use the defaults"
    arr = q._host_thr(np.zeros({2: 1, 3: 3}[bits], np.float32), bits, "test")
    assert arr is not None and list(arr) == [0.0] * {2: 1, 3: 3}[bits]


@pytest.mark.parametrize("algo", [q.F32_MFMA, q.F32_BF16X6, q.F32_FMAF_CHAIN])
def test_stem_fusion_bookkeeping(algo):
    """A 7x7/2 fp32 stem followed by 3x3/2 max pooling and a 2-bit quantize:
    with the matrix-core algorithms both later layers are written by the
    stem's epilogue and launch nothing (the bf16x6 one in its own kernel);
    with the fmaf chains each launches its own kernel.  Host-side only
    (nothing is launched)."""
    L = q.lib()
    net = q.Net(3, 224, 224, algo)
    h = net._h
    t1 = L.qnet_add_conv_f32(h, 0, FAKE, 64, 7, 2, 3, FAKE, FAKE, 1, 0)
    t2 = L.qnet_add_maxpool_f32(h, t1, 3, 2, 1)
    t3 = L.qnet_add_quantize(h, t2, 2)
    assert (t1, t2, t3) == (1, 2, 3)
    fused = [L.qnet_layer_fused_into(h, i) for i in range(3)]
    names = [net.layer_kernel(i, 8) for i in range(3)]
    if algo != q.F32_FMAF_CHAIN:
        assert fused == [0, 0, 0]
        kind = "bf16x6" if algo == q.F32_BF16X6 else "mfma"
        assert names == [f"conv_f32_{kind}_kernel<7, 2, 1, 2>", "", ""]
    else:
        assert fused == [0, 1, 2]
        assert names[0].startswith("conv_f32_kernel<") and names[1] and names[2]
    assert L.qnet_set_f32_algo(h, q.F32_MFMA) == q.QCONV_EINVAL  # layers already added
    assert L.qnet_layer_fused_into(h, 3) == q.QCONV_EINVAL
    assert L.qnet_layer_fused_into(h, -1) == q.QCONV_EINVAL
    assert L.qnet_layer_fused_into(None, 0) == q.QCONV_EINVAL


def test_bf16x6_only_takes_the_pooled_7x7_stride_2_geometry():
    """Under the bf16x6 algorithm, layers outside its geometry (3x3 stride 1,
    an unpooled conv, more than 3 input channels) keep the fp32 matrix
    cores; an unknown algorithm value is refused."""
    L = q.lib()
    net = q.Net(3, 32, 32, q.F32_BF16X6)
    t1 = L.qnet_add_conv_f32(net._h, 0, FAKE, 128, 3, 1, 1, FAKE, FAKE, 0, 1)
    assert t1 == 1 and net.layer_kernel(0, 4) == "conv_f32_mfma_kernel<3, 1, 0, 1>"
    net4 = q.Net(4, 64, 64, q.F32_BF16X6)
    t1 = L.qnet_add_conv_f32(net4._h, 0, FAKE, 64, 7, 2, 3, FAKE, FAKE, 1, 0)
    L.qnet_add_maxpool_f32(net4._h, t1, 3, 2, 1)
    assert net4.layer_kernel(0, 2).startswith("conv_f32_kernel<")  # the window of 4 channels: the chain
    net1 = q.Net(1, 64, 64, q.F32_BF16X6)
    t1 = L.qnet_add_conv_f32(net1._h, 0, FAKE, 40, 7, 2, 3, FAKE, FAKE, 1, 0)
    L.qnet_add_maxpool_f32(net1._h, t1, 3, 2, 1)
    assert net1.layer_kernel(0, 2) == "conv_f32_bf16x6_kernel<7, 2, 1, 0>"
    with pytest.raises(q.QconvError):
        q.Net(3, 8, 8, 3)
