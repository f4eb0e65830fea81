"""Plain CPU oracle for the MINW-Net inference path and the elementwise
steps of its AQE training.

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg are its only callers.  It never imports the GPU package and
the GPU package never imports it; the arithmetic lives in ``qoracle.c``
(plain nested loops, built with gcc) and this module only marshals numpy
arrays and composes layers in the order the paper gives.

Paper: Chen et al., "Propagating Asymptotic-Estimated Gradients for Low
Bitwidth Quantized Neural Networks".

Readings taken where the paper is silent (each also listed in the design notes):

* sign(0) = -1: Sec. II-A defines sign as +1 only for a positive input.
* ternary threshold for activations delta = 0.5 (nearest level on the
  HardTanh range); for weights delta_c = 0.7 * mean|W_c| (the rule of the
  ternary-weight work that Eq. 21 defers to).
* 3-bit thresholds t = (1/8, 3/8, 3/4): the midpoints of adjacent levels of
  Eq. 22 / Sec. IV-C, so the quantizer rounds to the nearest level and
  saturates at 1; weights use t * mean|W_c|.
* ties (|x| equal to a threshold) go to the smaller magnitude (the "<=" of
  Eqs. 21-22).
* padding taps of a quantized conv hold Q(0): -1 for 1 bit, 0 otherwise.
* batch norm is folded in double to (k, b) and applied as one fmaf; pooling
  sits before BN (Sec. III-E); HardTanh is applied before requantization.
* fp32 layers accumulate each output as one fmaf chain in (ci, kh, kw)
  order from +0.
* "16-bit floating" inputs (Tables I and IV) are IEEE binary16; their
  product with weight codes is the exact sum rounded once to fp32, and the
  fp32 epilogue of the quantized layers follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "qoracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

# Quantizer thresholds (readings of Eqs. 21-22, see module docstring).
ACT_THRESHOLDS = {1: (), 2: (0.5,), 3: (0.125, 0.375, 0.75)}
WEIGHT_BASE_THRESHOLDS = {1: (), 2: (0.7,), 3: (0.125, 0.375, 0.75)}


def build(force: bool = True) -> str:
    """Compile qoracle.c with gcc (OpenMP, no contraction, no fast-math)."""
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
               "-fPIC", "-shared", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
            build(force=True)
        _lib = ctypes.CDLL(_LIB_PATH)
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _f32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float32))


def _i8(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int8))


def num_threads() -> int:
    return int(lib().oracle_num_threads())


# ---------------------------------------------------------------------------
# Quantizers (Sec. III-C, Eqs. 4, 20-22)
# ---------------------------------------------------------------------------


def quantize(x, bits: int, thr=None) -> np.ndarray:
    """Integer level codes of h(x) (3 bits: codes are 4x the level)."""
    x = _f32(x)
    thr = ACT_THRESHOLDS[bits] if thr is None else tuple(thr)
    t = _f32(thr if len(thr) else (0.0,))
    out = np.empty(x.shape, dtype=np.int8)
    rc = lib().oracle_quantize(_p(x), ctypes.c_int64(x.size), bits, _p(t), _p(out))
    if rc != 0:
        raise ValueError(f"oracle_quantize failed ({rc})")
    return out


def pad_level(bits: int) -> int:
    """Level taken by a padding tap: Q(0)."""
    return int(quantize(np.zeros(1, np.float32), bits)[0])


def level_shift(bits: int) -> int:
    """Codes are 2^shift x the level (4x for 3 bits)."""
    return 2 if bits == 3 else 0


def weight_scale(w) -> np.ndarray:
    """s_c = mean |W_c| per output channel (double sum in a fixed order:
    256 strided partial sums, added pairwise; one rounding to float)."""
    w = _f32(w)
    cout = w.shape[0]
    k = w.size // cout
    s = np.empty(cout, dtype=np.float32)
    lib().oracle_weight_scale(_p(w), cout, ctypes.c_int64(k), _p(s))
    return s


def quantize_weights(w, bits: int, base_thr=None):
    """(levels int8 with w's shape, s_c float32 [cout])."""
    w = _f32(w)
    cout = w.shape[0]
    k = w.size // cout
    s = weight_scale(w)
    bt = WEIGHT_BASE_THRESHOLDS[bits] if base_thr is None else tuple(base_thr)
    t = _f32(bt if len(bt) else (0.0,))
    out = np.empty(w.shape, dtype=np.int8)
    rc = lib().oracle_quantize_weights(_p(w), cout, ctypes.c_int64(k), bits, _p(s), _p(t), _p(out))
    if rc != 0:
        raise ValueError(f"oracle_quantize_weights failed ({rc})")
    return out, s


def quantize_weights_with_scale(w, bits: int, s, base_thr=None) -> np.ndarray:
    """Integer level codes of the weights with given per-channel scales s_c."""
    w = _f32(w)
    cout = w.shape[0]
    k = w.size // cout
    s = _f32(s)
    bt = WEIGHT_BASE_THRESHOLDS[bits] if base_thr is None else tuple(base_thr)
    t = _f32(bt if len(bt) else (0.0,))
    out = np.empty(w.shape, dtype=np.int8)
    rc = lib().oracle_quantize_weights(_p(w), cout, ctypes.c_int64(k), bits, _p(s), _p(t), _p(out))
    if rc != 0:
        raise ValueError(f"oracle_quantize_weights failed ({rc})")
    return out


# ---------------------------------------------------------------------------
# Training with the asymptotic-quantized estimator (Sec. III-B and III-D,
# Eqs. activation and weight; Algorithm 1, training branch).  Every float32
# operation below is one rounded numpy float32 operation, in the order the
# equations write them.
# ---------------------------------------------------------------------------


def levels_f32(codes, bits: int) -> np.ndarray:
    """Level values of integer codes (3 bits: codes are 4x the level)."""
    v = np.asarray(codes).astype(np.float32)
    return v / np.float32(4) if bits == 3 else v


def aqe_forward(x, bits: int, alpha: float, thr=None) -> np.ndarray:
    """Activations: alpha h(x) + (1 - alpha) x with h the quantizer level."""
    x = _f32(x)
    h = levels_f32(quantize(x, bits, thr), bits)
    a = np.float32(alpha)
    om = np.float32(np.float32(1) - a)
    with np.errstate(invalid="ignore"):  # 0 * inf is NaN, as on the GPU
        return (a * h + om * x).astype(np.float32)


def aqe_forward_weights(w, bits: int, alpha: float, s, base_thr=None) -> np.ndarray:
    """Weights (OIHW, one group per output channel) with given s_c."""
    w = _f32(w)
    h = levels_f32(quantize_weights_with_scale(w, bits, s, base_thr), bits)
    a = np.float32(alpha)
    om = np.float32(np.float32(1) - a)
    with np.errstate(invalid="ignore"):
        return (a * h + om * w).astype(np.float32)


def aqe_backward(x, gy, alpha: float) -> np.ndarray:
    """2 alpha gy where |x| <= 1, else 0."""
    x = _f32(x)
    gy = _f32(gy)
    twoa = np.float32(2) * np.float32(alpha)
    with np.errstate(invalid="ignore"):
        return np.where(np.abs(x) <= np.float32(1), twoa * gy, np.float32(0)).astype(np.float32)


def ste_backward(x, gy) -> np.ndarray:
    """The straight-through estimator of Sec. II-B: gy 1{|x| <= 1}."""
    x = _f32(x)
    gy = _f32(gy)
    return np.where(np.abs(x) <= np.float32(1), gy, np.float32(0)).astype(np.float32)


def sgd_clip(w, g, lr: float) -> np.ndarray:
    """Algorithm 1's update with plain SGD, then the clip to [-1, 1]."""
    w = _f32(w)
    g = _f32(g)
    v = (w - np.float32(lr) * g).astype(np.float32)
    v = np.where(v > np.float32(1), np.float32(1), v)
    v = np.where(v < np.float32(-1), np.float32(-1), v)
    return v.astype(np.float32)


# ---------------------------------------------------------------------------
# Quantized product (Algorithm 1, inference branch)
# ---------------------------------------------------------------------------


def out_size(h: int, k: int, stride: int, pad: int) -> int:
    return (h + 2 * pad - k) // stride + 1


def conv_levels(a, w, stride: int = 1, pad: int = 0, pad_level_value: int = 0) -> np.ndarray:
    """Direct convolution over level codes, int64 accumulation, int32 result."""
    a = _i8(a)
    w = _i8(w)
    n, cin, h, wd = a.shape
    cout, cin2, kh, kw = w.shape
    if cin2 != cin:
        raise ValueError("channel mismatch")
    ho, wo = out_size(h, kh, stride, pad), out_size(wd, kw, stride, pad)
    out = np.empty((n, cout, ho, wo), dtype=np.int32)
    rc = lib().oracle_conv_levels(_p(a), _p(w), n, cin, h, wd, cout, kh, kw, stride, pad,
                                  int(pad_level_value), _p(out))
    if rc == -4:
        raise OverflowError("accumulator does not fit int32")
    if rc != 0:
        raise ValueError(f"oracle_conv_levels failed ({rc})")
    return out


def conv_levels_at(a, w, idx, stride: int = 1, pad: int = 0, pad_level_value: int = 0) -> np.ndarray:
    """The same product at flat NCHW output indices ``idx`` only."""
    a = _i8(a)
    w = _i8(w)
    idx = np.ascontiguousarray(np.asarray(idx, dtype=np.int64))
    n, cin, h, wd = a.shape
    cout, _, kh, kw = w.shape
    out = np.empty(idx.shape, dtype=np.int32)
    rc = lib().oracle_conv_levels_at(_p(a), _p(w), n, cin, h, wd, cout, kh, kw, stride, pad,
                                     int(pad_level_value), _p(idx), ctypes.c_int64(idx.size), _p(out))
    if rc != 0:
        raise ValueError(f"oracle_conv_levels_at failed ({rc})")
    return out


# ---------------------------------------------------------------------------
# Epilogue steps (Sec. III-E), one pass each
# ---------------------------------------------------------------------------


def epi_scale(acc, s, shift: int = 0) -> np.ndarray:
    acc = np.ascontiguousarray(acc, dtype=np.int32)
    n, c = acc.shape[:2]
    hw = acc.size // max(1, n * c)
    y = np.empty(acc.shape, dtype=np.float32)
    lib().oracle_epi_scale(_p(acc), n, c, ctypes.c_int64(hw), shift, _p(_f32(s)), _p(y))
    return y


def bn_fold(bn: dict):
    """(k, b) float32 from gamma, beta, mean, var, eps (double arithmetic)."""
    g, be, m, v = (_f32(bn[key]) for key in ("gamma", "beta", "mean", "var"))
    c = g.size
    k = np.empty(c, np.float32)
    b = np.empty(c, np.float32)
    lib().oracle_bn_fold(_p(g), _p(be), _p(m), _p(v), ctypes.c_double(float(bn["eps"])), c, _p(k), _p(b))
    return k, b


def epi_bn(acc, k, b, shift: int = 0) -> np.ndarray:
    acc = np.ascontiguousarray(acc, dtype=np.int32)
    n, c = acc.shape[:2]
    hw = acc.size // max(1, n * c)
    z = np.empty(acc.shape, dtype=np.float32)
    lib().oracle_epi_bn(_p(acc), n, c, ctypes.c_int64(hw), shift, _p(_f32(k)), _p(_f32(b)), _p(z))
    return z


def bn_f32(x, k, b) -> np.ndarray:
    """BN on an fp32 activation: fmaf(k_c, x, b_c)."""
    x = _f32(x)
    n, c = x.shape[:2]
    hw = x.size // max(1, n * c)
    z = np.empty(x.shape, np.float32)
    lib().oracle_bn_f32(_p(x), n, c, ctypes.c_int64(hw), _p(_f32(k)), _p(_f32(b)), _p(z))
    return z


def maxpool2_int(acc) -> np.ndarray:
    acc = np.ascontiguousarray(acc, dtype=np.int32)
    n, c, h, w = acc.shape
    y = np.empty((n, c, h // 2, w // 2), np.int32)
    lib().oracle_maxpool2_int(_p(acc), n, c, h, w, _p(y))
    return y


def hardtanh(x) -> np.ndarray:
    x = _f32(x)
    y = np.empty_like(x)
    lib().oracle_hardtanh(_p(x), ctypes.c_int64(x.size), _p(y))
    return y


def relu(x) -> np.ndarray:
    x = _f32(x)
    y = np.empty_like(x)
    lib().oracle_relu(_p(x), ctypes.c_int64(x.size), _p(y))
    return y


def add(x, r) -> np.ndarray:
    x = _f32(x)
    r = _f32(r)
    y = np.empty_like(x)
    lib().oracle_add(_p(x), _p(r), ctypes.c_int64(x.size), _p(y))
    return y


# ---------------------------------------------------------------------------
# Full-precision support layers
# ---------------------------------------------------------------------------


def conv_f32(x, w, stride: int = 1, pad: int = 0) -> np.ndarray:
    x = _f32(x)
    w = _f32(w)
    n, cin, h, wd = x.shape
    cout, _, kh, kw = w.shape
    y = np.empty((n, cout, out_size(h, kh, stride, pad), out_size(wd, kw, stride, pad)), np.float32)
    rc = lib().oracle_conv_f32(_p(x), _p(w), n, cin, h, wd, cout, kh, kw, stride, pad, _p(y))
    if rc != 0:
        raise ValueError("oracle_conv_f32 failed")
    return y


def conv_f64(x, w, stride: int = 1, pad: int = 0) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float64)
    w = np.ascontiguousarray(w, dtype=np.float64)
    n, cin, h, wd = x.shape
    cout, _, kh, kw = w.shape
    y = np.empty((n, cout, out_size(h, kh, stride, pad), out_size(wd, kw, stride, pad)), np.float64)
    rc = lib().oracle_conv_f64(_p(x), _p(w), n, cin, h, wd, cout, kh, kw, stride, pad, _p(y))
    if rc != 0:
        raise ValueError("oracle_conv_f64 failed")
    return y


def fc_f32(x, w, bias=None) -> np.ndarray:
    x = _f32(x)
    w = _f32(w)
    n = x.shape[0]
    fin = x.size // n
    fout = w.shape[0]
    y = np.empty((n, fout), np.float32)
    bias_arr = _f32(bias) if bias is not None else None
    lib().oracle_fc_f32(_p(x), _p(w), _p(bias_arr) if bias_arr is not None else None, n, fin, fout,
                        _p(y))
    return y


def maxpool_f32(x, k: int = 3, s: int = 2, p: int = 1) -> np.ndarray:
    x = _f32(x)
    n, c, h, w = x.shape
    y = np.empty((n, c, out_size(h, k, s, p), out_size(w, k, s, p)), np.float32)
    lib().oracle_maxpool_f32(_p(x), n, c, h, w, k, s, p, _p(y))
    return y


def avgpool_f32(x) -> np.ndarray:
    x = _f32(x)
    n, c, h, w = x.shape
    y = np.empty((n, c), np.float32)
    lib().oracle_avgpool_f32(_p(x), n, c, h, w, _p(y))
    return y


# ---------------------------------------------------------------------------
# Layers and networks (Algorithm 1 inference branch + Sec. III-E constructs)
# ---------------------------------------------------------------------------


def qconv_acc(a_levels, w_levels, a_bits: int, stride: int, pad: int) -> np.ndarray:
    return conv_levels(a_levels, w_levels, stride, pad, pad_level(a_bits))


def _np(t):
    return t.numpy() if hasattr(t, "numpy") else np.asarray(t)


def convnet_forward(p: dict, return_levels: bool = False):
    """ConvNet (Model A family), 1-bit weights and activations inside, fp32
    first conv and last FC.  Each hidden layer: product -> [2x2 max pool] ->
    BN -> HardTanh -> sign (Sec. III-E constructs)."""
    x = _np(p["x"])
    levels = []
    c1 = p["convs"][0]
    z = conv_f32(x, _np(c1["w"]), 1, 1)
    k, b = bn_fold({kk: _np(v) if kk != "eps" else v for kk, v in c1["bn"].items()})
    z = bn_f32(z, k, b)
    a = quantize(hardtanh(z), 1)
    levels.append(a)
    for i, layer in enumerate(p["convs"][1:], start=1):
        wq, _ = quantize_weights(_np(layer["w"]), 1)
        acc = qconv_acc(a, wq, 1, 1, 1)
        if p["pools"][i]:
            acc = maxpool2_int(acc)
        k, b = bn_fold({kk: _np(v) if kk != "eps" else v for kk, v in layer["bn"].items()})
        a = quantize(hardtanh(epi_bn(acc, k, b)), 1)
        levels.append(a)
    n = a.shape[0]
    for fc in p["fcs"]:
        w = _np(fc["w"])
        # An FC layer over a [n, c, h, w] input is the convolution whose kernel
        # covers the whole map, with the weight columns in (c, h, w) order.
        a4 = a.reshape(n, -1, 1, 1) if a.ndim == 2 else a
        w4 = w.reshape(w.shape[0], a4.shape[1], a4.shape[2], a4.shape[3])
        wq, _ = quantize_weights(w4, 1)
        acc = qconv_acc(a4, wq, 1, 1, 0)
        k, b = bn_fold({kk: _np(v) if kk != "eps" else v for kk, v in fc["bn"].items()})
        a = quantize(hardtanh(epi_bn(acc, k, b)), 1).reshape(n, -1)
        levels.append(a)
    logits = fc_f32(a.astype(np.float32), _np(p["fc_out"]["w"]), _np(p["fc_out"]["b"]))
    return (logits, levels) if return_levels else logits


def convnet16w_forward(p: dict, a_bits: int = 1, return_levels: bool = False):
    """ConvNet (Model A family) with 16-bit weights and a_bits-bit
    activations inside (Table I rows M x 16): fp32 first conv -> BN ->
    Q(HardTanh); each hidden layer: the product of the input levels with the
    fp16 weights (exact, rounded once to fp32) -> [2x2 max pool] -> BN ->
    Q(HardTanh) (the last FC quantizes with 1 bit); fp32 last FC."""
    def fold(bn):
        return bn_fold({kk: _np(v) if kk != "eps" else v for kk, v in bn.items()})

    x = _np(p["x"])
    levels = []
    c1 = p["convs"][0]
    k, b = fold(c1["bn"])
    a = quantize(hardtanh(bn_f32(conv_f32(x, _np(c1["w"]), 1, 1), k, b)), a_bits)
    levels.append(a)
    for i, layer in enumerate(p["convs"][1:], start=1):
        k, b = fold(layer["bn"])
        _, a = qconv16w_layer(a, to_f16(_np(layer["w"])), a_bits, 1, 1, "bn", k=k, b=b, pool=p["pools"][i],
                              out_bits=a_bits)
        levels.append(a)
    n = a.shape[0]
    for j, fc in enumerate(p["fcs"]):
        w = _np(fc["w"])
        a4 = a.reshape(n, -1, 1, 1) if a.ndim == 2 else a
        w4 = w.reshape(w.shape[0], a4.shape[1], a4.shape[2], a4.shape[3])
        k, b = fold(fc["bn"])
        ob = 1 if j == len(p["fcs"]) - 1 else a_bits
        _, a = qconv16w_layer(a4, to_f16(w4), a_bits, 1, 0, "bn", k=k, b=b, out_bits=ob)
        a = a.reshape(n, -1)
        levels.append(a)
    logits = fc_f32(a.astype(np.float32), _np(p["fc_out"]["w"]), _np(p["fc_out"]["b"]))
    return (logits, levels) if return_levels else logits


def resnet18_forward(p: dict, a_bits: int = 2, w_bits: int = 2, return_acts: bool = False):
    """ResNet-18 with quantized 3x3/1x1 convs, fp32 stem and FC.

    stem: conv 7x7/2 p3 -> BN -> ReLU -> maxpool 3x3/2 p1 (fp32).
    block: q = Q(x); y = Q(HardTanh(BN1(q * W1))); z = BN2(y * W2);
           out = z + (x  or  BN_d(q * W_d)) in fp32.
    head: global average pool -> FC + bias (fp32)."""
    def fold(bn):
        return bn_fold({kk: _np(v) if kk != "eps" else v for kk, v in bn.items()})

    x = _np(p["x"])
    st = p["stem"]
    z = conv_f32(x, _np(st["w"]), 2, 3)
    k, b = fold(st["bn"])
    x = maxpool_f32(relu(bn_f32(z, k, b)), 3, 2, 1)
    acts = [x]
    sh_a = level_shift(a_bits)
    for blk in p["blocks"]:
        s = blk["stride"]
        q = quantize(x, a_bits)
        w1, _ = quantize_weights(_np(blk["w1"]), w_bits)
        w2, _ = quantize_weights(_np(blk["w2"]), w_bits)
        sh = sh_a + level_shift(w_bits)
        k1, b1 = fold(blk["bn1"])
        y = quantize(hardtanh(epi_bn(qconv_acc(q, w1, a_bits, s, 1), k1, b1, sh)), a_bits)
        k2, b2 = fold(blk["bn2"])
        z = epi_bn(qconv_acc(y, w2, a_bits, 1, 1), k2, b2, sh)
        if "wd" in blk:
            wd, _ = quantize_weights(_np(blk["wd"]), w_bits)
            kd, bd = fold(blk["bnd"])
            sc = epi_bn(qconv_acc(q, wd, a_bits, s, 0), kd, bd, sh)
        else:
            sc = x
        x = add(z, sc)
        acts.append(x)
    feat = avgpool_f32(x)
    logits = fc_f32(feat, _np(p["fc"]["w"]), _np(p["fc"]["b"]))
    return (logits, acts) if return_acts else logits


# ---------------------------------------------------------------------------
# 16-bit inputs with 1..3-bit weights (Table I rows with 16-bit inputs;
# Table IV "reduce weights" rows): the "XNOR ADDER" / "SHIFT ADDER" product
# at 16-bit floating precision
# ---------------------------------------------------------------------------


def to_f16(x) -> np.ndarray:
    """A 16-bit floating input: fp32 rounded to IEEE binary16 (nearest, ties
    to even, beyond the range to +-inf, NaN stays NaN) by numpy's conversion."""
    with np.errstate(over="ignore"):
        return np.asarray(x, dtype=np.float32).astype(np.float16)


def conv16_acc(x16, w_levels, stride: int = 1, pad: int = 0) -> np.ndarray:
    """The product of 16-bit inputs and weight level codes, in code units,
    summed in fp64 (plain loops in qoracle.c).  Padding taps hold 0: the
    quantizer of a 16-bit input is the identity.  Every term x * code is a
    multiple of 2^-24 (the fp16 grid) times a code of at most 4, so each
    partial sum is exact in fp64 while the sum of |terms| stays below 2^29."""
    x = np.asarray(x16, dtype=np.float16).astype(np.float64)
    return conv_f64(x, np.asarray(w_levels).astype(np.float64), stride, pad)


def conv16_acc_at(x16, w_levels, idx, stride: int = 1, pad: int = 0) -> np.ndarray:
    """conv16_acc at flat NCHW output indices ``idx`` only (one fp64 dot
    product per output over its zero-padded receptive field)."""
    x = np.asarray(x16, dtype=np.float16).astype(np.float64)
    w = np.asarray(w_levels).astype(np.float64)
    n, cin, h, wd = x.shape
    cout, _, kh, kw = w.shape
    ho, wo = out_size(h, kh, stride, pad), out_size(wd, kw, stride, pad)
    xp = np.zeros((n, cin, h + 2 * pad + stride * kh, wd + 2 * pad + stride * kw), np.float64)
    xp[:, :, pad:pad + h, pad:pad + wd] = x
    idx = np.asarray(idx, dtype=np.int64).reshape(-1)
    out = np.empty(idx.size, np.float64)
    for t, f in enumerate(idx):
        b, rem = divmod(int(f), cout * ho * wo)
        co, rem = divmod(rem, ho * wo)
        oy, ox = divmod(rem, wo)
        patch = xp[b, :, oy * stride:oy * stride + kh, ox * stride:ox * stride + kw]
        out[t] = float(np.sum(patch * w[co]))
    return out


def conv16w_acc(a_levels, w16, a_bits: int, stride: int = 1, pad: int = 0) -> np.ndarray:
    """The product of M-bit input level codes and 16-bit weights (Table I
    rows with 1..3-bit inputs and 16-bit weights), in code units, summed in
    fp64: padding taps hold Q(0), the level an all-zero packed word encodes
    (-1 for 1 bit).  Exact on the same grounds as conv16_acc."""
    a = np.asarray(a_levels, dtype=np.float64)
    if pad:
        a = np.pad(a, ((0, 0), (0, 0), (pad, pad), (pad, pad)), constant_values=float(pad_level(a_bits)))
    return conv_f64(a, np.asarray(w16, dtype=np.float16).astype(np.float64), stride, 0)


def f32_acc_epilogue(acc, shift: int, mode: str, s=None, k=None, b=None, residual=None, pool: bool = False,
                     out_bits: int = 0):
    """The layer epilogue on an exact product rounded once to fp32 (the
    16-bit rows): 2x2 max pooling of the accumulators, acc * 2^-shift, then
      mode "scale": s_c * acc_real;  "bn": fmaf(k_c, acc_real, b_c) [+ residual];
    out_bits > 0 also returns Q(HardTanh(z)) with the activation quantizer.
    Returns (z, levels or None)."""
    acc = np.asarray(acc, np.float64).astype(np.float32)
    if pool:
        acc = maxpool_f32(acc, 2, 2, 0)
    a = (acc * np.float32(2.0 ** -shift)).astype(np.float32)
    if mode == "scale":
        z = (_f32(s)[None, :, None, None] * a).astype(np.float32)
    elif mode == "bn":
        z = bn_f32(a, k, b)
        if residual is not None:
            z = add(z, residual)
    else:
        raise ValueError(mode)
    lv = quantize(hardtanh(z), out_bits) if out_bits else None
    return z, lv


def qconv16_layer(x16, w_levels, w_bits: int, stride: int, pad: int, mode: str, s=None, k=None, b=None,
                  residual=None, pool: bool = False, out_bits: int = 0, acc=None):
    """One layer on 16-bit inputs (Sec. III-E layer constructs): the exact
    product rounded once to fp32, then f32_acc_epilogue with the weights'
    code shift (3-bit codes are 4 x level).  ``acc``: conv16_acc(x16,
    w_levels, stride, pad) when already computed."""
    if acc is None:
        acc = conv16_acc(x16, w_levels, stride, pad)
    return f32_acc_epilogue(acc, level_shift(w_bits), mode, s, k, b, residual, pool, out_bits)


def qconv16w_layer(a_levels, w16, a_bits: int, stride: int, pad: int, mode: str, s=None, k=None, b=None,
                   residual=None, pool: bool = False, out_bits: int = 0, acc=None):
    """One layer on M-bit inputs with 16-bit weights: conv16w_acc rounded
    once to fp32, then f32_acc_epilogue with the inputs' code shift."""
    if acc is None:
        acc = conv16w_acc(a_levels, w16, a_bits, stride, pad)
    return f32_acc_epilogue(acc, level_shift(a_bits), mode, s, k, b, residual, pool, out_bits)
