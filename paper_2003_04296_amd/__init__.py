"""Python binding of libqconv.so (the C ABI in include/qconv.h).

Argument marshalling only: every step of the quantized path runs in the HIP
kernels of the shared library.  PyTorch supplies device memory and the
current stream.  If the library is not built, every call raises -- there is
no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libqconv.so")

QCONV_OK, QCONV_EINVAL, QCONV_EUNSUPPORTED, QCONV_EWORKSPACE, QCONV_EOVERFLOW, QCONV_EHIP = 0, -1, -2, -3, -4, -5
QCONV_ESCRATCH = -6
ALGO_AUTO, ALGO_BITPLANE, ALGO_MFMA_I8, ALGO_MFMA_FP4, ALGO_MFMA_F16 = 0, 1, 2, 3, 4
EPI_INT32, EPI_SCALE_F32, EPI_BN_F32, EPI_BN_PACK = 0, 1, 2, 3
EPI_POOL2, EPI_RESIDUAL = 1, 2
F32_FMAF_CHAIN, F32_MFMA, F32_BF16X6 = 0, 1, 2
OP_NAMES = {1: "XNOR", 2: "SHIFT", 3: "XNOR-ADDER", 4: "SHIFT-ADDER", 5: "MAC"}

EXPORTED = (
    "qconv_error_string", "qconv_version", "qconv_inference_op", "qconv_packed_act_bytes",
    "qconv_pack_act", "qconv_packed_weight_bytes", "qconv_pack_weight", "qconv_fold_bn",
    "qconv_out_size", "qconv_forward", "qnet_create", "qnet_destroy", "qnet_add_conv_f32",
    "qnet_add_maxpool_f32", "qnet_add_quantize", "qnet_add_qconv", "qnet_add_avgpool",
    "qnet_add_fc_f32", "qnet_workspace_bytes", "qnet_forward", "qnet_forward_range", "qnet_num_layers",
    "qnet_forward_noalloc", "qnet_noalloc_bytes", "qnet_noalloc_limit", "qnet_set_f32_algo", "qnet_layer_fused_into",
    "qnet_layer_kernel",
    "qnet_tensor_info", "qconv_resolve_algo",
    "qconv_kernel_name", "aqe_forward", "aqe_backward", "aqe_sgd_clip",
)


class QconvError(RuntimeError):
    def __init__(self, status: int, what: str = ""):
        self.status = status
        msg = _lib_or_none().qconv_error_string(status).decode() if _lib_or_none() else str(status)
        super().__init__(f"{what}: {msg} ({status})" if what else f"{msg} ({status})")


class qconv_desc(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int) for name in
                ("n", "cin", "h", "w", "cout", "kh", "kw", "stride", "pad", "a_bits", "w_bits", "algo")]


class qconv_epilogue(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int), ("flags", ctypes.c_int), ("scale", ctypes.c_void_p),
                ("bn_k", ctypes.c_void_p), ("bn_b", ctypes.c_void_p), ("residual", ctypes.c_void_p),
                ("out_bits", ctypes.c_int), ("out_thresholds", ctypes.c_void_p)]


_lib = None


def _lib_or_none():
    return _lib


def lib() -> ctypes.CDLL:
    """Load the HIP library; raise loudly if it was not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -c 'import __graft_entry__ as g; g.build()'`"
                           " (the quantized path has no CPU fallback)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    L.qconv_error_string.restype = ctypes.c_char_p
    L.qconv_error_string.argtypes = [i32]
    L.qconv_version.restype = i32
    L.qconv_inference_op.argtypes = [i32, i32, ctypes.POINTER(i32), ctypes.POINTER(i32)]
    L.qconv_packed_act_bytes.restype = sz
    L.qconv_packed_act_bytes.argtypes = [i32] * 5
    L.qconv_pack_act.argtypes = [vp, i32, i32, i32, i32, i32, vp, vp, vp]
    L.qconv_packed_weight_bytes.restype = sz
    L.qconv_packed_weight_bytes.argtypes = [i32] * 5
    L.qconv_pack_weight.argtypes = [vp, i32, i32, i32, i32, i32, vp, vp, vp, vp]
    L.qconv_fold_bn.argtypes = [vp, vp, vp, vp, ctypes.c_double, i32, vp, vp]
    L.qconv_out_size.argtypes = [i32] * 4
    L.qconv_forward.argtypes = [ctypes.POINTER(qconv_desc), vp, vp, ctypes.POINTER(qconv_epilogue), vp, vp, vp]
    L.qconv_resolve_algo.argtypes = [ctypes.POINTER(qconv_desc), ctypes.POINTER(qconv_epilogue)]
    L.qconv_kernel_name.argtypes = [ctypes.POINTER(qconv_desc), ctypes.POINTER(qconv_epilogue), i32,
                                    ctypes.c_char_p, i32]
    i64 = ctypes.c_int64
    f32 = ctypes.c_float
    L.aqe_forward.argtypes = [vp, i64, i32, f32, vp, vp, i64, vp, vp]
    L.aqe_backward.argtypes = [vp, vp, i64, f32, vp, vp]
    L.aqe_sgd_clip.argtypes = [vp, vp, i64, f32, vp]
    L.qnet_create.restype = vp
    L.qnet_create.argtypes = [i32, i32, i32]
    L.qnet_destroy.argtypes = [vp]
    L.qnet_add_conv_f32.argtypes = [vp, i32, vp, i32, i32, i32, i32, vp, vp, i32, i32]
    L.qnet_add_maxpool_f32.argtypes = [vp, i32, i32, i32, i32]
    L.qnet_add_quantize.argtypes = [vp, i32, i32]
    L.qnet_add_qconv.argtypes = [vp, i32, vp, i32, i32, i32, i32, i32, i32, vp, vp, i32, i32]
    L.qnet_add_avgpool.argtypes = [vp, i32]
    L.qnet_add_fc_f32.argtypes = [vp, i32, vp, vp, i32]
    L.qnet_workspace_bytes.restype = sz
    L.qnet_workspace_bytes.argtypes = [vp, i32]
    L.qnet_forward.argtypes = [vp, vp, i32, vp, vp, sz, vp]
    L.qnet_forward_range.argtypes = [vp, vp, i32, vp, vp, sz, i32, i32, vp]
    L.qnet_num_layers.argtypes = [vp]
    L.qnet_forward_noalloc.argtypes = [vp, vp, i32, vp, vp]
    L.qnet_noalloc_bytes.restype = sz
    L.qnet_noalloc_bytes.argtypes = [vp, i32]
    L.qnet_noalloc_limit.restype = sz
    L.qnet_noalloc_limit.argtypes = []
    L.qnet_set_f32_algo.argtypes = [vp, i32]
    L.qnet_layer_fused_into.argtypes = [vp, i32]
    L.qnet_layer_kernel.argtypes = [vp, i32, i32, ctypes.c_char_p, i32]
    L.qnet_tensor_info.argtypes = [vp, i32, i32] + [ctypes.POINTER(i32)] * 4 + [ctypes.POINTER(sz)]
    _lib = L
    return L


def _check(rc: int, what: str) -> int:
    if rc < 0:
        raise QconvError(rc, what)
    return rc


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch

    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


# threshold values a quantizer of `bits` reads (Eq. 21: one delta; Eq. 22: three)
_THR_COUNT = {1: 0, 2: 1, 3: 3}


def _host_thr(vals, bits: int, what: str):
    """Host float array of the thresholds for `bits` (None = the defaults).
    The C side reads exactly 1 value for 2 bits and 3 for 3 bits, so the
    length is checked here; 1-bit and 16-bit quantizers take none."""
    if vals is None:
        return None
    vals = [float(v) for v in (vals.tolist() if hasattr(vals, "tolist") else vals)]
    need = _THR_COUNT.get(bits, 0)
    if need == 0:
        return None
    if len(vals) != need:
        raise ValueError(f"{what}: {bits}-bit thresholds take {need} value(s), got {len(vals)}")
    return (ctypes.c_float * need)(*vals)


def planes(bits: int) -> int:
    return {1: 1, 2: 2, 3: 4}[bits]


def out_size(n: int, k: int, stride: int, pad: int) -> int:
    return _check(lib().qconv_out_size(n, k, stride, pad), "qconv_out_size")


def inference_op(m_bits: int, n_bits: int):
    op, prec = ctypes.c_int(), ctypes.c_int()
    _check(lib().qconv_inference_op(m_bits, n_bits, ctypes.byref(op), ctypes.byref(prec)), "qconv_inference_op")
    return OP_NAMES[op.value], prec.value


def packed_act_words(n, c, h, w, bits) -> int:
    return lib().qconv_packed_act_bytes(n, c, h, w, bits) // 4


def packed_weight_words(cout, cin, kh, kw, bits) -> int:
    return lib().qconv_packed_weight_bytes(cout, cin, kh, kw, bits) // 4


def pack_act(x, bits: int, thresholds=None, out=None, stream=None):
    """fp32 NCHW device tensor -> packed bitplanes [n][h][w][cw][P] (int32 view);
    bits = 16: the fp16 channel-last tensor [n][h][w][cw * 32] (int32 view)."""
    import torch

    n, c, h, w = x.shape
    if out is None:
        out = torch.empty(packed_act_words(n, c, h, w, bits), dtype=torch.int32, device=x.device)
    t = _host_thr(thresholds, bits, "pack_act")
    _check(lib().qconv_pack_act(_ptr(x), n, c, h, w, bits, t, _ptr(out), _stream(stream)), "qconv_pack_act")
    return out


def pack_weight(w, bits: int, base_thresholds=None, stream=None, out=None):
    """fp32 OIHW device tensor -> (packed weights, s_c); out = (words, scale)
    reuses existing buffers."""
    import torch

    cout, cin, kh, kw = w.shape
    if out is None:
        out = torch.empty(packed_weight_words(cout, cin, kh, kw, bits), dtype=torch.int32, device=w.device)
        scale = torch.empty(cout, dtype=torch.float32, device=w.device)
    else:
        out, scale = out
    t = _host_thr(base_thresholds, bits, "pack_weight")
    _check(lib().qconv_pack_weight(_ptr(w), cout, cin, kh, kw, bits, t, _ptr(out), _ptr(scale), _stream(stream)),
           "qconv_pack_weight")
    return out, scale


def aqe_forward(x, bits: int, alpha: float, thresholds=None, scale=None, group_size: int = 0, out=None, stream=None):
    """AQE forward y = alpha h(x) + (1 - alpha) x (device fp32 tensors);
    weights: pass scale (s_c per group) and group_size (values per group)."""
    import torch

    y = torch.empty_like(x) if out is None else out
    t = _host_thr(thresholds, bits, "aqe_forward")
    _check(lib().aqe_forward(_ptr(x), x.numel(), bits, float(alpha), t, _ptr(scale), int(group_size), _ptr(y),
                             _stream(stream)), "aqe_forward")
    return y


def aqe_backward(x, gy, alpha: float, out=None, stream=None):
    """AQE backward gx = 2 alpha gy 1{|x| <= 1}."""
    import torch

    gx = torch.empty_like(gy) if out is None else out
    _check(lib().aqe_backward(_ptr(x), _ptr(gy), x.numel(), float(alpha), _ptr(gx), _stream(stream)), "aqe_backward")
    return gx


def aqe_sgd_clip(w, g, lr: float, stream=None):
    """In place: w = clip(w - lr g, -1, 1)."""
    _check(lib().aqe_sgd_clip(_ptr(w), _ptr(g), w.numel(), float(lr), _stream(stream)), "aqe_sgd_clip")
    return w


def fold_bn(gamma, beta, mean, var, eps):
    """Host fold of BN parameters (numpy/CPU arrays) -> (k, b) float32 numpy."""
    import numpy as np

    g, b, m, v = (np.ascontiguousarray(np.asarray(a, dtype=np.float32)) for a in (gamma, beta, mean, var))
    c = g.size
    k = np.empty(c, np.float32)
    bb = np.empty(c, np.float32)
    P = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    _check(lib().qconv_fold_bn(P(g), P(b), P(m), P(v), ctypes.c_double(float(eps)), c, P(k), P(bb)), "qconv_fold_bn")
    return k, bb


def conv(act_packed, w_packed, n, cin, h, w, cout, k, stride, pad, a_bits, w_bits, mode=EPI_INT32,
         flags=0, scale=None, bn_k=None, bn_b=None, residual=None, out_bits=0, out=None, out_packed=None,
         algo=ALGO_AUTO, stream=None, out_thresholds=None):
    """qconv_forward; allocates the outputs the epilogue needs when not given."""
    import torch

    ho, wo = out_size(h, k, stride, pad), out_size(w, k, stride, pad)
    if flags & EPI_POOL2:
        ho, wo = ho // 2, wo // 2
    dev = act_packed.device
    if out is None and mode != EPI_BN_PACK:
        dt = torch.int32 if mode == EPI_INT32 else torch.float32
        out = torch.empty((n, cout, ho, wo), dtype=dt, device=dev)
    if out_packed is None and mode == EPI_BN_PACK:
        out_packed = torch.empty(packed_act_words(n, cout, ho, wo, out_bits), dtype=torch.int32, device=dev)
    d = qconv_desc(n, cin, h, w, cout, k, k, stride, pad, a_bits, w_bits, algo)
    thr = _host_thr(out_thresholds, out_bits, "conv") if out_thresholds is not None else None  # alive across the call
    e = qconv_epilogue(mode, flags, _ptr(scale), _ptr(bn_k), _ptr(bn_b), _ptr(residual), out_bits,
                       ctypes.cast(thr, ctypes.c_void_p) if thr is not None else None)
    _check(lib().qconv_forward(ctypes.byref(d), _ptr(act_packed), _ptr(w_packed), ctypes.byref(e), _ptr(out),
                               _ptr(out_packed), _stream(stream)), "qconv_forward")
    return out, out_packed


ALGO_NAMES = {ALGO_BITPLANE: "bitplane", ALGO_MFMA_I8: "mfma_i8", ALGO_MFMA_FP4: "mfma_fp4", ALGO_MFMA_F16: "mfma_f16"}


def resolve_algo(n, cin, h, w, cout, k, stride, pad, a_bits, w_bits, mode=EPI_INT32, flags=0, out_bits=0,
                 algo=ALGO_AUTO) -> int:
    """The concrete algorithm qconv_forward would run (launches nothing)."""
    d = qconv_desc(n, cin, h, w, cout, k, k, stride, pad, a_bits, w_bits, algo)
    e = qconv_epilogue(mode, flags, None, None, None, None, out_bits, None)
    return _check(lib().qconv_resolve_algo(ctypes.byref(d), ctypes.byref(e)), "qconv_resolve_algo")


def kernel_name(n, cin, h, w, cout, k, stride, pad, a_bits, w_bits, mode=EPI_INT32, flags=0, out_bits=0,
                algo=ALGO_AUTO, packed_out=False) -> str:
    """The GPU kernel instantiation qconv_forward would launch on the current
    device, as a profiler names it (launches nothing)."""
    d = qconv_desc(n, cin, h, w, cout, k, k, stride, pad, a_bits, w_bits, algo)
    e = qconv_epilogue(mode, flags, None, None, None, None, out_bits, None)
    buf = ctypes.create_string_buffer(128)
    _check(lib().qconv_kernel_name(ctypes.byref(d), ctypes.byref(e), int(bool(packed_out)), buf, 128),
           "qconv_kernel_name")
    return buf.value.decode()


class Net:
    """A qnet layer list (tensor ids as in include/qconv.h)."""

    def __init__(self, in_c: int, in_h: int, in_w: int, f32_algo: int = F32_MFMA):
        self._h = lib().qnet_create(in_c, in_h, in_w)
        if not self._h:
            raise QconvError(QCONV_EINVAL, "qnet_create")
        _check(lib().qnet_set_f32_algo(self._h, int(f32_algo)), "qnet_set_f32_algo")
        self.f32_algo = f32_algo
        self._keep = []  # device tensors the layers point at
        self.layers = []  # per layer: what was added (kind, source, parameters), for reports

    def __del__(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.qnet_destroy(self._h)
            self._h = None

    def _add(self, rc, what, *keep, **info):
        self._keep.extend(k for k in keep if k is not None)
        tid = _check(rc, what)
        self.layers.append(dict(kind=what.replace("qnet_add_", ""), dst=tid, **info))
        return tid

    def fused_into(self, layer):
        """The earlier layer whose epilogue writes layer `layer`'s tensor, or None."""
        if layer < 0:
            return None
        r = _check(lib().qnet_layer_fused_into(self._h, layer), "qnet_layer_fused_into")
        return None if r == layer else r

    def layer_kernel(self, layer, batch):
        """The GPU kernel layer `layer` launches ("" when an earlier layer writes its tensor)."""
        buf = ctypes.create_string_buffer(128)
        _check(lib().qnet_layer_kernel(self._h, layer, batch, buf, 128), "qnet_layer_kernel")
        return buf.value.decode()

    def _mark_fused(self, tid):
        """Record (for reports) which layer writes the tensor a layer just added."""
        li = tid - 1
        prod = self.fused_into(li)
        self.layers[li]["fused_into"] = prod
        if prod is not None:
            key = "pool_dst" if self.layers[li]["kind"] == "maxpool_f32" else "pack_dst"
            self.layers[prod][key] = tid
        return tid

    def conv_f32(self, src, w, bn_k, bn_b, stride=1, pad=0, relu=False, out_bits=0):
        cout, _, k, _ = w.shape
        return self._add(lib().qnet_add_conv_f32(self._h, src, _ptr(w), cout, k, stride, pad, _ptr(bn_k), _ptr(bn_b),
                                                 int(relu), out_bits), "qnet_add_conv_f32", w, bn_k, bn_b,
                         src=src, cout=cout, k=k, stride=stride, pad=pad, out_bits=out_bits)

    def maxpool_f32(self, src, k, stride, pad):
        return self._mark_fused(self._add(lib().qnet_add_maxpool_f32(self._h, src, k, stride, pad),
                                          "qnet_add_maxpool_f32", src=src, k=k, stride=stride, pad=pad))

    def quantize(self, src, bits):
        return self._mark_fused(self._add(lib().qnet_add_quantize(self._h, src, bits), "qnet_add_quantize", src=src,
                                          out_bits=bits))

    def qconv(self, src, w_packed, cout, k, stride, pad, w_bits, bn_k, bn_b, pool2=False, residual_src=-1,
              out_bits=0):
        return self._add(lib().qnet_add_qconv(self._h, src, _ptr(w_packed), cout, k, stride, pad, w_bits, int(pool2),
                                              _ptr(bn_k), _ptr(bn_b), residual_src, out_bits),
                         "qnet_add_qconv", w_packed, bn_k, bn_b, src=src, cout=cout, k=k, stride=stride, pad=pad,
                         w_bits=w_bits, pool2=bool(pool2), residual_src=residual_src, out_bits=out_bits)

    def avgpool(self, src):
        return self._add(lib().qnet_add_avgpool(self._h, src), "qnet_add_avgpool", src=src)

    def fc_f32(self, src, w, bias=None):
        return self._add(lib().qnet_add_fc_f32(self._h, src, _ptr(w), _ptr(bias), w.shape[0]), "qnet_add_fc_f32",
                         w, bias, src=src, cout=w.shape[0])

    def workspace_bytes(self, batch):
        return lib().qnet_workspace_bytes(self._h, batch)

    def tensor_info(self, tid, batch):
        c, h, w, b = (ctypes.c_int() for _ in range(4))
        off = ctypes.c_size_t()
        _check(lib().qnet_tensor_info(self._h, tid, batch, ctypes.byref(c), ctypes.byref(h), ctypes.byref(w),
                                      ctypes.byref(b), ctypes.byref(off)), "qnet_tensor_info")
        return c.value, h.value, w.value, b.value, off.value

    def forward(self, x, logits, workspace, stream=None):
        nbytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
        _check(lib().qnet_forward(self._h, _ptr(x), x.shape[0], _ptr(logits), _ptr(workspace), nbytes,
                                  _stream(stream)), "qnet_forward")
        return logits

    def forward_range(self, x, logits, workspace, first, count, stream=None):
        """Layers [first, first + count) of forward() on the same workspace."""
        nbytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
        _check(lib().qnet_forward_range(self._h, _ptr(x), x.shape[0], _ptr(logits), _ptr(workspace), nbytes,
                                        int(first), int(count), _stream(stream)), "qnet_forward_range")
        return logits

    def forward_noalloc(self, x, logits, stream=None):
        """forward() on the library's fixed scratch array instead of a workspace."""
        _check(lib().qnet_forward_noalloc(self._h, _ptr(x), x.shape[0], _ptr(logits), _stream(stream)),
               "qnet_forward_noalloc")
        return logits

    def noalloc_bytes(self, batch):
        return lib().qnet_noalloc_bytes(self._h, batch)

    def num_layers(self):
        return _check(lib().qnet_num_layers(self._h), "qnet_num_layers")
