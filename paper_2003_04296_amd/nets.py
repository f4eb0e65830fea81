"""Network builders on the qnet API: the ConvNet used as Model A (Sec. IV-C)
and ResNet-18 (Sec. IV-D, Table V), from a parameter dict of fp32 host
tensors (see synth.py for the layout).

Weights are quantized and packed on the GPU by qconv_pack_weight, BN is
folded on the host by qconv_fold_bn; the returned object keeps every device
buffer alive and runs qnet_forward."""
from __future__ import annotations

import torch

from . import F32_BF16X6, F32_MFMA, Net, fold_bn, pack_weight


def _dev_bn(bn, device):
    k, b = fold_bn(bn["gamma"].numpy(), bn["beta"].numpy(), bn["mean"].numpy(), bn["var"].numpy(), bn["eps"])
    return torch.from_numpy(k).to(device), torch.from_numpy(b).to(device)


class QNetwork:
    def __init__(self, net: Net, in_shape, out_features: int, device, ids: dict):
        self.net = net
        self.in_shape = in_shape
        self.out_features = out_features
        self.device = device
        self.ids = ids
        self._ws = None
        self._ws_batch = -1

    def workspace(self, batch: int):
        if self._ws_batch != batch:
            nbytes = self.net.workspace_bytes(batch)
            self._ws = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=self.device)
            self._ws_batch = batch
        return self._ws

    def forward(self, x, logits=None, stream=None):
        batch = x.shape[0]
        if logits is None:
            logits = torch.empty((batch, self.out_features), dtype=torch.float32, device=self.device)
        self.net.forward(x, logits, self.workspace(batch), stream)
        return logits

    def tensor(self, tid: int, batch: int):
        """View of intermediate tensor `tid` in the workspace after forward()."""
        c, h, w, bits, off = self.net.tensor_info(tid, batch)
        ws = self._ws
        if bits == 0:
            n = batch * c * h * w
            return ws[off:off + 4 * n].view(torch.float32).view(batch, c, h, w), bits
        words = batch * h * w * ((c + 31) // 32) * {1: 1, 2: 2, 3: 4}[bits]
        return ws[off:off + 4 * words].view(torch.int32), bits


def build_convnet(p: dict, device, a_bits: int = 1, w_bits: int = 1, f32_algo: int = F32_MFMA) -> QNetwork:
    """fp32 conv1 -> BN -> sign; binary convs with 2x2 max pool before BN
    where the topology has one; binary FCs (the first as a conv covering the
    whole 4x4 map, so its (c, h, w) weight order is the conv's OIHW order);
    fp32 FC + bias.  f32_algo: the fp32 first conv on the matrix cores
    (default) or as fixed fmaf chains (bit-exact against the oracle)."""
    hw = p["hw"]
    net = Net(3, hw, hw, f32_algo)
    ids = {}
    c1 = p["convs"][0]
    k, b = _dev_bn(c1["bn"], device)
    t = net.conv_f32(0, c1["w"].to(device), k, b, stride=1, pad=1, relu=False, out_bits=a_bits)
    ids["conv1"] = t
    cin = c1["w"].shape[0]
    for i, layer in enumerate(p["convs"][1:], start=1):
        w = layer["w"].to(device)
        wq, _ = pack_weight(w, w_bits)
        k, b = _dev_bn(layer["bn"], device)
        t = net.qconv(t, wq, w.shape[0], 3, 1, 1, w_bits, k, b, pool2=p["pools"][i], out_bits=a_bits)
        ids[f"conv{i + 1}"] = t
        cin = w.shape[0]
    side = hw // 8
    for j, fc in enumerate(p["fcs"]):
        w = fc["w"]
        kk = side if j == 0 else 1
        w4 = w.reshape(w.shape[0], -1, kk, kk).contiguous().to(device)
        wq, _ = pack_weight(w4, w_bits)
        k, b = _dev_bn(fc["bn"], device)
        t = net.qconv(t, wq, w.shape[0], kk, 1, 0, w_bits, k, b, out_bits=1 if j == len(p["fcs"]) - 1 else a_bits)
        ids[f"fc{j + 1}"] = t
    fo = p["fc_out"]
    t = net.fc_f32(t, fo["w"].to(device), fo["b"].to(device))
    ids["logits"] = t
    return QNetwork(net, (3, hw, hw), fo["w"].shape[0], device, ids)


def build_resnet18(p: dict, device, a_bits: int = 2, w_bits: int = 2, f32_algo: int = F32_BF16X6) -> QNetwork:
    """fp32 stem conv 7x7/2 -> BN -> ReLU -> max pool 3x3/2; eight basic
    blocks with quantized convs (q = Q(x); y = Q(BN1(q*W1)); out = BN2(y*W2)
    + shortcut, shortcut = x or BN_d(q*W_d)); average pool; fp32 FC.  With a
    matrix-core fp32 algorithm the stem's max pooling and the first block's
    quantize run in the stem conv's epilogue; the default runs the stem on
    the bf16 matrix cores through exact three-way splits (fp32 accuracy, see
    QNET_F32_BF16X6 in include/qconv.h)."""
    _, _, hh, ww = p["x"].shape
    net = Net(3, hh, ww, f32_algo)
    ids = {}
    st = p["stem"]
    k, b = _dev_bn(st["bn"], device)
    t = net.conv_f32(0, st["w"].to(device), k, b, stride=2, pad=3, relu=True, out_bits=0)
    x = net.maxpool_f32(t, 3, 2, 1)
    ids["stem"] = x
    for i, blk in enumerate(p["blocks"]):
        s = blk["stride"]
        q = net.quantize(x, a_bits)
        w1 = blk["w1"].to(device)
        c = w1.shape[0]
        wq1, _ = pack_weight(w1, w_bits)
        k1, b1 = _dev_bn(blk["bn1"], device)
        y = net.qconv(q, wq1, c, 3, s, 1, w_bits, k1, b1, out_bits=a_bits)
        if "wd" in blk:
            wqd, _ = pack_weight(blk["wd"].to(device), w_bits)
            kd, bd = _dev_bn(blk["bnd"], device)
            sc = net.qconv(q, wqd, c, 1, s, 0, w_bits, kd, bd, out_bits=0)
        else:
            sc = x
        wq2, _ = pack_weight(blk["w2"].to(device), w_bits)
        k2, b2 = _dev_bn(blk["bn2"], device)
        x = net.qconv(y, wq2, c, 3, 1, 1, w_bits, k2, b2, residual_src=sc, out_bits=0)
        ids[f"block{i}"] = x
    f = net.avgpool(x)
    fc = p["fc"]
    t = net.fc_f32(f, fc["w"].to(device), fc["b"].to(device))
    ids["logits"] = t
    return QNetwork(net, (3, hh, ww), fc["w"].shape[0], device, ids)
