"""Seeded synthetic inputs shaped like the paper's workloads.

This module only draws random numbers (``torch.Generator`` on the CPU) and
lays them out in the shapes of the workloads; it holds none of the method's
arithmetic (no quantization, packing, convolution or normalisation).  Both
the GPU path and the CPU oracle consume the same host arrays drawn here.

Recipe (stands in for CIFAR-10 32x32x3 and ImageNet 224x224x3 crops, which
are not available; Sec. IV-B and IV-D describe the real data):

* one generator per workload, seed = 1000 + workload number;
* tensors drawn in the order they are listed by each function;
* "uniform +-1" operands are drawn as a latent U(-1, 1) and quantized later
  by the sign quantizer, which gives exactly uniform +-1;
* ``N(0, v)`` is a variance ``v``; weights of He-initialised layers use
  ``v = 2 / fan_in``;
* batch-norm statistics are fixed, not drawn: mean 0, variance = fan-in for
  quantized layers (integer-level units), 2 for the fp32 first layer;
  eps = 1e-5; gamma ~ U(0.5, 1.5), beta ~ N(0, 0.1).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import torch

BN_EPS = 1e-5


def generator(seed: int) -> torch.Generator:
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed))
    return g


def uniform(g: torch.Generator, shape, lo: float = -1.0, hi: float = 1.0) -> torch.Tensor:
    return torch.rand(shape, generator=g, dtype=torch.float32) * (hi - lo) + lo


def normal(g: torch.Generator, shape, var: float = 1.0) -> torch.Tensor:
    return torch.randn(shape, generator=g, dtype=torch.float32) * math.sqrt(var)


def bn_params(g: torch.Generator, c: int, var: float) -> dict:
    """gamma ~ U(0.5, 1.5), beta ~ N(0, 0.1) drawn in that order; mean 0, var fixed."""
    gamma = uniform(g, (c,), 0.5, 1.5)
    beta = normal(g, (c,), 0.1)
    return {
        "gamma": gamma,
        "beta": beta,
        "mean": torch.zeros(c, dtype=torch.float32),
        "var": torch.full((c,), float(var), dtype=torch.float32),
        "eps": BN_EPS,
    }


@dataclass
class ConvLayerCase:
    """One convolution workload: input, weights and (optionally) BN params."""

    name: str
    x: torch.Tensor
    w: torch.Tensor
    a_bits: int
    w_bits: int
    stride: int = 1
    pad: int = 1
    bn: dict | None = None
    meta: dict = field(default_factory=dict)


def conv_case(
    seed: int,
    n: int,
    cin: int,
    h: int,
    w: int,
    cout: int,
    k: int = 3,
    stride: int = 1,
    pad: int = 1,
    a_bits: int = 1,
    w_bits: int = 1,
    x_dist: str = "normal",
    w_dist: str = "uniform",
    with_bn: bool = True,
    name: str = "conv",
) -> ConvLayerCase:
    """Draw x, then W, then (gamma, beta) from one seeded generator."""
    g = generator(seed)
    xs = (n, cin, h, w)
    x = uniform(g, xs) if x_dist == "uniform" else normal(g, xs, 1.0)
    ws = (cout, cin, k, k)
    fan_in = cin * k * k
    wt = uniform(g, ws) if w_dist == "uniform" else normal(g, ws, 2.0 / fan_in)
    bn = bn_params(g, cout, float(fan_in)) if with_bn else None
    return ConvLayerCase(name, x, wt, a_bits, w_bits, stride, pad, bn)


# ---------------------------------------------------------------------------
# Single-layer workloads (sizes of the paper's ConvNet and ResNet-18 layers)
# ---------------------------------------------------------------------------


def workload1(n: int = 4, c: int = 128, hw: int = 32) -> ConvLayerCase:
    """1W1A 3x3 conv, x and W uniform +-1 (latent U(-1,1)), pad value -1.
    Outputs: int32 accumulator and fp32 s_c * acc."""
    return conv_case(1001, n, c, hw, hw, c, 3, 1, 1, 1, 1, "uniform", "uniform", False,
                     f"1w1a_conv_{n}x{c}x{hw}x{hw}")


def workload2(n: int = 256, c: int = 128, hw: int = 32) -> ConvLayerCase:
    """1-bit weights / 2-bit activations 3x3 conv with an fp32 BN epilogue."""
    return conv_case(1002, n, c, hw, hw, c, 3, 1, 1, 2, 1, "normal", "uniform", True,
                     f"1w2a_conv_bn_{n}x{c}x{hw}x{hw}")


def workload7(w_bits: int = 1, n: int = 256, c: int = 128, hw: int = 32) -> ConvLayerCase:
    """16-bit (fp16) inputs with ``w_bits``-bit weights (Table I / Table IV
    rows with 16-bit floating inputs), the 3x3 layer shape of workload 2 with
    an fp32 BN epilogue; seed 1007 + w_bits."""
    return conv_case(1007 + w_bits, n, c, hw, hw, c, 3, 1, 1, 16, w_bits, "normal", "normal", True,
                     f"a16w{w_bits}_conv_bn_{n}x{c}x{hw}x{hw}")


def workload8(a_bits: int = 2, n: int = 256, c: int = 128, hw: int = 32) -> ConvLayerCase:
    """``a_bits``-bit inputs with 16-bit (fp16) weights (Table I rows with
    16-bit weights), the 3x3 layer shape of workload 2 with an fp32 BN
    epilogue; seed 1010 + a_bits."""
    return conv_case(1010 + a_bits, n, c, hw, hw, c, 3, 1, 1, a_bits, 16, "normal", "normal", True,
                     f"a{a_bits}w16_conv_bn_{n}x{c}x{hw}x{hw}")


WORKLOAD5_LAYERS = ((64, 56), (128, 28), (256, 14), (512, 7))


def workload5(layer: int, n: int = 256, c: int | None = None, hw: int | None = None) -> ConvLayerCase:
    """3W3A ResNet-18 3x3 layer ``layer`` (0..3); seed 1005 + 10 * layer."""
    c0, hw0 = WORKLOAD5_LAYERS[layer]
    c = c0 if c is None else c
    hw = hw0 if hw is None else hw
    return conv_case(1005 + 10 * layer, n, c, hw, hw, c, 3, 1, 1, 3, 3, "normal", "normal",
                     True, f"3w3a_conv_{n}x{c}x{hw}x{hw}")


# ---------------------------------------------------------------------------
# Networks
# ---------------------------------------------------------------------------

# ConvNet of the BNN paper used as Model A (Sec. IV-C):
# 128C3-128C3-MP2-256C3-256C3-MP2-512C3-512C3-MP2-FC1024-FC1024-FC10.
CONVNET_A = {"convs": (128, 128, 256, 256, 512, 512), "pools": (False, True, False, True, False, True),
             "fcs": (1024, 1024), "classes": 10}


def convnet_params(seed: int = 1003, batch: int = 256, width: float = 1.0, fc_width: float = 1.0,
                   hw: int = 32, classes: int = 10) -> dict:
    """Input x ~ N(0,1) [batch,3,hw,hw]; then for each layer in order its
    weight (N(0, 2/fan_in)) and, where it has BN, gamma then beta.

    ``width``/``fc_width`` scale the channel counts (Models B-D halve them)."""
    g = generator(seed)
    convs = [max(1, int(round(c * width))) for c in CONVNET_A["convs"]]
    fcs = [max(1, int(round(f * fc_width))) for f in CONVNET_A["fcs"]]
    p: dict = {"x": normal(g, (batch, 3, hw, hw), 1.0), "convs": [], "fcs": [],
               "pools": CONVNET_A["pools"], "hw": hw}
    cin = 3
    for i, co in enumerate(convs):
        fan = cin * 9
        w = normal(g, (co, cin, 3, 3), 2.0 / fan)
        bn = bn_params(g, co, 2.0 if i == 0 else float(fan))
        p["convs"].append({"w": w, "bn": bn})
        cin = co
    side = hw // 8
    fin = cin * side * side
    for f in fcs:
        w = normal(g, (f, fin), 2.0 / fin)
        bn = bn_params(g, f, float(fin))
        p["fcs"].append({"w": w, "bn": bn})
        fin = f
    p["fc_out"] = {"w": normal(g, (classes, fin), 2.0 / fin),
                   "b": torch.zeros(classes, dtype=torch.float32)}
    return p


RESNET18_STAGES = ((64, 1), (128, 2), (256, 2), (512, 2))


def resnet18_params(seed: int = 1004, batch: int = 64, hw: int = 224, classes: int = 1000,
                    width: float = 1.0) -> dict:
    """Input x ~ N(0,1) [batch,3,hw,hw]; stem conv 7x7/2 weight then BN; then
    per block: conv1 weight, bn1, conv2 weight, bn2, [downsample weight, bn];
    then the fc weight (bias 0).  Every weight ~ N(0, 2/fan_in)."""
    g = generator(seed)
    p: dict = {"x": normal(g, (batch, 3, hw, hw), 1.0), "blocks": []}
    c0 = max(1, int(round(64 * width)))
    p["stem"] = {"w": normal(g, (c0, 3, 7, 7), 2.0 / 147.0), "bn": bn_params(g, c0, 2.0)}
    cin = c0
    for cs, stride in RESNET18_STAGES:
        c = max(1, int(round(cs * width)))
        for b in range(2):
            s = stride if b == 0 else 1
            blk: dict = {"stride": s}
            blk["w1"] = normal(g, (c, cin, 3, 3), 2.0 / (cin * 9))
            blk["bn1"] = bn_params(g, c, float(cin * 9))
            blk["w2"] = normal(g, (c, c, 3, 3), 2.0 / (c * 9))
            blk["bn2"] = bn_params(g, c, float(c * 9))
            if s != 1 or cin != c:
                blk["wd"] = normal(g, (c, cin, 1, 1), 2.0 / cin)
                blk["bnd"] = bn_params(g, c, float(cin))
            p["blocks"].append(blk)
            cin = c
    p["fc"] = {"w": normal(g, (classes, cin), 2.0 / cin), "b": torch.zeros(classes, dtype=torch.float32)}
    return p
