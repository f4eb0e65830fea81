#!/usr/bin/env python3
"""Throughput of the quantized-convolution hot path on one MI355X.

The default run measures the five workloads of the metric ("quantized-conv
GOPS (1W1A, 2W2A, 3W3A) + images/sec fwd; % of roofline") and prints ONE
JSON line.  Its headline fields are the 1-bit-weight / 2-bit-activation 3x3
convolution over a batch of 256 x 128 x 32 x 32 fp32 activations with 128
output channels and a fused fp32 batch-norm epilogue; one step = quantize +
pack the fp32 input (qconv_pack_act) + the convolution with its epilogue
(qconv_forward); weights are packed once beforehand, as at inference.  The
"configs" object carries every workload:

  1  1W1A layer 4 x 128 x 32 x 32 -> 128, int32 accumulators scaled by s_c
  2  the headline layer above
  3  ConvNet (Model A widths) forward at 1W1A, batch 256, 32 x 32 (images/s)
  4  ResNet-18 forward at 2W2A, batch 64, 224 x 224 (images/s)
  5  the four ResNet-18 3x3 layer shapes at 3W3A, batch 256, int32 output

Each entry gives the throughput of its step, the roofline of its dominant
kernel (achieved = algorithmic work of one launch / its average duration,
measured with HIP events on the launch stream) and the CPU oracle timed on a
bounded sample of the same workload.  Networks also report every layer's
time against its own roofline.

Other single workloads: --workload 1w1a | 1w2a | 3w3a-L{0..3} |
a16w{1,2,3} | a{1,2,3}w16 | convnet | convnet_w16 | resnet18 | aqe.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import paper_2003_04296_amd as q  # noqa: E402
from paper_2003_04296_amd import synth  # noqa: E402

METRIC = "quantized-conv GOPS (1W1A, 2W2A, 3W3A) + images/sec fwd; % of roofline"

# MI355X figures: 256 CUs x 64 lanes x 2.4 GHz of 32-bit VALU issue.
VALU_LANE_OPS = 256 * 64 * 2.4e9
HBM_PEAK_GBS = 8000.0
FP32_PEAK_GOPS = 157.3e3  # fp32 vector and fp32 matrix cores alike
# dense matrix-core peaks (ops = 2 per MAC), in G: int8 5.0 POP/s, fp4 10.1 PFLOP/s, fp16 2.5 PFLOP/s
MFMA_PEAK_GOPS = {"mfma_i8": 5.0e6, "mfma_fp4": 10.1e6, "mfma_f16": 2.5e6, "mfma_bf16": 2.5e6}
# an fp32 conv through exact three-way bf16 splits costs six bf16 products
# per multiply-add: its roofline is the bf16 peak over six, in fp32 conv-ops
BF16X6_PEAK_GOPS = MFMA_PEAK_GOPS["mfma_bf16"] / 6
# Minimal VALU recipe (lane-ops per 32-channel word pair) of the bitplane
# product on gfx950, where v_bitop3_b32 fuses any 3-input bit function:
#   1W1A: xor, bcnt                         -> 2
#   1W2A / 2W1A: bitop3(xor & mask), bcnt   -> 2  (activation-only popcount amortised)
#   2W2A: bitop3, and, and, 2 bcnt          -> 5
#   3W3A: 9 and/and_or (shift classes), 5 x (bitop3 + 2 bcnt) -> 24
LANE_OPS_PER_WORD = {(1, 1): 2, (2, 1): 2, (1, 2): 2, (2, 2): 5, (3, 3): 24}
# the arithmetic each contraction really performs
ALGO_DTYPE = {"mfma_fp4": "e2m1 x e2m1 -> f32 (exact integers)", "mfma_i8": "i8 x i8 -> i32",
              "bitplane": "u32 bitplanes, popcount -> i32", "mfma_f16": "f16 x f16 -> f32"}


def valu_peak_gops(a_bits, w_bits):
    ops = LANE_OPS_PER_WORD.get((a_bits, w_bits))
    if ops is None:
        return None
    return VALU_LANE_OPS * 32.0 / ops * 2.0 / 1e9  # conv-ops (2 per MAC) per second, in G


def compute_peak(used, a_bits, w_bits):
    """(peak in GOPS, bound name) of the contraction an algorithm runs."""
    if used == "bitplane":
        return valu_peak_gops(a_bits, w_bits), "alu"
    return MFMA_PEAK_GOPS[used], "mfma"


def _fold(bn, dev):
    k, b = q.fold_bn(bn["gamma"].numpy(), bn["beta"].numpy(), bn["mean"].numpy(), bn["var"].numpy(), bn["eps"])
    return torch.from_numpy(k).to(dev), torch.from_numpy(b).to(dev)


def packed_bytes(n, c, h, w, bits):
    return q.packed_act_words(n, c, h, w, bits) * 4 if bits else n * c * h * w * 4


def weight_operand_bytes(cout, cin, k, used, w_bits):
    """Bytes of the part of the packed weights an algorithm reads."""
    taps, cw, cop = k * k, (cin + 31) // 32, (cout + 127) // 128 * 128
    if used == "bitplane":
        return taps * cw * cop * q.planes(w_bits) * 4
    return {"mfma_i8": taps * cw * cop * 32, "mfma_fp4": taps * ((cw + 1) // 2) * cop * 32,
            "mfma_f16": taps * 2 * cw * cop * 32}[used]


class ConvWorkload:
    """pack_act + qconv_forward on one synthetic layer."""

    def __init__(self, case, dev, mode, algo, out_bits=0):
        self.case = case
        self.dev = dev
        self.mode = mode
        self.algo = algo
        self.out_bits = out_bits
        n, c, h, w = case.x.shape
        self.shape = (n, c, h, w)
        self.cout = case.w.shape[0]
        self.k = case.w.shape[2]
        self.x = case.x.to(dev)
        self.wq, self.scale = q.pack_weight(case.w.to(dev), case.w_bits)
        if case.bn is not None:
            self.bn_k, self.bn_b = _fold(case.bn, dev)
        else:
            self.bn_k = self.bn_b = None
        self.act = torch.empty(q.packed_act_words(n, c, h, w, case.a_bits), dtype=torch.int32, device=dev)
        ho = q.out_size(h, self.k, case.stride, case.pad)
        wo = q.out_size(w, self.k, case.stride, case.pad)
        self.out_shape = (n, self.cout, ho, wo)
        if mode == q.EPI_BN_PACK:
            self.out = None
            self.outp = torch.empty(q.packed_act_words(n, self.cout, ho, wo, out_bits), dtype=torch.int32, device=dev)
        else:
            dt = torch.int32 if mode == q.EPI_INT32 else torch.float32
            self.out = torch.empty(self.out_shape, dtype=dt, device=dev)
            self.outp = None
        self.macs = n * self.cout * ho * wo * c * self.k * self.k
        self.used = q.ALGO_NAMES[q.resolve_algo(n, c, h, w, self.cout, self.k, case.stride, case.pad, case.a_bits,
                                                case.w_bits, mode, 0, out_bits, algo)]
        self.kname = q.kernel_name(n, c, h, w, self.cout, self.k, case.stride, case.pad, case.a_bits, case.w_bits,
                                   mode=mode, out_bits=out_bits, algo=algo, packed_out=mode == q.EPI_BN_PACK)

    def pack(self):
        q.pack_act(self.x, self.case.a_bits, out=self.act)

    def conv(self):
        n, c, h, w = self.shape
        q.conv(self.act, self.wq, n, c, h, w, self.cout, self.k, self.case.stride, self.case.pad,
               self.case.a_bits, self.case.w_bits, mode=self.mode, scale=self.scale, bn_k=self.bn_k,
               bn_b=self.bn_b, out=self.out, out_packed=self.outp, out_bits=self.out_bits, algo=self.algo)

    def step(self):
        self.pack()
        self.conv()

    def conv_bytes(self):
        """Algorithmic HBM bytes of one conv launch: packed (or fp16) input +
        the part of the packed weights the algorithm reads + output."""
        n, c, h, w = self.shape
        a = packed_bytes(n, c, h, w, self.case.a_bits)
        wb = weight_operand_bytes(self.cout, c, self.k, self.used, self.case.w_bits)
        if self.mode == q.EPI_BN_PACK:
            o = packed_bytes(*self.out_shape, self.out_bits)
        else:
            o = int(np.prod(self.out_shape)) * 4
        return a + wb + o

    def pack_bytes(self):
        n, c, h, w = self.shape
        return n * c * h * w * 4 + q.packed_act_words(n, c, h, w, self.case.a_bits) * 4


def measured_traffic(workload: str, kernel: str, layer=None):
    """HBM bytes per launch of `kernel` on `workload` (of network layer `layer`
    when given) from the committed rocprofv3 counter runs, or None when there
    is no record or the kernel's sources changed since the counters were
    taken."""
    import hashlib

    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path)).get(workload)
    if not rec:
        return None

    def unchanged(sources, digest):
        h = hashlib.sha256()
        for src in sources:
            fp = os.path.join(ROOT, src)
            if not os.path.exists(fp):
                return False
            h.update(open(fp, "rb").read())
        return h.hexdigest() == digest

    if layer is not None and str(layer) in rec.get("layers", {}):
        lr = rec["layers"][str(layer)]
        if lr["kernel"] != kernel or not unchanged(rec["layer_sources"], rec["layer_sources_sha256"]):
            return None
        return lr["fetch_bytes"] + lr["write_bytes"]
    if rec["kernel"] != kernel or not unchanged(rec["sources"], rec["sources_sha256"]):
        return None
    return rec["fetch_bytes"] + rec["write_bytes"]


def _fill_queue(stream, us=3000):
    """Keep the GPU busy for about `us` microseconds (a device-side spin on
    the launch stream), so that the launches enqueued behind it run back to
    back: the events then time the kernels, not the host's launch rate."""
    sleep = getattr(torch.cuda, "_sleep", None)
    if sleep is not None:
        with torch.cuda.stream(stream):
            sleep(int(us * 2000))  # about 2 k cycles per microsecond


def time_kernel(fn, reps, stream):
    """Average duration of fn's launches with HIP events on the launch stream
    (the launches queued behind a device-side spin, so that they run back to
    back)."""
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    fn()  # first launch outside the timed region (one-time set-up)
    _fill_queue(stream)
    start.record(stream)
    for _ in range(reps):
        fn()
    end.record(stream)
    end.synchronize()
    return start.elapsed_time(end) / 1e3 / reps


def time_steps(fn, steps, warmup):
    """Wall-clock seconds per step over `steps` steps after `warmup` untimed
    ones, bracketed by device synchronisation."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        fn()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) / steps


def roofline(kernel, ops, nbytes, seconds, peak_gops, cbound, traffic=None):
    """Roofline of one kernel: the binding roof is the one whose ideal time
    (ops / compute peak, or bytes / HBM peak) is longer; frac = achieved /
    peak on that roof."""
    t_c = ops / (peak_gops * 1e9) if peak_gops else 0.0
    t_h = nbytes / (HBM_PEAK_GBS * 1e9)
    gops = ops / seconds / 1e9
    gbs = nbytes / seconds / 1e9
    if t_h >= t_c:
        r = {"bound": "hbm", "kernel": kernel, "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
             "frac": round(gbs / HBM_PEAK_GBS, 4),
             "compute": {"bound": cbound, "achieved_gops": round(gops, 1), "peak_gops": round(peak_gops or 0, 1),
                         "frac": round(gops / peak_gops, 4) if peak_gops else None}}
    else:
        r = {"bound": cbound, "kernel": kernel, "achieved": round(gops, 1), "peak": round(peak_gops, 1),
             "unit": "GOPS", "frac": round(gops / peak_gops, 4),
             "hbm": {"achieved_gbs": round(gbs, 1), "peak_gbs": HBM_PEAK_GBS, "frac": round(gbs / HBM_PEAK_GBS, 4)}}
    r.update({"traffic": traffic, "traffic_unit": "HBM bytes per launch", "algorithmic_bytes": int(nbytes),
              "algorithmic_ops": int(ops), "avg_us": round(seconds * 1e6, 2)})
    return r


def ideal_seconds(ops, nbytes, peak_gops):
    t_c = ops / (peak_gops * 1e9) if peak_gops else 0.0
    return max(t_c, nbytes / (HBM_PEAK_GBS * 1e9))


# ---------------------------------------------------------------------------
# CPU oracle baselines (bounded samples)
# ---------------------------------------------------------------------------

def _bn_np(case):
    return {key: (v.numpy() if hasattr(v, "numpy") else v) for key, v in case.bn.items()}


def cpu_baseline_conv(case, mode, budget_s=8.0):
    """The oracle (untuned) on a bounded sample of the same layer: quantize the
    sampled images + weights, direct conv, epilogue; GOPS over that sample."""
    import oracle

    n, c, h, w = case.x.shape
    cout, _, k, _ = case.w.shape
    ho = q.out_size(h, k, case.stride, case.pad)
    wo = q.out_size(w, k, case.stride, case.pad)
    macs_per_img = cout * ho * wo * c * k * k

    def run(m):
        t0 = time.perf_counter()
        if case.w_bits == 16:
            kk, bb = oracle.bn_fold(_bn_np(case))
            oracle.qconv16w_layer(oracle.quantize(case.x[:m].numpy(), case.a_bits), oracle.to_f16(case.w.numpy()),
                                  case.a_bits, case.stride, case.pad, "bn", k=kk, b=bb)
            return time.perf_counter() - t0
        if case.a_bits == 16:
            lw, _ = oracle.quantize_weights(case.w.numpy(), case.w_bits)
            kk, bb = oracle.bn_fold(_bn_np(case))
            oracle.qconv16_layer(oracle.to_f16(case.x[:m].numpy()), lw, case.w_bits, case.stride, case.pad, "bn",
                                 k=kk, b=bb)
            return time.perf_counter() - t0
        la = oracle.quantize(case.x[:m].numpy(), case.a_bits)
        lw, s = oracle.quantize_weights(case.w.numpy(), case.w_bits)
        acc = oracle.qconv_acc(la, lw, case.a_bits, case.stride, case.pad)
        shift = oracle.level_shift(case.a_bits) + oracle.level_shift(case.w_bits)
        if mode in (q.EPI_BN_F32, q.EPI_BN_PACK):
            kk, bb = oracle.bn_fold(_bn_np(case))
            z = oracle.epi_bn(acc, kk, bb, shift)
            if mode == q.EPI_BN_PACK:
                oracle.quantize(oracle.hardtanh(z), case.a_bits)
        elif mode == q.EPI_SCALE_F32:
            oracle.epi_scale(acc, s, shift)
        return time.perf_counter() - t0

    t1 = run(1)
    m = int(max(1, min(n, budget_s / max(t1, 1e-6))))
    tm = run(m) if m > 1 else t1
    return {"value": round(2.0 * macs_per_img * m / tm / 1e9, 3), "unit": "GOPS", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"{m} of {n} images of the same layer (quantize + direct conv + epilogue), {tm:.1f} s"}


def cpu_baseline_net(params, wl, budget_s=8.0):
    import oracle

    if wl == "convnet":
        forward = oracle.convnet_forward
    elif wl == "convnet_w16":
        def forward(p):
            return oracle.convnet16w_forward(p, 1)
    else:
        def forward(p):
            return oracle.resnet18_forward(p, 2, 2)
    n = params["x"].shape[0]

    def run(m):
        sub = dict(params)
        sub["x"] = params["x"][:m]
        t0 = time.perf_counter()
        forward(sub)
        return time.perf_counter() - t0

    t1 = run(1)
    m = int(max(1, min(n, budget_s / max(t1, 1e-6))))
    tm = run(m) if m > 1 else t1
    return {"value": round(m / tm, 3), "unit": "images/s", "cores": oracle.num_threads(), "kind": "oracle",
            "sample": f"{m} of {n} images through the whole network, {tm:.1f} s"}


# ---------------------------------------------------------------------------
# workloads
# ---------------------------------------------------------------------------

def conv_entry(case, mode, dev, stream, steps, warmup, algo, cpu, out_bits=0, cpu_budget=8.0):
    """One layer: step = pack + conv; roofline of the conv launch."""
    W = ConvWorkload(case, dev, mode, algo, out_bits)
    dt = time_steps(W.step, steps, warmup)
    t_conv = time_kernel(W.conv, steps, stream)
    t_pack = time_kernel(W.pack, steps, stream)
    n, c, h, w = W.shape
    peak, cbound = compute_peak(W.used, case.a_bits, case.w_bits)
    e = {"workload": case.name, "value": round(2.0 * W.macs / dt / 1e9, 1), "unit": "GOPS",
         "ms_per_step": round(dt * 1e3, 4),
         "dtype": "f16 x code -> f32" if 16 in (case.a_bits, case.w_bits) else ALGO_DTYPE[W.used],
         "config": {"batch": n, "cin": c, "hw": h, "cout": W.cout, "k": W.k, "stride": case.stride,
                    "a_bits": case.a_bits, "w_bits": case.w_bits, "algo": W.used,
                    "epilogue": {q.EPI_INT32: "int32", q.EPI_SCALE_F32: "scale_f32", q.EPI_BN_F32: "bn_f32",
                                 q.EPI_BN_PACK: f"bn_requantize_pack{out_bits}"}[mode],
                    "weights": "packed once before timing"},
         "roofline": roofline(W.kname, 2.0 * W.macs, W.conv_bytes(), t_conv, peak, cbound,
                              measured_traffic(case.name, W.kname)),
         "pack_act": {"avg_us": round(t_pack * 1e6, 2), "achieved_gbs": round(W.pack_bytes() / t_pack / 1e9, 1),
                      "peak_gbs": HBM_PEAK_GBS, "frac": round(W.pack_bytes() / t_pack / 1e9 / HBM_PEAK_GBS, 4)}}
    if cpu:
        e["cpu_baseline"] = cpu_baseline_conv(case, mode, cpu_budget)
    return e, W


def layer_work(net, li, batch, dev):
    """(ops, algorithmic bytes, compute peak GOPS, bound name, kernel name) of
    layer li of a qnet; the bytes of tensors a layer's epilogue writes for
    later (folded) layers count as its output."""
    L = net.layers[li]
    kind = L["kind"]
    ci, hi, wi, bi, _ = net.tensor_info(L["src"], batch)
    co, ho, wo, bo, _ = net.tensor_info(L["dst"], batch)
    n = batch
    bin_ = packed_bytes(n, ci, hi, wi, bi)
    bout = packed_bytes(n, co, ho, wo, bo)
    kname = net.layer_kernel(li, batch)
    extra = 0
    for key in ("pool_dst", "pack_dst"):
        if L.get(key):
            pc, ph, pw, pb, _ = net.tensor_info(L[key], batch)
            extra += packed_bytes(n, pc, ph, pw, pb)
    if L.get("pool_dst"):
        bout = 0  # the unpooled output is never written
    if kind == "conv_f32":
        k = L["k"]
        ops = 2.0 * n * co * ho * wo * ci * k * k
        if "bf16x6" in kname:
            return ops, bin_ + co * ci * k * k * 4 + bout + extra, BF16X6_PEAK_GOPS, "mfma_bf16x6", kname
        return ops, bin_ + co * ci * k * k * 4 + bout + extra, FP32_PEAK_GOPS, "fp32", kname
    if kind == "qconv":
        k, s, p = L["k"], L["stride"], L["pad"]
        hc, wc = q.out_size(hi, k, s, p), q.out_size(wi, k, s, p)
        ops = 2.0 * n * co * hc * wc * ci * k * k
        mode = q.EPI_BN_PACK if L["out_bits"] else q.EPI_BN_F32
        flags = (q.EPI_POOL2 if L["pool2"] else 0) | (q.EPI_RESIDUAL if L["residual_src"] > 0 else 0)
        ob = L["out_bits"]
        if L.get("pack_dst"):  # a folded quantize layer: the packed copy of the fp32 output
            ob = net.tensor_info(L["pack_dst"], batch)[3]
        used = q.ALGO_NAMES[q.resolve_algo(n, ci, hi, wi, co, k, s, p, bi, L["w_bits"], mode, flags, ob)]
        nb = bin_ + weight_operand_bytes(co, ci, k, used, L["w_bits"]) + bout + extra
        if L["residual_src"] > 0:
            nb += bout
        peak, cb = compute_peak(used, bi, L["w_bits"]) if L["w_bits"] != 16 else (MFMA_PEAK_GOPS["mfma_f16"], "mfma")
        return ops, nb, peak, cb, kname
    if kind == "fc_f32":
        fin = ci * hi * wi
        return 2.0 * n * fin * co, bin_ + fin * co * 4 + bout, FP32_PEAK_GOPS, "fp32", kname
    return 0.0, bin_ + bout, None, "hbm", kname


def net_entry(wl, dev, stream, steps, warmup, cpu, cpu_budget=8.0):
    """Whole forward (images/s) plus each layer against its own roofline."""
    from paper_2003_04296_amd.nets import build_convnet, build_resnet18

    f32_note = None
    if wl == "convnet":
        params = synth.convnet_params(seed=1003, batch=256)
        qn = build_convnet(params, dev)
        name, dtype = "convnet_1w1a_batch256_32x32", ALGO_DTYPE["mfma_fp4"]
    elif wl == "convnet_w16":
        params = synth.convnet_params(seed=1003, batch=256)
        qn = build_convnet(params, dev, a_bits=1, w_bits=16)
        name, dtype = "convnet_1a16w_batch256_32x32", "f16 x code -> f32"
    else:
        params = synth.resnet18_params(seed=1004, batch=64)
        qn = build_resnet18(params, dev)
        name, dtype = "resnet18_2w2a_batch64_224x224", ALGO_DTYPE["mfma_fp4"]
        f32_note = ("stem: fp32 conv as exact three-way bf16 splits, six bf16 x bf16 -> f32 products "
                    "per multiply-add (fp32 accuracy)")
    x = params["x"].to(dev)
    batch = x.shape[0]
    logits = torch.empty((batch, qn.out_features), dtype=torch.float32, device=dev)
    dt = time_steps(lambda: qn.forward(x, logits), steps, warmup)
    t_fwd = time_kernel(lambda: qn.forward(x, logits), steps, stream)
    ws = qn.workspace(batch)
    net = qn.net
    layers = []
    tot_ideal = 0.0
    for li in range(net.num_layers()):
        if net.layers[li].get("fused_into") is not None:
            layers.append({"layer": li, "kind": net.layers[li]["kind"], "fused_into": net.layers[li]["fused_into"],
                           "avg_us": 0.0, "ideal_us": 0.0, "ops": 0, "bytes": 0, "kernel": None, "_peak": None})
            continue
        t = time_kernel(lambda: net.forward_range(x, logits, ws, li, 1), max(5, steps // 2), stream)
        ops, nb, peak, cb, kname = layer_work(net, li, batch, dev)
        ideal = ideal_seconds(ops, nb, peak)
        tot_ideal += ideal
        layers.append({"layer": li, "kind": net.layers[li]["kind"], "kernel": kname, "avg_us": round(t * 1e6, 2),
                       "ideal_us": round(ideal * 1e6, 2), "frac": round(ideal / t, 4), "ops": int(ops),
                       "bytes": int(nb), "bound": cb if peak and ops / (peak * 1e9) >= nb / (HBM_PEAK_GBS * 1e9)
                       else "hbm", "traffic": measured_traffic(name, kname, li), "_peak": peak})
    dom = max(layers, key=lambda r: r["avg_us"])
    peak = dom.pop("_peak")
    for r in layers:
        r.pop("_peak", None)
    rf = roofline(dom["kernel"], dom["ops"], dom["bytes"], dom["avg_us"] / 1e6, peak,
                  dom["bound"] if dom["bound"] != "hbm" else ("fp32" if dom["kind"] == "conv_f32" else "mfma"),
                  measured_traffic(name, dom["kernel"], dom["layer"]))
    rf.update({"layer": dom["layer"],
               "network": {"ideal_us": round(tot_ideal * 1e6, 2), "forward_us": round(t_fwd * 1e6, 2),
                           "frac": round(tot_ideal / t_fwd, 4),
                           "note": "sum over layers of max(ops / compute peak, bytes / HBM peak) / forward time"}})
    e = {"workload": name, "value": round(batch / dt, 1), "unit": "images/s", "ms_per_step": round(dt * 1e3, 4),
         "dtype": dtype, "config": {"batch": batch, "weights": "packed once before timing"}, "roofline": rf,
         "layers": layers}
    if f32_note:
        e["config"]["f32_layers"] = f32_note
    if cpu:
        e["cpu_baseline"] = cpu_baseline_net(params, wl, cpu_budget)
    return e


def layers5_entry(dev, stream, steps, warmup, cpu, algo=q.ALGO_AUTO, cpu_budget=2.5):
    """The four 3W3A ResNet-18 3x3 layer shapes at batch 256 (int32 output,
    and the fused BN + requantize + pack epilogue beside it)."""
    parts, tot_ops, tot_step, tot_conv = [], 0.0, 0.0, 0.0
    cpu_gops = []
    for li in range(4):
        case = synth.workload5(li)
        e, W = conv_entry(case, q.EPI_INT32, dev, stream, steps, warmup, algo, cpu, cpu_budget=cpu_budget)
        tot_ops += 2.0 * W.macs
        tot_step += e["ms_per_step"] / 1e3
        tot_conv += e["roofline"]["avg_us"] / 1e6
        # the same layer with the fused {BN-HardTanh-quantize-pack} epilogue (3-bit output)
        g = synth.generator(1105 + li)
        case.bn = synth.bn_params(g, case.w.shape[0], float(case.w.shape[1] * 9 * 16))
        Wp = ConvWorkload(case, dev, q.EPI_BN_PACK, algo, 3)
        tp = time_kernel(Wp.conv, steps, stream)
        pk, pcb = compute_peak(Wp.used, 3, 3)
        e["packed_out"] = roofline(Wp.kname, 2.0 * Wp.macs, Wp.conv_bytes(), tp, pk, pcb)
        parts.append(e)
        del W, Wp
        if cpu:
            cpu_gops.append(e["cpu_baseline"])
    dom = max(parts, key=lambda r: r["roofline"]["avg_us"])
    out = {"workload": "resnet18_3x3_layers_3w3a_batch256", "value": round(tot_ops / tot_step / 1e9, 1),
           "unit": "GOPS", "ms_per_step": round(tot_step * 1e3, 4), "dtype": dom["dtype"],
           "conv_gops": round(tot_ops / tot_conv / 1e9, 1),
           "config": {"batch": 256, "layers": ["64@56x56", "128@28x28", "256@14x14", "512@7x7"],
                      "a_bits": 3, "w_bits": 3, "epilogue": "int32"},
           "roofline": dict(dom["roofline"], layer=dom["workload"]), "layers": parts}
    if cpu:
        ops_s = sum(float(c["value"]) for c in cpu_gops) / len(cpu_gops)
        out["cpu_baseline"] = {"value": round(ops_s, 3), "unit": "GOPS", "cores": cpu_gops[0]["cores"],
                               "kind": "oracle", "sample": "mean over the four layers of: " +
                               "; ".join(c["sample"] for c in cpu_gops)}
    return out


def aqe_entry(dev, stream, steps, warmup, cpu):
    # the elementwise AQE work of one training step of ResNet-18 2W2A at
    # batch 64: s_c of 11.2 M weights, their forward (per-channel thresholds)
    # and that of one 64 x 64 x 56 x 56 activation tensor, their AQE
    # gradients, and the SGD update + clip of the weights
    g = synth.generator(1006)
    wt = synth.normal(g, (2432, 512, 3, 3), 2.0 / 4608).to(dev)
    act = synth.normal(g, (64, 64, 56, 56), 1.0).to(dev)
    gact = synth.normal(g, (64, 64, 56, 56), 1e-3).to(dev)
    gw = synth.normal(g, (2432, 512, 3, 3), 1e-3).to(dev)
    wq, s_c = q.pack_weight(wt, 2)
    wh, ah, ga, gwx = torch.empty_like(wt), torch.empty_like(act), torch.empty_like(act), torch.empty_like(wt)
    nw, na = wt.numel(), act.numel()

    def aqe_step():
        q.pack_weight(wt, 2, out=(wq, s_c))
        q.aqe_forward(wt, 2, 0.5, scale=s_c, group_size=4608, out=wh)
        q.aqe_forward(act, 2, 0.5, out=ah)
        q.aqe_backward(act, gact, 0.5, out=ga)
        q.aqe_backward(wt, gw, 0.5, out=gwx)
        q.aqe_sgd_clip(wt, gwx, 1e-3)

    dt = time_steps(aqe_step, steps, warmup)
    step_bytes = 32 * nw + 20 * na  # reads + writes of the five elementwise passes
    t_bwd = time_kernel(lambda: q.aqe_backward(act, gact, 0.5, out=ga), steps, stream)
    gbs = step_bytes / dt / 1e9
    bwd_gbs = 12 * na / t_bwd / 1e9
    e = {"metric": "AQE training elementwise throughput", "value": round(gbs, 1), "unit": "GB/s",
         "ms_per_step": round(dt * 1e3, 4), "dtype": "f32",
         "config": {"workload": "aqe_resnet18_2w2a_batch64", "weights": nw, "activations": na,
                    "step": "s_c + weight packing, AQE forward of weights and activations, their backward, SGD + clip"},
         "roofline": {"bound": "hbm", "kernel": "aqe_backward_kernel<4>", "achieved": round(bwd_gbs, 1),
                      "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(bwd_gbs / HBM_PEAK_GBS, 4),
                      "traffic": None, "algorithmic_bytes": 12 * na, "avg_us": round(t_bwd * 1e6, 2),
                      "step_achieved_gbs": round(gbs, 1)}}
    if cpu:
        import oracle

        m = 1 << 22
        xs, gs = act.view(-1)[:m].cpu().numpy(), gact.view(-1)[:m].cpu().numpy()
        t0 = time.perf_counter()
        oracle.aqe_forward(xs, 2, 0.5)
        oracle.aqe_backward(xs, gs, 0.5)
        oracle.sgd_clip(xs, gs, 1e-3)
        tc = time.perf_counter() - t0
        e["cpu_baseline"] = {"value": round((8 + 12 + 12) * m / tc / 1e9, 2), "unit": "GB/s", "cores": 1,
                             "kind": "oracle",
                             "sample": f"forward + backward + update over {m} activations (numpy, one thread), "
                                       f"{tc:.2f} s"}
    return e


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="all")
    ap.add_argument("--algo", default="auto", choices=["auto", "bitplane", "mfma_i8", "mfma_fp4", "mfma_f16"])
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baselines")
    ap.add_argument("--copy-ref-mib", type=int, default=0,
                    help="after timing, run one device copy of this many MiB (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(images are independent, so the batch would shard across GPUs without communication)",
              file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    algo = {"auto": q.ALGO_AUTO, "bitplane": q.ALGO_BITPLANE, "mfma_i8": q.ALGO_MFMA_I8,
            "mfma_fp4": q.ALGO_MFMA_FP4, "mfma_f16": q.ALGO_MFMA_F16}[args.algo]
    wl = args.workload
    cpu = not args.no_cpu
    out = {"metric": METRIC, "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "data": "synthetic"}
    single = {"1w1a": (synth.workload1, q.EPI_SCALE_F32), "1w2a": (synth.workload2, q.EPI_BN_F32)}

    def headline(e):
        out.update({k: e[k] for k in ("value", "unit", "ms_per_step", "dtype", "roofline")})
        out["config"] = dict(workload=e["workload"], **e["config"])
        for k in ("cpu_baseline", "pack_act", "layers"):
            if k in e:
                out[k] = e[k]

    if wl == "all":
        configs = {}
        e1, W = conv_entry(synth.workload1(), q.EPI_SCALE_F32, dev, stream, args.steps, args.warmup, algo, cpu)
        configs["1"] = e1
        del W
        e2, W = conv_entry(synth.workload2(), q.EPI_BN_F32, dev, stream, args.steps, args.warmup, algo, cpu)
        configs["2"] = e2
        del W
        torch.cuda.empty_cache()
        configs["3"] = net_entry("convnet", dev, stream, args.steps, args.warmup, cpu)
        torch.cuda.empty_cache()
        configs["4"] = net_entry("resnet18", dev, stream, args.steps, args.warmup, cpu)
        torch.cuda.empty_cache()
        configs["5"] = layers5_entry(dev, stream, args.steps, args.warmup, cpu, algo)
        headline(e2)
        out["configs"] = configs
    elif wl in single:
        fn, mode = single[wl]
        e, _ = conv_entry(fn(), mode, dev, stream, args.steps, args.warmup, algo, cpu)
        headline(e)
    elif wl.startswith("a16") or (wl.endswith("w16") and wl[0] == "a"):
        case = synth.workload7(int(wl[-1])) if wl.startswith("a16") else synth.workload8(int(wl[1]))
        e, _ = conv_entry(case, q.EPI_BN_F32, dev, stream, args.steps, args.warmup, algo, cpu)
        headline(e)
    elif wl.startswith("3w3a-L"):
        e, _ = conv_entry(synth.workload5(int(wl.split("L")[1])), q.EPI_INT32, dev, stream, args.steps, args.warmup,
                          algo, cpu)
        headline(e)
    elif wl == "3w3a":
        headline(layers5_entry(dev, stream, args.steps, args.warmup, cpu, algo))
    elif wl in ("convnet", "convnet_w16", "resnet18"):
        headline(net_entry(wl, dev, stream, args.steps, args.warmup, cpu))
    elif wl == "aqe":
        e = aqe_entry(dev, stream, args.steps, args.warmup, cpu)
        out.update(e)
    else:
        print(f"unknown workload {wl}", file=sys.stderr)
        sys.exit(2)
    if args.copy_ref_mib:
        src = torch.empty(args.copy_ref_mib * (1 << 20) // 4, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        out["copy_ref_bytes"] = src.numel() * 4
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
