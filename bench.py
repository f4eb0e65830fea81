#!/usr/bin/env python3
"""Throughput of the quantized-convolution hot path on one MI355X.

Default workload: the 1-bit-weight / 2-bit-activation 3x3 convolution over a
batch of 256 x 128 x 32 x 32 fp32 activations with 128 output channels and a
fused fp32 batch-norm epilogue.  One step = quantize + pack the fp32 input
(qconv_pack_act) + the bitplane convolution with its epilogue
(qconv_forward); weights are packed once beforehand, as at inference.

Prints ONE JSON line: GOPS = 2 * MACs (all taps, padding included) / step
time, plus the roofline of the dominant kernel (measured with HIP events on
the launch stream) and the CPU oracle timed on a bounded sample.

Other workloads: --workload 1w1a | 1w2a (default) | 3w3a-L{0..3} |
a16w{1,2,3} (fp16 inputs, same layer shape; the step converts fp32 -> fp16) |
a{1,2,3}w16 (quantized inputs with fp16 weights, same layer shape) |
convnet_w16 (ConvNet with 1-bit activations and fp16 weights) |
aqe | convnet | resnet18 (the last two report images/s).
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
# dense matrix-core peaks (ops = 2 per MAC), in G: int8 5.0 POP/s, fp4 10.1 PFLOP/s, fp16 2.5 PFLOP/s
MFMA_PEAK_GOPS = {"mfma_i8": 5.0e6, "mfma_fp4": 10.1e6, "mfma_f16": 2.5e6}
# Minimal VALU recipe (lane-ops per 32-channel word pair) of the bitplane
# product on gfx950, where v_bitop3_b32 fuses any 3-input bit function:
#   1W1A: xor, bcnt                         -> 2
#   1W2A / 2W1A: bitop3(xor & mask), bcnt   -> 2  (activation-only popcount amortised)
#   2W2A: bitop3, and, and, 2 bcnt          -> 5
#   3W3A: 9 and/and_or (shift classes), 5 x (bitop3 + 2 bcnt) -> 24
LANE_OPS_PER_WORD = {(1, 1): 2, (2, 1): 2, (1, 2): 2, (2, 2): 5, (3, 3): 24}


def valu_peak_gops(a_bits, w_bits):
    ops = LANE_OPS_PER_WORD.get((a_bits, w_bits))
    if ops is None:
        return None
    return VALU_LANE_OPS * 32.0 / ops * 2.0 / 1e9  # conv-ops (2 per MAC) per second, in G


def _fold(bn, dev):
    k, b = q.fold_bn(bn["gamma"].numpy(), bn["beta"].numpy(), bn["mean"].numpy(), bn["var"].numpy(), bn["eps"])
    return torch.from_numpy(k).to(dev), torch.from_numpy(b).to(dev)


class ConvWorkload:
    """pack_act + qconv_forward on one synthetic layer."""

    def __init__(self, case, dev, mode, algo):
        self.case = case
        self.dev = dev
        self.mode = mode
        self.algo = algo
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
        dt = torch.int32 if mode == q.EPI_INT32 else torch.float32
        self.out = torch.empty(self.out_shape, dtype=dt, device=dev)
        self.macs = n * self.cout * ho * wo * c * self.k * self.k

    def pack(self):
        q.pack_act(self.x, self.case.a_bits, out=self.act)

    def conv(self):
        n, c, h, w = self.shape
        q.conv(self.act, self.wq, n, c, h, w, self.cout, self.k, self.case.stride, self.case.pad,
               self.case.a_bits, self.case.w_bits, mode=self.mode, scale=self.scale, bn_k=self.bn_k,
               bn_b=self.bn_b, out=self.out, algo=self.algo)

    def step(self):
        self.pack()
        self.conv()

    def conv_bytes(self, used):
        """Algorithmic HBM bytes of one conv launch: packed (or fp16) input + the
        part of the packed weights the algorithm reads + output."""
        n, c, h, w = self.shape
        a = q.packed_act_words(n, c, h, w, self.case.a_bits) * 4
        taps, cw, cop = self.k * self.k, (c + 31) // 32, (self.cout + 127) // 128 * 128
        if used == "bitplane":
            wb = taps * cw * cop * q.planes(self.case.w_bits) * 4
        else:
            wb = {"mfma_i8": taps * cw * cop * 32, "mfma_fp4": taps * ((cw + 1) // 2) * cop * 32,
                  "mfma_f16": taps * 2 * cw * cop * 32}[used]
        return a + wb + int(np.prod(self.out_shape)) * 4

    def pack_bytes(self):
        n, c, h, w = self.shape
        return n * c * h * w * 4 + q.packed_act_words(n, c, h, w, self.case.a_bits) * 4


def measured_traffic(workload: str, kernel: str):
    """HBM bytes per launch of `kernel` on `workload` from the
    committed rocprofv3 counter runs, or None when there is no record or the
    kernel's sources changed since the counters were taken."""
    import hashlib

    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path)).get(workload)
    if not rec or rec["kernel"] != kernel:
        return None
    h = hashlib.sha256()
    for src in rec["sources"]:
        h.update(open(os.path.join(ROOT, src), "rb").read())
    if h.hexdigest() != rec["sources_sha256"]:
        return None
    return rec["fetch_bytes"] + rec["write_bytes"]


def time_kernel(fn, reps, stream):
    """Average duration of fn's launches with HIP events on the launch stream."""
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(reps):
        fn()
    end.record(stream)
    end.synchronize()
    return start.elapsed_time(end) / 1e3 / reps


def cpu_baseline_conv(case, mode, budget_s=12.0):
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
            kk, bb = oracle.bn_fold({key: (v.numpy() if hasattr(v, "numpy") else v) for key, v in case.bn.items()})
            oracle.qconv16w_layer(oracle.quantize(case.x[:m].numpy(), case.a_bits), oracle.to_f16(case.w.numpy()),
                                  case.a_bits, case.stride, case.pad, "bn", k=kk, b=bb)
            return time.perf_counter() - t0
        if case.a_bits == 16:
            lw, _ = oracle.quantize_weights(case.w.numpy(), case.w_bits)
            kk, bb = oracle.bn_fold({key: (v.numpy() if hasattr(v, "numpy") else v) for key, v in case.bn.items()})
            oracle.qconv16_layer(oracle.to_f16(case.x[:m].numpy()), lw, case.w_bits, case.stride, case.pad, "bn",
                                 k=kk, b=bb)
            return time.perf_counter() - t0
        la = oracle.quantize(case.x[:m].numpy(), case.a_bits)
        lw, s = oracle.quantize_weights(case.w.numpy(), case.w_bits)
        acc = oracle.qconv_acc(la, lw, case.a_bits, case.stride, case.pad)
        if mode == q.EPI_BN_F32:
            kk, bb = oracle.bn_fold({key: (v.numpy() if hasattr(v, "numpy") else v) for key, v in case.bn.items()})
            oracle.epi_bn(acc, kk, bb, oracle.level_shift(case.a_bits) + oracle.level_shift(case.w_bits))
        elif mode == q.EPI_SCALE_F32:
            oracle.epi_scale(acc, s)
        return time.perf_counter() - t0

    t1 = run(1)
    m = int(max(1, min(n, budget_s / max(t1, 1e-6))))
    tm = run(m) if m > 1 else t1
    return {"value": round(2.0 * macs_per_img * m / tm / 1e9, 3), "unit": "GOPS", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"{m} of {n} images of the same layer (quantize + direct conv + epilogue), {tm:.1f} s"}


def cpu_baseline_net(params, wl, budget_s=12.0):
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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="1w2a")
    ap.add_argument("--algo", default="auto", choices=["auto", "bitplane", "mfma_i8", "mfma_fp4", "mfma_f16"])
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
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
    out = {"metric": METRIC, "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "data": "synthetic"}

    if wl in ("1w1a", "1w2a", "a16w1", "a16w2", "a16w3", "a1w16", "a2w16", "a3w16") or wl.startswith("3w3a"):
        if wl == "1w1a":
            case, mode = synth.workload1(), q.EPI_SCALE_F32
        elif wl == "1w2a":
            case, mode = synth.workload2(), q.EPI_BN_F32
        elif wl.startswith("a16"):
            case, mode = synth.workload7(int(wl[-1])), q.EPI_BN_F32
        elif wl.endswith("w16"):
            case, mode = synth.workload8(int(wl[1])), q.EPI_BN_F32
        else:
            case, mode = synth.workload5(int(wl.split("L")[1])), q.EPI_INT32
        W = ConvWorkload(case, dev, mode, algo)
        for _ in range(args.warmup):
            W.step()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            W.step()
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / args.steps
        t_conv = time_kernel(W.conv, args.steps, stream)
        t_pack = time_kernel(W.pack, args.steps, stream)
        gops_step = 2.0 * W.macs / dt / 1e9
        gops_conv = 2.0 * W.macs / t_conv / 1e9
        n, c, h, w = W.shape
        used = q.ALGO_NAMES[q.resolve_algo(n, c, h, w, W.cout, W.k, case.stride, case.pad, case.a_bits,
                                           case.w_bits, mode, 0, 0, algo)]
        # the instantiation the library launches for this layer (as the profiler names it)
        kname = q.kernel_name(n, c, h, w, W.cout, W.k, case.stride, case.pad, case.a_bits, case.w_bits,
                              mode=mode, algo=algo)
        if used == "bitplane":
            peak, cbound = valu_peak_gops(case.a_bits, case.w_bits), "alu"
        else:
            peak, cbound = MFMA_PEAK_GOPS[used], "mfma"
        hbm_gbs = W.conv_bytes(used) / t_conv / 1e9
        frac_c = gops_conv / peak if peak else 0.0
        frac_h = hbm_gbs / HBM_PEAK_GBS
        n, c, h, w = W.shape
        out.update({
            "value": round(gops_step, 1), "unit": "GOPS", "ms_per_step": round(dt * 1e3, 4),
            "dtype": "f16" if 16 in (case.a_bits, case.w_bits) else "int32",
            "config": {"workload": case.name, "batch": n, "cin": c, "hw": h, "cout": W.cout, "k": W.k,
                       "a_bits": case.a_bits, "w_bits": case.w_bits,
                       "epilogue": {q.EPI_INT32: "int32", q.EPI_SCALE_F32: "scale_f32",
                                    q.EPI_BN_F32: "bn_f32"}[mode],
                       "algo": used, "weights": "packed once before timing"},
            "roofline": ({"bound": "hbm", "kernel": kname, "achieved": round(hbm_gbs, 1), "peak": HBM_PEAK_GBS,
                          "unit": "GB/s", "frac": round(frac_h, 4),
                          "compute": {"bound": cbound, "achieved_gops": round(gops_conv, 1),
                                      "peak_gops": round(peak, 1), "frac": round(frac_c, 4)}}
                         if frac_h > frac_c else
                         {"bound": cbound, "kernel": kname, "achieved": round(gops_conv, 1),
                          "peak": round(peak, 1), "unit": "GOPS", "frac": round(frac_c, 4),
                          "hbm": {"achieved_gbs": round(hbm_gbs, 1), "peak_gbs": HBM_PEAK_GBS,
                                  "frac": round(frac_h, 4)}}),
        })
        out["roofline"].update({
            "traffic": measured_traffic(case.name, kname), "traffic_unit": "HBM bytes per launch",
            "algorithmic_bytes": W.conv_bytes(used), "avg_us": round(t_conv * 1e6, 2)})
        out.update({
            "pack_act": {"avg_us": round(t_pack * 1e6, 2), "achieved_gbs": round(W.pack_bytes() / t_pack / 1e9, 1),
                         "peak_gbs": HBM_PEAK_GBS},
        })
        if not args.no_cpu:
            out["cpu_baseline"] = cpu_baseline_conv(case, mode)
    elif wl == "aqe":
        # the elementwise AQE work of one training step of ResNet-18 2W2A at
        # batch 64: forward of 11.2 M weights (per-channel thresholds) and of
        # one 64 x 64 x 56 x 56 activation tensor, their AQE gradients, and the
        # SGD update + clip of the weights
        g = synth.generator(1006)
        wt = synth.normal(g, (2432, 512, 3, 3), 2.0 / 4608).to(dev)
        act = synth.normal(g, (64, 64, 56, 56), 1.0).to(dev)
        gact = synth.normal(g, (64, 64, 56, 56), 1e-3).to(dev)
        gw = synth.normal(g, (2432, 512, 3, 3), 1e-3).to(dev)
        _, s_c = q.pack_weight(wt, 2)
        wh, ah, ga, gwx = torch.empty_like(wt), torch.empty_like(act), torch.empty_like(act), torch.empty_like(wt)
        nw, na = wt.numel(), act.numel()

        def aqe_step():
            q.aqe_forward(wt, 2, 0.5, scale=s_c, group_size=4608, out=wh)
            q.aqe_forward(act, 2, 0.5, out=ah)
            q.aqe_backward(act, gact, 0.5, out=ga)
            q.aqe_backward(wt, gw, 0.5, out=gwx)
            q.aqe_sgd_clip(wt, gwx, 1e-3)

        for _ in range(args.warmup):
            aqe_step()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            aqe_step()
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / args.steps
        step_bytes = 32 * nw + 20 * na  # reads + writes of the five passes
        t_bwd = time_kernel(lambda: q.aqe_backward(act, gact, 0.5, out=ga), args.steps, stream)
        gbs = step_bytes / dt / 1e9
        bwd_gbs = 12 * na / t_bwd / 1e9
        out.update({"metric": "AQE training elementwise throughput", "value": round(gbs, 1), "unit": "GB/s",
                    "ms_per_step": round(dt * 1e3, 4), "dtype": "f32",
                    "config": {"workload": "aqe_resnet18_2w2a_batch64", "weights": nw, "activations": na},
                    "roofline": {"bound": "hbm", "kernel": "aqe_backward_kernel<4>", "achieved": round(bwd_gbs, 1),
                                 "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(bwd_gbs / HBM_PEAK_GBS, 4),
                                 "traffic": None, "algorithmic_bytes": 12 * na, "avg_us": round(t_bwd * 1e6, 2),
                                 "step_achieved_gbs": round(gbs, 1)}})
        if not args.no_cpu:
            import oracle

            m = 1 << 22
            xs, gs = act.view(-1)[:m].cpu().numpy(), gact.view(-1)[:m].cpu().numpy()
            t0 = time.perf_counter()
            oracle.aqe_forward(xs, 2, 0.5)
            oracle.aqe_backward(xs, gs, 0.5)
            oracle.sgd_clip(xs, gs, 1e-3)
            tc = time.perf_counter() - t0
            out["cpu_baseline"] = {"value": round((8 + 12 + 12) * m / tc / 1e9, 2), "unit": "GB/s", "cores": 1,
                                   "kind": "oracle",
                                   "sample": f"forward + backward + update over {m} activations (numpy, one thread), "
                                             f"{tc:.2f} s"}
    elif wl in ("convnet", "convnet_w16", "resnet18"):
        from paper_2003_04296_amd.nets import build_convnet, build_resnet18

        if wl == "convnet":
            params = synth.convnet_params(seed=1003, batch=256)
            net = build_convnet(params, dev)
        elif wl == "convnet_w16":
            params = synth.convnet_params(seed=1003, batch=256)
            net = build_convnet(params, dev, a_bits=1, w_bits=16)
        else:
            params = synth.resnet18_params(seed=1004, batch=64)
            net = build_resnet18(params, dev)
        x = params["x"].to(dev)
        logits = torch.empty((x.shape[0], net.out_features), dtype=torch.float32, device=dev)
        for _ in range(args.warmup):
            net.forward(x, logits)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            net.forward(x, logits)
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / args.steps
        out.update({"value": round(x.shape[0] / dt, 1), "unit": "images/s", "ms_per_step": round(dt * 1e3, 4),
                    "dtype": "f16" if wl == "convnet_w16" else "int32", "roofline": None,
                    "config": {"workload": wl + {"convnet": "_1w1a_batch256_32x32", "convnet_w16": "_1a16w_batch256_32x32",
                                                 "resnet18": "_2w2a_batch64_224x224"}[wl],
                               "batch": int(x.shape[0])}})
        if not args.no_cpu:
            out["cpu_baseline"] = cpu_baseline_net(params, wl)
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
