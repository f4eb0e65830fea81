"""Pins for the oracle's network composition (layer order, pool placement,
flatten order, residual wiring) -- CPU only, at reduced widths.

The reference here is built from torch library ops that are exact on the
integer level tensors (float64 conv2d, max_pool2d) plus the oracle's
separately pinned rounding steps, so a wiring mistake in the oracle's
networks (a missing pool, a transposed flatten, a wrong shortcut) fails."""
import numpy as np
import torch
import torch.nn.functional as F

from paper_2003_04296_amd import synth


def _t(a):
    return torch.from_numpy(np.asarray(a, dtype=np.float64))


def _fold(oracle_mod, bn):
    return oracle_mod.bn_fold({k: (v.numpy() if hasattr(v, "numpy") else v) for k, v in bn.items()})


def test_convnet_wiring(oracle_mod):
    p = synth.convnet_params(seed=77, batch=2, width=1 / 16, fc_width=1 / 32)
    logits, levels = oracle_mod.convnet_forward(p, return_levels=True)
    x = p["x"].numpy()
    c0 = p["convs"][0]
    k, b = _fold(oracle_mod, c0["bn"])
    a = oracle_mod.quantize(oracle_mod.bn_f32(oracle_mod.conv_f32(x, c0["w"].numpy(), 1, 1), k, b), 1)
    np.testing.assert_array_equal(levels[0], a)
    for i, layer in enumerate(p["convs"][1:], start=1):
        wq = np.where(layer["w"].numpy() > 0, 1, -1)
        acc = F.conv2d(F.pad(_t(a), (1, 1, 1, 1), value=-1.0), _t(wq))
        if p["pools"][i]:
            acc = F.max_pool2d(acc, 2)
        k, b = _fold(oracle_mod, layer["bn"])
        a = oracle_mod.quantize(oracle_mod.epi_bn(acc.numpy().astype(np.int32), k, b), 1)
        np.testing.assert_array_equal(levels[i], a, err_msg=f"conv{i + 1}")
    assert a.shape[2] == a.shape[3] == 4
    flat = a.reshape(a.shape[0], -1)  # (c, h, w) order, as torch.flatten
    for j, fc in enumerate(p["fcs"]):
        wq = np.where(fc["w"].numpy() > 0, 1, -1)
        acc = (_t(flat) @ _t(wq).T).numpy().astype(np.int32)
        k, b = _fold(oracle_mod, fc["bn"])
        flat = oracle_mod.quantize(oracle_mod.epi_bn(acc[:, :, None, None], k, b)[:, :, 0, 0], 1)
        np.testing.assert_array_equal(levels[len(p["convs"]) + j], flat)
    ref = _t(flat) @ _t(p["fc_out"]["w"].numpy()).T + _t(p["fc_out"]["b"].numpy())
    np.testing.assert_allclose(logits, ref.numpy(), rtol=1e-5, atol=1e-5)


def test_resnet18_wiring(oracle_mod):
    p = synth.resnet18_params(seed=78, batch=1, hw=64, classes=12, width=1 / 8)
    logits, acts = oracle_mod.resnet18_forward(p, 2, 2, return_acts=True)
    st = p["stem"]
    k, b = _fold(oracle_mod, st["bn"])
    z = oracle_mod.bn_f32(oracle_mod.conv_f32(p["x"].numpy(), st["w"].numpy(), 2, 3), k, b)
    x = F.max_pool2d(_t(np.maximum(z, 0)), 3, 2, 1).numpy().astype(np.float32)
    np.testing.assert_array_equal(acts[0], x)
    for i, blk in enumerate(p["blocks"]):
        s = blk["stride"]
        q = oracle_mod.quantize(x, 2)
        w1, _ = oracle_mod.quantize_weights(blk["w1"].numpy(), 2)
        w2, _ = oracle_mod.quantize_weights(blk["w2"].numpy(), 2)
        acc1 = F.conv2d(_t(q), _t(w1), stride=s, padding=1).numpy().astype(np.int32)
        k1, b1 = _fold(oracle_mod, blk["bn1"])
        y = oracle_mod.quantize(oracle_mod.epi_bn(acc1, k1, b1), 2)
        acc2 = F.conv2d(_t(y), _t(w2), padding=1).numpy().astype(np.int32)
        k2, b2 = _fold(oracle_mod, blk["bn2"])
        zz = oracle_mod.epi_bn(acc2, k2, b2)
        if "wd" in blk:
            wd, _ = oracle_mod.quantize_weights(blk["wd"].numpy(), 2)
            accd = F.conv2d(_t(q), _t(wd), stride=s).numpy().astype(np.int32)
            kd, bd = _fold(oracle_mod, blk["bnd"])
            sc = oracle_mod.epi_bn(accd, kd, bd)
        else:
            sc = x
        x = (zz + sc).astype(np.float32)
        np.testing.assert_array_equal(acts[i + 1], x, err_msg=f"block {i}")
    assert len(p["blocks"]) == 8
    feat = _t(x).mean(dim=(2, 3))
    ref = feat @ _t(p["fc"]["w"].numpy()).T
    np.testing.assert_allclose(logits, ref.numpy(), rtol=1e-4, atol=1e-5)
