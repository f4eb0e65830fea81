"""Test-side helpers: decode packed bitplanes back to integer level codes
(the layout documented in include/qconv.h) and small utilities.  Shared by
the GPU parity tests only; neither the oracle nor the library uses them."""
import numpy as np

PLANES = {1: 1, 2: 2, 3: 4}


def unpack_act(words, n, c, h, w, bits) -> np.ndarray:
    """[n][h][w][cw][P] uint32 words -> int8 levels [n][c][h][w]."""
    P = PLANES[bits]
    cw = (c + 31) // 32
    wd = np.asarray(words).view(np.uint32).reshape(n, h, w, cw, P)
    bitidx = np.arange(32, dtype=np.uint32)
    bitsarr = ((wd[..., None] >> bitidx) & 1).astype(np.int8)  # n,h,w,cw,P,32
    bitsarr = np.moveaxis(bitsarr, 4, 3).reshape(n, h, w, P, cw * 32)[..., :c]  # n,h,w,P,c
    s = bitsarr[:, :, :, 0]
    if bits == 1:
        lv = 2 * s - 1
    elif bits == 2:
        lv = np.where(bitsarr[:, :, :, 1] == 1, 2 * s - 1, 0)
    else:
        mag = 4 * bitsarr[:, :, :, 1] + 2 * bitsarr[:, :, :, 2] + 1 * bitsarr[:, :, :, 3]
        lv = np.where(mag > 0, (2 * s - 1) * mag, 0)
    return np.ascontiguousarray(np.transpose(lv, (0, 3, 1, 2))).astype(np.int8)


def unpack_weight(words, cout, cin, kh, kw, bits) -> np.ndarray:
    """[kh][kw][cw][cout_pad][P] -> int8 levels [cout][cin][kh][kw]."""
    P = PLANES[bits]
    cw = (cin + 31) // 32
    cop = (cout + 63) // 64 * 64
    wd = np.asarray(words).view(np.uint32).reshape(kh, kw, cw, cop, P)
    bitidx = np.arange(32, dtype=np.uint32)
    b = ((wd[..., None] >> bitidx) & 1).astype(np.int8)  # kh,kw,cw,cop,P,32
    b = np.moveaxis(b, 2, 4)  # kh,kw,cop,P,cw,32
    b = b.reshape(kh, kw, cop, P, cw * 32)[:, :, :cout, :, :cin]  # kh,kw,cout,P,cin
    s = b[:, :, :, 0]
    if bits == 1:
        lv = 2 * s - 1
    elif bits == 2:
        lv = np.where(b[:, :, :, 1] == 1, 2 * s - 1, 0)
    else:
        mag = 4 * b[:, :, :, 1] + 2 * b[:, :, :, 2] + b[:, :, :, 3]
        lv = np.where(mag > 0, (2 * s - 1) * mag, 0)
    return np.ascontiguousarray(np.transpose(lv, (2, 3, 0, 1))).astype(np.int8)  # cout,cin,kh,kw


def tail_bits_zero(words, c, bits) -> bool:
    P = PLANES[bits]
    cw = (c + 31) // 32
    if c % 32 == 0:
        return True
    wd = np.asarray(words).view(np.uint32).reshape(-1, cw, P)
    mask = np.uint32((0xFFFFFFFF << (c % 32)) & 0xFFFFFFFF)
    return bool(np.all((wd[:, cw - 1, :] & mask) == 0))
