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
    cop = (cout + 127) // 128 * 128
    wd = np.asarray(words).view(np.uint32)[:kh * kw * cw * cop * P].reshape(kh, kw, cw, cop, P)
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


def weight_copies(words, cout, cin, kh, kw, bits):
    """Decode the int8 and fp4 operand copies that follow the bitplanes in a
    packed weight buffer -> two int8 level arrays [cout][cin][kh][kw]."""
    P = PLANES[bits]
    cw = (cin + 31) // 32
    cwp = (cw + 1) // 2
    cop = (cout + 127) // 128 * 128
    raw = np.asarray(words).view(np.uint8)
    off = kh * kw * cw * cop * P * 4
    i8 = raw[off:off + kh * kw * cw * cop * 32].view(np.int8).reshape(kh, kw, cw, cop, 32)
    off += kh * kw * cw * cop * 32
    f4 = raw[off:off + kh * kw * cwp * cop * 32].reshape(kh, kw, cwp, cop, 2, 4, 4)  # pair, word, u32 q, byte
    # levels from int8: channel cw*32 + c at byte c
    lv8 = np.moveaxis(i8, 2, 3).reshape(kh, kw, cop, cw * 32)[:, :, :cout, :cin]
    # fp4: u32 q of a word holds channels q, q + 4, ..., q + 28 in nibbles 0..7
    u32 = f4.copy().view(np.uint32).reshape(kh, kw, cwp, cop, 2, 4)
    nib = np.stack([(u32 >> (4 * k)) & 0xF for k in range(8)], axis=-1)  # ..., q, nibble k
    nib = np.swapaxes(nib, -1, -2)  # ..., k, q: channel 4k + q in row-major order
    mag = np.array([0, 0, 1, 0, 2, 0, 4, 0] * 2, np.int64)[nib]
    sgn = np.where(nib & 8, -1, 1)
    val = (mag * sgn).reshape(kh, kw, cwp, cop, 2 * 32)  # pair, 64 channels
    lv4 = np.moveaxis(val, 2, 3).reshape(kh, kw, cop, cwp * 64)[:, :, :cout, :cin]
    to_oihw = lambda a: np.ascontiguousarray(np.transpose(a, (2, 3, 0, 1))).astype(np.int8)
    return to_oihw(lv8), to_oihw(lv4)


def weight_copy_f16(words, cout, cin, kh, kw, bits) -> np.ndarray:
    """Decode the fp16 operand copy (the fourth part of a packed weight
    buffer, [kh][kw][2 cw][cout_pad][16 halves]) -> int8 levels [cout][cin][kh][kw]."""
    P = PLANES[bits]
    cw = (cin + 31) // 32
    cwp = (cw + 1) // 2
    cop = (cout + 127) // 128 * 128
    raw = np.asarray(words).view(np.uint8)
    off = kh * kw * cw * cop * (P * 4 + 32) + kh * kw * cwp * cop * 32
    h = raw[off:off + kh * kw * 2 * cw * cop * 32].view(np.float16).reshape(kh, kw, 2 * cw, cop, 16)
    lv = np.moveaxis(h, 2, 3).reshape(kh, kw, cop, 2 * cw * 16)[:, :, :cout, :cin].astype(np.float64)
    assert np.all(lv == np.round(lv))
    return np.ascontiguousarray(np.transpose(lv, (2, 3, 0, 1))).astype(np.int8)


def unpack_act16(words, n, c, h, w) -> np.ndarray:
    """fp16 [n][h][w][cw * 32] (int32 view) -> fp16 [n][c][h][w], and whether
    the padding channels are +0."""
    cw = (c + 31) // 32
    a = np.asarray(words).view(np.float16).reshape(n, h, w, cw * 32)
    pad_ok = bool(np.all(a[..., c:].view(np.uint16) == 0))
    return np.ascontiguousarray(np.transpose(a[..., :c], (0, 3, 1, 2))), pad_ok
