"""The 2-bit code layouts (test infrastructure).

k-bit feature maps (Table 3, Table 4) stored at 2 bits per code:
  pack2         NHWC with four codes per byte along C, channel c in bits
                2*(c%4) .. 2*(c%4)+1 of byte c // 4 (little-endian within the
                byte); C a multiple of 4
  pack_block64  the same bytes regrouped into channel blocks of 64:
                [n][c/64][h][w][16 bytes]; C a multiple of 64
"""
import numpy as np


def tensor_bits(shape, bits):
    n = 1
    for d in shape:
        n *= int(d)
    return n * bits


def pack2(codes):
    codes = np.asarray(codes, dtype=np.uint8)
    c = codes.shape[-1]
    if c % 4:
        raise ValueError("C must be a multiple of 4")
    if codes.size and codes.max() > 3:
        raise ValueError("codes must be < 4")
    g = codes.reshape(codes.shape[:-1] + (c // 4, 4)).astype(np.uint8)
    out = np.zeros(g.shape[:-1], dtype=np.uint8)
    for j in range(4):
        out |= (g[..., j] << (2 * j)).astype(np.uint8)
    return out


def unpack2(packed, c):
    packed = np.asarray(packed, dtype=np.uint8)
    assert packed.shape[-1] * 4 == c
    out = np.empty(packed.shape[:-1] + (packed.shape[-1], 4), dtype=np.uint8)
    for j in range(4):
        out[..., j] = (packed >> (2 * j)) & 3
    return out.reshape(packed.shape[:-1] + (c,))


def pack_block64(codes):
    """NHWC codes (n, h, w, c) -> uint8 (n, c/64, h, w, 16)."""
    p = pack2(codes)
    n, h, w, cb = p.shape
    if cb % 16:
        raise ValueError("C must be a multiple of 64")
    return np.ascontiguousarray(p.reshape(n, h, w, cb // 16, 16).transpose(0, 3, 1, 2, 4))


def unpack_block64(packed, c):
    """uint8 (n, c/64, h, w, 16) -> NHWC codes (n, h, w, c)."""
    packed = np.asarray(packed, dtype=np.uint8)
    n, g, h, w, _ = packed.shape
    assert g * 64 == c
    return unpack2(packed.transpose(0, 2, 3, 1, 4).reshape(n, h, w, g * 16), c)
