"""The 2-bit packed code layout (test infrastructure).

k-bit feature maps (Table 3, Table 4) stored at 2 bits per code: NHWC with
four codes per byte along C, channel c in bits 2*(c%4) .. 2*(c%4)+1 of byte
c // 4 (little-endian within the byte). C must be a multiple of 4.
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
