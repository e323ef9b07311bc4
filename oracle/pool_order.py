"""Max-pooling in the paper's order, before BN and the quantizer (Eq. 4 on
the conv output, Sec. 2.1), against pooling the codes. Test infrastructure,
host only.

With the folded thresholds of Eq. 7-8 a channel's code is a monotone function
of its integer sum: non-decreasing where the sign s is +1, non-increasing
where s is -1 (negative BN scale). Pooling the sums with max where s = +1 and
min where s = -1 and thresholding once therefore gives exactly the max of the
codes, the order the library computes in (its fused conv + pool takes the max
over the codes of each window). Taking the max of the float conv output for
every channel, as the paper's order reads literally, gives the same codes
where the BN scale is positive and can differ where it is negative, since BN
then reverses the order of the values.

Windows are those of the library's pool: "valid" (every window inside the
input) or "same" (ho = ceil(h / stride), windows clipped at the bottom and
right edges, only in-bounds elements taken).
"""
import numpy as np

from . import core
from . import float_chain


def _out_hw(h, w, k, stride, mode):
    if mode == "valid":
        return (h - k) // stride + 1, (w - k) // stride + 1
    return -(-h // stride), -(-w // stride)


def pool_values(v, k, stride, mode, reduce_max):
    """Window max (reduce_max True) or min of v [n][h][w][c], elementwise per
    channel: reduce_max is a bool or a per-channel bool array."""
    n, h, w, c = v.shape
    ho, wo = _out_hw(h, w, k, stride, mode)
    reduce_max = np.broadcast_to(np.asarray(reduce_max, dtype=bool), (c,))
    out = np.empty((n, ho, wo, c), dtype=v.dtype)
    for oy in range(ho):
        y0, y1 = oy * stride, min(oy * stride + k, h)
        for ox in range(wo):
            x0, x1 = ox * stride, min(ox * stride + k, w)
            win = v[:, y0:y1, x0:x1, :]
            out[:, oy, ox, :] = np.where(reduce_max, win.max(axis=(1, 2)), win.min(axis=(1, 2)))
    return out


def pooled_sums_then_codes(acc, s, t, k, stride, mode):
    """The paper's order on the integer path: pool the sums (max where
    s = +1, min where s = -1), then the thresholds of Eq. 7-8 once."""
    pooled = pool_values(acc, k, stride, mode, np.asarray(s) > 0)
    return core.codes(pooled, s, t)


def float_max_then_quantize(x, p, stride, pad, k, pool_stride, mode):
    """The paper's order read literally on the float chain: the max of the
    conv output Y over each window for every channel, then BN and the
    quantizer (Eq. 2-3). Returns (codes, margin) as float_chain.quantize."""
    y = float_chain.conv(x, p["beta_in"], p["w"], p["alpha"], p["bias"], stride, pad)
    ym = pool_values(y, k, pool_stride, mode, True)
    ybn = float_chain.bn(ym, p["mean"], p["var"], p["gamma"], p["bn_beta"], p["eps"])
    return float_chain.quantize(ybn, p["q_thr"])
