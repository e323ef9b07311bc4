"""Compact thresholds of a uniform quantizer (Sec. 3.2, Eq. 8). Test
infrastructure, host only.

For thresholds q_i = i*base + offset (i = 1 .. 2^k - 1), moving the quantizer
through BN and the conv scale (Eq. 6-8) keeps them uniform: t_i = i*base' +
offset' with

  base'   = base * sd / gamma / (alpha * beta_in)
  offset' = (mean - bias + (offset - bn_beta) * sd / gamma) / (alpha * beta_in)

(sd = sqrt(var + eps)). Two numbers per channel then stand for all 2^k - 1
thresholds; the integer thresholds are T_i = floor(s * t_i) with s the sign of
gamma, taken for each i (the floor is not affine in i), clamped to the sum
bound [-B-1, B]. gamma = 0 makes the code a constant, #{i : bn_beta > q_i}.
Arithmetic in float64, each operation rounded on its own, in the order written
in fold_compact and expand.
"""
import numpy as np


def fold_compact(p, base, offset, out_bits):
    """Per-channel (base', offset', s, cstar) of one layer's parameters p."""
    alpha = np.asarray(p["alpha"], np.float64)
    c = alpha.shape[0]
    full = lambda key, default: np.broadcast_to(
        np.asarray(p.get(key, default) if p.get(key) is not None else default, np.float64), (c,))
    bias, mean = full("bias", 0.0), full("mean", 0.0)
    var, gamma, bn_beta = full("var", 1.0), full("gamma", 1.0), full("bn_beta", 0.0)
    sd = np.sqrt(var + float(p["eps"]))
    ab = alpha * float(p["beta_in"])
    g = np.where(gamma == 0.0, 1.0, gamma)
    b = base * sd
    b = b / g
    basep = b / ab
    o = offset - bn_beta
    o = o * sd
    o = o / g
    o = o + mean
    o = o - bias
    offp = o / ab
    s = np.sign(gamma).astype(np.int32)
    nq = (1 << out_bits) - 1
    q = np.array([np.float64(i) * base + offset for i in range(1, nq + 1)])
    cstar = (bn_beta[:, None] > q[None, :]).sum(axis=1).astype(np.int32)
    zero = gamma == 0.0
    return {"base": np.where(zero, 0.0, basep), "offset": np.where(zero, 0.0, offp),
            "s": s, "cstar": np.where(zero, cstar, 0).astype(np.int32)}


def expand(rec, out_bits, bound):
    """(s, T) in the form oracle.codes takes: s [c] int32, T [c][2^k - 1]."""
    nq = (1 << out_bits) - 1
    i = np.arange(1, nq + 1, dtype=np.float64)
    t = i[None, :] * rec["base"][:, None]
    t = t + rec["offset"][:, None]
    sign = np.where(rec["s"] < 0, -1.0, 1.0)[:, None]
    f = np.clip(np.floor(sign * t), -bound - 1.0, bound)
    const = rec["s"] == 0
    fconst = np.where(np.arange(1, nq + 1)[None, :] <= rec["cstar"][:, None], -bound - 1.0, bound)
    T = np.where(const[:, None], fconst, f).astype(np.int32)
    s = np.where(const, 1, rec["s"]).astype(np.int32)
    return s, T
