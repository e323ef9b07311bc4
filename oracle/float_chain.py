"""O_float: the float chain that defines what one substructure computes.

  Y_conv = (alpha * W_b) (x) (beta * X_q) + b      Eq. (1), in fp64
  Y_bn   = gamma * (Y_conv - mean) / sqrt(var + eps) + bn_beta
           Eq. (2), with sigma read as the standard deviation sqrt(var + eps)
           and the BN affine scale/shift included
  code   = #{ i : Y_bn > q_i }                     Eq. (3), ties go low

The convolution is an im2col followed by a float64 matrix product (a library
primitive). The integer-threshold path must give the same codes for every
element whose Y_bn is farther than a small band from every q_i (Table 2: the
integrated conversion matches the float network exactly). Residual joins add
the dequantized shortcut to Y_bn before the quantizer. Test infrastructure.
"""
import numpy as np


def _out_hw(h, w, k, stride, pad):
    return (h + 2 * pad - k) // stride + 1, (w + 2 * pad - k) // stride + 1


def conv(x, beta_in, w, alpha, bias, stride, pad, chunk=8):
    """Y_conv in fp64, NHWC [n][ho][wo][cout]."""
    n, h, wd, cin = x.shape
    cout, _, kh, kw = w.shape
    ho, wo = _out_hw(h, wd, kh, stride, pad)
    # the real filter alpha * W_b, laid out as [cout][(kh, kw, cin)]
    wf = (w.astype(np.float64) * np.asarray(alpha, np.float64)[:, None, None, None])
    wf = wf.transpose(0, 2, 3, 1).reshape(cout, kh * kw * cin)
    out = np.empty((n, ho, wo, cout), dtype=np.float64)
    for b0 in range(0, n, chunk):
        xb = x[b0:b0 + chunk].astype(np.float64) * beta_in
        xb = np.pad(xb, ((0, 0), (pad, pad), (pad, pad), (0, 0)))
        nb = xb.shape[0]
        cols = np.empty((nb, ho, wo, kh, kw, cin), dtype=np.float64)
        for i in range(kh):
            for j in range(kw):
                cols[:, :, :, i, j, :] = xb[:, i:i + stride * (ho - 1) + 1:stride,
                                            j:j + stride * (wo - 1) + 1:stride, :]
        y = cols.reshape(-1, kh * kw * cin) @ wf.T
        out[b0:b0 + nb] = y.reshape(nb, ho, wo, cout) + np.asarray(bias, np.float64)
    return out


def bn(y, mean, var, gamma, bn_beta, eps):
    return gamma * (y - mean) / np.sqrt(var + eps) + bn_beta


def quantize(ybn, q_thr):
    """Codes and the distance of each element to the nearest threshold."""
    q = np.asarray(q_thr, np.float64)
    code = np.zeros(ybn.shape, dtype=np.uint8)
    margin = np.full(ybn.shape, np.inf)
    for qi in q:
        code += (ybn > qi).astype(np.uint8)
        margin = np.minimum(margin, np.abs(ybn - qi))
    return code, margin


def substructure(x, p, stride, pad):
    """conv -> BN -> quantizer of one layer; returns (codes, margin)."""
    y = conv(x, p["beta_in"], p["w"], p["alpha"], p["bias"], stride, pad)
    ybn = bn(y, p["mean"], p["var"], p["gamma"], p["bn_beta"], p["eps"])
    return quantize(ybn, p["q_thr"])


def joined(x, p, stride, pad, shortcut_value):
    """Residual join: quantize(BN2(Y_conv) + shortcut); returns (codes, margin)."""
    y = conv(x, p["beta_in"], p["w"], p["alpha"], p["bias"], stride, pad)
    z = bn(y, p["mean"], p["var"], p["gamma"], p["bn_beta"], p["eps"]) + shortcut_value
    return quantize(z, p["q_thr"])


def downsample_value(x, pd, stride, pad):
    """BN_d of the 1x1 downsample conv's real output (the conv shortcut)."""
    y = conv(x, pd["beta_in"], pd["w"], pd["alpha"], pd["bias"], stride, pad)
    return bn(y, pd["mean"], pd["var"], pd["gamma"], pd["bn_beta"], pd["eps"])
