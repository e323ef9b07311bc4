"""Pure-Python brute force for tiny layers (test infrastructure).

Nothing here is vectorised: every sum is a Python loop over Python ints, and
every code is decided by evaluating the composed float inequality of Eq. (6)
directly, so that a reader can check each line against the paper.
"""
import math


def conv_acc(x, w, stride, pad):
    """x: nested lists / array [n][h][w][cin]; w: [cout][cin][kh][kw]."""
    n, h, wd, cin = len(x), len(x[0]), len(x[0][0]), len(x[0][0][0])
    cout, kh, kw = len(w), len(w[0][0]), len(w[0][0][0])
    ho = (h + 2 * pad - kh) // stride + 1
    wo = (wd + 2 * pad - kw) // stride + 1
    out = [[[[0] * cout for _ in range(wo)] for _ in range(ho)] for _ in range(n)]
    for b in range(n):
        for oy in range(ho):
            for ox in range(wo):
                for o in range(cout):
                    s = 0
                    for i in range(kh):
                        for j in range(kw):
                            iy, ix = oy * stride - pad + i, ox * stride - pad + j
                            if 0 <= iy < h and 0 <= ix < wd:
                                for c in range(cin):
                                    s += int(w[o][c][i][j]) * int(x[b][iy][ix][c])
                    out[b][oy][ox][o] = s
    return out


def code_eq6(a, alpha, beta, bias, mean, var, gamma, bn_beta, eps, q_thr):
    """Eq. (6): quantize BN(alpha*beta*a + b) with thresholds q_thr, ties low."""
    y = alpha * beta * a + bias
    ybn = gamma * (y - mean) / math.sqrt(var + eps) + bn_beta
    return sum(1 for q in q_thr if ybn > q), min(abs(ybn - q) for q in q_thr)


def maxpool(x, k, stride, mode):
    n, h, wd, c = len(x), len(x[0]), len(x[0][0]), len(x[0][0][0])
    if mode == "valid":
        ho, wo = (h - k) // stride + 1, (wd - k) // stride + 1
    else:
        ho, wo = -(-h // stride), -(-wd // stride)
    out = [[[[0] * c for _ in range(wo)] for _ in range(ho)] for _ in range(n)]
    for b in range(n):
        for py in range(ho):
            for px in range(wo):
                for ch in range(c):
                    vals = [int(x[b][py * stride + i][px * stride + j][ch])
                            for i in range(k) for j in range(k)
                            if py * stride + i < h and px * stride + j < wd]
                    out[b][py][px][ch] = max(vals)
    return out
