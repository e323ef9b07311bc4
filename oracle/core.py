"""ctypes wrappers over the C oracle (ifq_oracle.c). Test infrastructure."""
import ctypes
import os
import numpy as np

from .build import OUT as _LIB, build as _build

MUTATE_NO_FLIP = 1

_lib = None


def lib_path():
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            _build()
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i32, i64, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
        L.oracle_conv_acc.argtypes = [P, i32, i32, i32, i32, P, i32, i32, i32,
                                      i32, i32, i32, P]
        L.oracle_conv_acc.restype = i32
        L.oracle_fold.argtypes = [i32, i32, i64, i32, P, f64, P, P, P, P, P,
                                  f64, P, i32, P, P]
        L.oracle_fold.restype = i32
        L.oracle_codes.argtypes = [P, i64, i32, P, P, i32, P]
        L.oracle_codes.restype = None
        L.oracle_maxpool.argtypes = [P, i32, i32, i32, i32, i32, i32, i32, P]
        L.oracle_maxpool.restype = i32
        L.oracle_join_coeffs.argtypes = ([i32, i32, P, f64, P, P, P, P, P, f64,
                                          f64, P, P, P, P, P, P, f64, P])
        L.oracle_join_coeffs.restype = i32
        L.oracle_join_codes.argtypes = [P, P, i64, i32, P, P, i32, P]
        L.oracle_join_codes.restype = None
        L.oracle_num_threads.argtypes = []
        L.oracle_num_threads.restype = i32
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _f64(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float64)


def num_threads():
    return int(_load().oracle_num_threads())


def out_hw(h, w, k, stride, pad):
    return (h + 2 * pad - k) // stride + 1, (w + 2 * pad - k) // stride + 1


def conv_acc(x, w, stride, pad, in_bits):
    """Integer sums of Eq. (1). x: NHWC uint8 codes; w: OIHW int8 (+-1)."""
    x = np.ascontiguousarray(x, dtype=np.uint8)
    w = np.ascontiguousarray(w, dtype=np.int8)
    n, h, wd, cin = x.shape
    cout, cin2, kh, kw = w.shape
    assert cin2 == cin
    ho, wo = out_hw(h, wd, kh, stride, pad)
    acc = np.empty((n, ho, wo, cout), dtype=np.int32)
    rc = _load().oracle_conv_acc(_p(x), n, h, wd, cin, _p(w), cout, kh, kw,
                                 stride, pad, in_bits, _p(acc))
    if rc != 0:
        raise ValueError("oracle_conv_acc: sum outside the bound")
    return acc


def fold(alpha, beta_in, mean, var, gamma, bn_beta, eps, q_thr, k, in_bits,
         bias=None, flags=0):
    """Per-channel sign s and integer thresholds T (Eq. 6 -> Eq. 7, floored)."""
    alpha = _f64(alpha)
    q_thr = _f64(q_thr)
    c_out = alpha.shape[0]
    nq = q_thr.shape[0]
    out_bits = int(np.log2(nq + 1))
    assert (1 << out_bits) - 1 == nq
    s = np.empty(c_out, dtype=np.int32)
    t = np.empty((c_out, nq), dtype=np.int32)
    keep = [_f64(bias), _f64(mean), _f64(var), _f64(gamma), _f64(bn_beta)]
    rc = _load().oracle_fold(c_out, in_bits, int(k), out_bits, _p(alpha),
                             float(beta_in), *[_p(a) for a in keep],
                             float(eps), _p(q_thr), int(flags), _p(s), _p(t))
    if rc != 0:
        raise ValueError("oracle_fold: invalid parameters")
    return s, t


def codes(acc, s, t):
    acc = np.ascontiguousarray(acc, dtype=np.int32)
    s = np.ascontiguousarray(s, dtype=np.int32)
    t = np.ascontiguousarray(t, dtype=np.int32)
    c_out = acc.shape[-1]
    out = np.empty(acc.shape, dtype=np.uint8)
    _load().oracle_codes(_p(acc), acc.size // c_out, c_out, _p(s), _p(t),
                         t.shape[1], _p(out))
    return out


def maxpool(x, k, stride, mode):
    x = np.ascontiguousarray(x, dtype=np.uint8)
    n, h, w, c = x.shape
    m = {"valid": 0, "same": 1}[mode]
    if m == 0:
        ho, wo = (h - k) // stride + 1, (w - k) // stride + 1
    else:
        ho, wo = -(-h // stride), -(-w // stride)
    y = np.empty((n, ho, wo, c), dtype=np.uint8)
    rc = _load().oracle_maxpool(_p(x), n, h, w, c, k, stride, m, _p(y))
    if rc != 0:
        raise ValueError("oracle_maxpool: bad mode")
    return y


def join_coeffs(kind, main, beta2, beta_x, down=None):
    """(p, q, cc) per channel; main/down are dicts of per-channel params."""
    c_out = main["alpha"].shape[0]
    out = np.empty((c_out, 3), dtype=np.float64)
    m = {k: _f64(v) for k, v in main.items() if isinstance(v, np.ndarray)}
    if kind == "identity":
        kd, d = 1, {}
        epsd = 0.0
    else:
        kd = 2
        d = {k: _f64(v) for k, v in down.items() if isinstance(v, np.ndarray)}
        epsd = float(down["eps"])
    g = lambda dd, key: _p(dd.get(key))
    rc = _load().oracle_join_coeffs(
        c_out, kd, _p(m["alpha"]), float(beta2), g(m, "bias"), _p(m["mean"]),
        _p(m["var"]), _p(m["gamma"]), _p(m["bn_beta"]), float(main["eps"]),
        float(beta_x), g(d, "alpha"), g(d, "bias"), g(d, "mean"), g(d, "var"),
        g(d, "gamma"), g(d, "bn_beta"), epsd, _p(out))
    if rc != 0:
        raise ValueError("oracle_join_coeffs: bad kind")
    return out


def join_codes(a, sc, coef, q_thr):
    a = np.ascontiguousarray(a, dtype=np.int32)
    sc = np.ascontiguousarray(sc, dtype=np.int32)
    assert a.shape == sc.shape
    q_thr = _f64(q_thr)
    c_out = a.shape[-1]
    out = np.empty(a.shape, dtype=np.uint8)
    _load().oracle_join_codes(_p(a), _p(sc), a.size // c_out, c_out,
                              _p(np.ascontiguousarray(coef)), _p(q_thr),
                              q_thr.shape[0], _p(out))
    return out
