"""Python binding of the C ABI: one function per entry point, same names.

Only argument marshalling happens here (descriptors, pointers, the stream
handle). Every step of the quantized substructure runs in libifq.so: host-side
packing and folding in its C++ code, everything else in its HIP kernels.
Device tensors are torch tensors; host arrays are NumPy arrays.
"""
import ctypes

import numpy as np

from . import _ffi
from ._ffi import (ConvDesc, FoldParams, JoinParams, Join, PoolDesc, Stack,
                   IFQ_OK, IFQ_JOIN_NONE, IFQ_MAX_THRESHOLDS)


class IfqError(RuntimeError):
    def __init__(self, status, func, message):
        super().__init__("%s failed with status %d: %s" % (func, status, message))
        self.status = status


def _lib():
    return _ffi.load()


def _check(status, func):
    if status != IFQ_OK:
        msg = _lib().ifq_last_error().decode(errors="replace")
        raise IfqError(status, func, msg)


def _ptr(t):
    """Device or host address of a torch tensor / NumPy array (None -> NULL)."""
    if t is None:
        return None
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _f64(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float64)


def conv_desc(n, h, w, c_in, c_out, k, stride, pad, in_bits, out_bits,
              in_layout=_ffi.IFQ_LAYOUT_I8_NHWC, out_layout=None, kw=None):
    if out_layout is None:
        out_layout = (_ffi.IFQ_LAYOUT_I32_NHWC if out_bits == 0
                      else _ffi.IFQ_LAYOUT_I8_NHWC)
    return ConvDesc(n, h, w, c_in, c_out, k, k if kw is None else kw, stride,
                    pad, in_bits, out_bits, in_layout, out_layout)


def pool_desc(n, h, w, c, k, stride, mode, bits=2,
              layout=_ffi.IFQ_LAYOUT_I8_NHWC):
    return PoolDesc(n, h, w, c, k, stride, mode, bits, layout)


def ifq_version():
    return _lib().ifq_version().decode()


def ifq_last_error():
    return _lib().ifq_last_error().decode(errors="replace")


def ifq_tensor_bytes(n, h, w, c, layout):
    return int(_lib().ifq_tensor_bytes(n, h, w, c, layout))


def ifq_conv_output_dims(desc):
    ho, wo = ctypes.c_int32(), ctypes.c_int32()
    _check(_lib().ifq_conv_output_dims(ctypes.byref(desc), ctypes.byref(ho),
                                       ctypes.byref(wo)), "ifq_conv_output_dims")
    return ho.value, wo.value


def ifq_packed_weight_bytes(desc):
    return int(_lib().ifq_packed_weight_bytes(ctypes.byref(desc)))


def ifq_pack_weights(desc, w_oihw, dst=None):
    """Pack +-1 OIHW int8 weights into the device blob (host uint8 array)."""
    w = np.ascontiguousarray(w_oihw, dtype=np.int8)
    nbytes = ifq_packed_weight_bytes(desc)
    if dst is None:
        dst = np.zeros(max(nbytes, 1), dtype=np.uint8)
    _check(_lib().ifq_pack_weights(ctypes.byref(desc), _ptr(w), _ptr(dst),
                                   dst.nbytes), "ifq_pack_weights")
    return dst


def ifq_fold_thresholds(c_out, in_bits, out_bits, k, alpha, beta_in, q_thr,
                        bias=None, mean=None, var=None, gamma=None,
                        bn_beta=None, eps=0.0):
    """Integer threshold records [c_out][2^out_bits] = {s, T_1..T_{2^k-1}}."""
    arrs = [_f64(a) for a in (alpha, bias, mean, var, gamma, bn_beta, q_thr)]
    p = FoldParams(c_out, in_bits, out_bits, 0, int(k), _ptr(arrs[0]),
                   float(beta_in), _ptr(arrs[1]), _ptr(arrs[2]), _ptr(arrs[3]),
                   _ptr(arrs[4]), _ptr(arrs[5]), float(eps), _ptr(arrs[6]))
    out = np.zeros((c_out, 1 << out_bits), dtype=np.int32)
    _check(_lib().ifq_fold_thresholds(ctypes.byref(p), _ptr(out)),
           "ifq_fold_thresholds")
    return out


# One compact threshold record (ifq_thr_compact): base', offset', s, cstar.
THR_COMPACT = np.dtype([("base", "<f8"), ("offset", "<f8"), ("s", "<i4"), ("cstar", "<i4")])


def ifq_fold_thresholds_compact(c_out, in_bits, out_bits, k, alpha, beta_in, base, offset,
                                bias=None, mean=None, var=None, gamma=None,
                                bn_beta=None, eps=0.0):
    """Compact records (THR_COMPACT, c_out of them) of a uniform quantizer
    q_i = i*base + offset."""
    arrs = [_f64(a) for a in (alpha, bias, mean, var, gamma, bn_beta)]
    p = FoldParams(c_out, in_bits, out_bits, 0, int(k), _ptr(arrs[0]),
                   float(beta_in), _ptr(arrs[1]), _ptr(arrs[2]), _ptr(arrs[3]),
                   _ptr(arrs[4]), _ptr(arrs[5]), float(eps), None)
    out = np.zeros(c_out, dtype=THR_COMPACT)
    _check(_lib().ifq_fold_thresholds_compact(ctypes.byref(p), float(base), float(offset),
                                              _ptr(out)), "ifq_fold_thresholds_compact")
    return out


def ifq_expand_thresholds(recs, c_out, in_bits, k, out_bits, thr, stream=None):
    """Device: compact records -> int32 records [c_out][2^out_bits] in thr."""
    _check(_lib().ifq_expand_thresholds(_ptr(recs), int(c_out), int(in_bits), int(k),
                                        int(out_bits), _ptr(thr), _stream(stream)),
           "ifq_expand_thresholds")


def _join_params(kind, main, beta_x, down=None):
    m = {k: _f64(main.get(k)) for k in ("alpha", "bias", "mean", "var", "gamma",
                                          "bn_beta")}
    d = {k: None for k in m}
    eps_d = 0.0
    if kind == _ffi.IFQ_JOIN_CONV:
        d = {k: _f64(down.get(k)) for k in m}
        eps_d = float(down["eps"])
    c_out = m["alpha"].shape[0]
    p = JoinParams(c_out, kind, _ptr(m["alpha"]), float(main["beta_in"]),
                   _ptr(m["bias"]), _ptr(m["mean"]), _ptr(m["var"]),
                   _ptr(m["gamma"]), _ptr(m["bn_beta"]), float(main["eps"]),
                   float(beta_x), _ptr(d["alpha"]), _ptr(d["bias"]),
                   _ptr(d["mean"]), _ptr(d["var"]), _ptr(d["gamma"]),
                   _ptr(d["bn_beta"]), eps_d)
    return p, c_out, (m, d)


def ifq_fold_join(kind, main, beta_x, down=None):
    """Join coefficients [c_out][3] = {p, q, cc}.

    main / down: dicts with alpha, beta_in, bias, mean, var, gamma, bn_beta,
    eps (down is used for IFQ_JOIN_CONV only).
    """
    p, c_out, keep = _join_params(kind, main, beta_x, down)
    out = np.zeros((c_out, 3), dtype=np.float64)
    _check(_lib().ifq_fold_join(ctypes.byref(p), _ptr(out)), "ifq_fold_join")
    return out


def ifq_fold_join_table(main, beta_x, in_bits, k, out_bits, q_thr, x_bits=2):
    """Integer records of an identity join: int32 [c_out][2^x_bits][2^out_bits]
    = {s, T_1 .. T_{2^out_bits - 1}} for every shortcut code x."""
    p, c_out, keep = _join_params(_ffi.IFQ_JOIN_IDENTITY, main, beta_x)
    q = _f64(q_thr)
    out = np.zeros((c_out, 1 << x_bits, 1 << out_bits), dtype=np.int32)
    _check(_lib().ifq_fold_join_table(ctypes.byref(p), int(in_bits), int(k),
                                      int(x_bits), int(out_bits), _ptr(q),
                                      _ptr(out)), "ifq_fold_join_table")
    return out


def make_join(kind, layout, shortcut, coef, q_thr, table=None, down_w=None,
              down=None):
    """ifq_join; down_w (packed 1x1 weights) and down (its ConvDesc) are for
    IFQ_JOIN_CONV_FUSED, whose coef comes from ifq_fold_join(IFQ_JOIN_CONV)."""
    j = Join()
    j.kind = kind
    j.layout = layout
    j.shortcut = _ptr(shortcut)
    j.coef = _ptr(coef)
    j.table = _ptr(table)
    q = list(np.asarray(q_thr, dtype=np.float64))
    j.n_q = len(q)
    for i, v in enumerate(q[:IFQ_MAX_THRESHOLDS]):
        j.q_thr[i] = float(v)
    j.down_w = _ptr(down_w)
    if down is not None:
        j.down = down
    return j


def ifq_conv_kernel_name(desc, join=None):
    return _lib().ifq_conv_kernel_name(
        ctypes.byref(desc), ctypes.byref(join) if join is not None else None).decode()


def ifq_conv_workspace_bytes(desc):
    return int(_lib().ifq_conv_workspace_bytes(ctypes.byref(desc)))


def ifq_conv_forward(desc, x, w_packed, thr, y, join=None, acc_dump=None,
                     ws=None, stream=None):
    """ws None: a zero-filled device workspace of ifq_conv_workspace_bytes
    bytes is made for this call where the layer needs one (a K split)."""
    if ws is None:
        need = ifq_conv_workspace_bytes(desc)
        if need:
            import torch
            ws = torch.zeros(need, dtype=torch.uint8, device=y.device)
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(_lib().ifq_conv_forward(
        ctypes.byref(desc), _ptr(x), _ptr(w_packed), _ptr(thr),
        None if join is None else ctypes.byref(join), _ptr(y), _ptr(acc_dump),
        _ptr(ws), ws_bytes, _stream(stream)), "ifq_conv_forward")


def ifq_pack_weights_fp4(desc, w_oihw):
    """The fp4 weight blob (uint8) of OIHW +-1 weights."""
    w = np.ascontiguousarray(w_oihw, dtype=np.int8)
    n = int(_lib().ifq_packed_weight_bytes_fp4(ctypes.byref(desc)))
    if n == 0:
        raise IfqError(-1, "ifq_packed_weight_bytes_fp4", "no fp4 layout for this layer")
    out = np.zeros(n, dtype=np.uint8)
    _check(_lib().ifq_pack_weights_fp4(ctypes.byref(desc), _ptr(w), _ptr(out), n),
           "ifq_pack_weights_fp4")
    return out


def ifq_conv_fp4_kernel_name(desc, join=None):
    return _lib().ifq_conv_fp4_kernel_name(
        ctypes.byref(desc), ctypes.byref(join) if join is not None else None).decode()


def ifq_conv_forward_fp4(desc, x, w_fp4, thr, y, join=None, stream=None):
    _check(_lib().ifq_conv_forward_fp4(
        ctypes.byref(desc), _ptr(x), _ptr(w_fp4), _ptr(thr),
        None if join is None else ctypes.byref(join), _ptr(y), _stream(stream)),
        "ifq_conv_forward_fp4")


def ifq_conv_pool_forward(desc, pool, x, w_packed, thr, y, stream=None):
    _check(_lib().ifq_conv_pool_forward(
        ctypes.byref(desc), ctypes.byref(pool), _ptr(x), _ptr(w_packed), _ptr(thr),
        _ptr(y), _stream(stream)), "ifq_conv_pool_forward")


def ifq_conv_pool_forward_fp4(desc, pool, x, w_fp4, thr, y, stream=None):
    _check(_lib().ifq_conv_pool_forward_fp4(
        ctypes.byref(desc), ctypes.byref(pool), _ptr(x), _ptr(w_fp4), _ptr(thr), _ptr(y),
        _stream(stream)), "ifq_conv_pool_forward_fp4")


def ifq_conv_pool_fp4_kernel_name(desc, pool):
    return _lib().ifq_conv_pool_fp4_kernel_name(ctypes.byref(desc), ctypes.byref(pool)).decode()


def ifq_conv_pool_kernel_name(desc, pool):
    return _lib().ifq_conv_pool_kernel_name(ctypes.byref(desc), ctypes.byref(pool)).decode()


def ifq_maxpool_codes(desc, x, y, stream=None):
    _check(_lib().ifq_maxpool_codes(ctypes.byref(desc), _ptr(x), _ptr(y),
                                    _stream(stream)), "ifq_maxpool_codes")


def ifq_convert_codes(n, h, w, c, src_layout, dst_layout, src, dst, stream=None):
    _check(_lib().ifq_convert_codes(int(n), int(h), int(w), int(c), src_layout,
                                    dst_layout, _ptr(src), _ptr(dst),
                                    _stream(stream)),
           "ifq_convert_codes")


def ifq_stack_workspace_bytes(stack):
    return int(_lib().ifq_stack_workspace_bytes(ctypes.byref(stack)))


def ifq_stack_slot_info(stack, slot):
    off, nb = ctypes.c_size_t(), ctypes.c_size_t()
    _check(_lib().ifq_stack_slot_info(ctypes.byref(stack), int(slot),
                                      ctypes.byref(off), ctypes.byref(nb)),
           "ifq_stack_slot_info")
    return off.value, nb.value


def ifq_run_stack(stack, x, y, ws, stream=None):
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(_lib().ifq_run_stack(ctypes.byref(stack), _ptr(x), _ptr(y),
                                _ptr(ws), ws_bytes, _stream(stream)),
           "ifq_run_stack")


def ifq_run_stack_static(stack, x, y, stream=None):
    _check(_lib().ifq_run_stack_static(ctypes.byref(stack), _ptr(x), _ptr(y), _stream(stream)),
           "ifq_run_stack_static")


def ifq_static_workspace_bytes():
    return int(_lib().ifq_static_workspace_bytes())


def ifq_conv_variant_count():
    return int(_lib().ifq_conv_variant_count())


def ifq_conv_variant_fp4(variant):
    """1: the variant runs on the fp4 scaled MFMA (takes the fp4 weight
    blob); 0: int8 MFMA; -1: no such variant."""
    return int(_lib().ifq_conv_variant_fp4(int(variant)))


def kernel_is_fp4(name):
    """Whether a kernel name (as ifq_conv_kernel_name returns it) is an fp4
    instance: the fp4 flag true (the windowed kernel's last template
    argument, conv_w2's ninth, conv_wp's fifth, conv_wv's and conv_wvh's second)."""
    if name.startswith("conv_halo<"):
        return name.endswith(", true>")
    for kern, pos in (("conv_w2<", 8), ("conv_wp<", 4), ("conv_wv<", 1), ("conv_wvh<", 1)):
        if name.startswith(kern):
            return name[len(kern):-1].split(", ")[pos] == "true"
    return False


def ifq_conv_variant_name(desc, join, variant):
    return _lib().ifq_conv_variant_name(
        ctypes.byref(desc), ctypes.byref(join) if join is not None else None,
        int(variant)).decode()


def ifq_conv_split_workspace_bytes(desc, variant, ksplit):
    return int(_lib().ifq_conv_split_workspace_bytes(ctypes.byref(desc), int(variant),
                                                     int(ksplit)))


def ifq_conv_forward_split(desc, x, w_packed, thr, y, variant, ksplit, ws, acc_dump=None,
                           stream=None):
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(_lib().ifq_conv_forward_split(
        ctypes.byref(desc), _ptr(x), _ptr(w_packed), _ptr(thr), _ptr(y), _ptr(acc_dump),
        int(variant), int(ksplit), _ptr(ws), ws_bytes, _stream(stream)),
        "ifq_conv_forward_split")


def ifq_conv_forward_variant(desc, x, w_packed, thr, y, variant, join=None, acc_dump=None,
                             stream=None):
    _check(_lib().ifq_conv_forward_variant(
        ctypes.byref(desc), _ptr(x), _ptr(w_packed), _ptr(thr),
        ctypes.byref(join) if join is not None else None, _ptr(y), _ptr(acc_dump),
        int(variant), _stream(stream)), "ifq_conv_forward_variant")
