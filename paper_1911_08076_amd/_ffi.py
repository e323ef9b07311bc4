"""ctypes mirror of include/ifq.h and the loader of libifq.so.

Loading fails loudly (ImportError) when the library has not been built: there
is no fallback implementation of any entry point.
"""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
# always the in-tree build next to this file
LIB_PATH = os.path.join(HERE, "libifq.so")

IFQ_OK = 0
IFQ_ERR_INVALID_ARGUMENT = -1
IFQ_ERR_UNSUPPORTED = -2
IFQ_ERR_HIP = -3
IFQ_ERR_INSUFFICIENT_BUFFER = -4

IFQ_LAYOUT_I8_NHWC = 0
IFQ_LAYOUT_U2_NHWC_PACKED = 1
IFQ_LAYOUT_I32_NHWC = 2
IFQ_LAYOUT_U2_BLOCK64 = 3

IFQ_POOL_VALID = 0
IFQ_POOL_SAME = 1

IFQ_JOIN_NONE = 0
IFQ_JOIN_IDENTITY = 1
IFQ_JOIN_CONV = 2
IFQ_JOIN_CONV_FUSED = 3

IFQ_LAYER_CONV = 0
IFQ_LAYER_POOL = 1
IFQ_LAYER_CONV_POOL = 2
IFQ_LAYER_CONV_FP4 = 3
IFQ_LAYER_CONV_POOL_FP4 = 4

IFQ_MAX_THRESHOLDS = 15

i32 = ctypes.c_int32
i64 = ctypes.c_int64
f64 = ctypes.c_double
vp = ctypes.c_void_p
dp = ctypes.POINTER(ctypes.c_double)
size_t = ctypes.c_size_t


class ConvDesc(ctypes.Structure):
    _fields_ = [("n", i32), ("h", i32), ("w", i32), ("c_in", i32),
                ("c_out", i32), ("kh", i32), ("kw", i32), ("stride", i32),
                ("pad", i32), ("in_bits", i32), ("out_bits", i32),
                ("in_layout", i32), ("out_layout", i32)]


class FoldParams(ctypes.Structure):
    _fields_ = [("c_out", i32), ("in_bits", i32), ("out_bits", i32),
                ("reserved", i32), ("k", i64), ("alpha", vp), ("beta_in", f64),
                ("bias", vp), ("mean", vp), ("var", vp), ("gamma", vp),
                ("bn_beta", vp), ("eps", f64), ("q_thr", vp)]


class JoinParams(ctypes.Structure):
    _fields_ = [("c_out", i32), ("kind", i32), ("alpha", vp), ("beta_in", f64),
                ("bias", vp), ("mean", vp), ("var", vp), ("gamma", vp),
                ("bn_beta", vp), ("eps", f64), ("beta_x", f64),
                ("alpha_d", vp), ("bias_d", vp), ("mean_d", vp), ("var_d", vp),
                ("gamma_d", vp), ("bn_beta_d", vp), ("eps_d", f64)]


class Join(ctypes.Structure):
    _fields_ = [("kind", i32), ("layout", i32), ("shortcut", vp), ("coef", vp),
                ("table", vp), ("n_q", i32), ("sc_bits", i32),
                ("q_thr", f64 * IFQ_MAX_THRESHOLDS), ("down_w", vp),
                ("down", ConvDesc)]


class PoolDesc(ctypes.Structure):
    _fields_ = [("n", i32), ("h", i32), ("w", i32), ("c", i32), ("k", i32),
                ("stride", i32), ("mode", i32), ("bits", i32), ("layout", i32)]


class Layer(ctypes.Structure):
    _fields_ = [("kind", i32), ("src", i32), ("dst", i32), ("join_src", i32),
                ("conv", ConvDesc), ("w_packed", vp), ("thr", vp),
                ("join", Join), ("pool", PoolDesc)]


class Stack(ctypes.Structure):
    _fields_ = [("n_layers", i32), ("n_slots", i32),
                ("layers", ctypes.POINTER(Layer)), ("events", vp)]


# (name, restype, argtypes) of every exported entry point
SIGNATURES = [
    ("ifq_version", ctypes.c_char_p, []),
    ("ifq_last_error", ctypes.c_char_p, []),
    ("ifq_tensor_bytes", size_t, [i64, i64, i64, i64, i32]),
    ("ifq_conv_output_dims", i32, [ctypes.POINTER(ConvDesc),
                                   ctypes.POINTER(i32), ctypes.POINTER(i32)]),
    ("ifq_packed_weight_bytes", size_t, [ctypes.POINTER(ConvDesc)]),
    ("ifq_pack_weights", i32, [ctypes.POINTER(ConvDesc), vp, vp, size_t]),
    ("ifq_fold_thresholds", i32, [ctypes.POINTER(FoldParams), vp]),
    ("ifq_fold_thresholds_compact", i32, [ctypes.POINTER(FoldParams), f64, f64, vp]),
    ("ifq_expand_thresholds", i32, [vp, i32, i32, i64, i32, vp, vp]),
    ("ifq_fold_join", i32, [ctypes.POINTER(JoinParams), vp]),
    ("ifq_fold_join_table", i32, [ctypes.POINTER(JoinParams), i32, i64, i32, i32,
                                  vp, vp]),
    ("ifq_conv_kernel_name", ctypes.c_char_p, [ctypes.POINTER(ConvDesc), ctypes.POINTER(Join)]),
    ("ifq_conv_workspace_bytes", size_t, [ctypes.POINTER(ConvDesc)]),
    ("ifq_conv_variant_count", i32, []),
    ("ifq_conv_variant_fp4", i32, [i32]),
    ("ifq_conv_variant_name", ctypes.c_char_p, [ctypes.POINTER(ConvDesc), ctypes.POINTER(Join),
                                               i32]),
    ("ifq_conv_forward_variant", i32, [ctypes.POINTER(ConvDesc), vp, vp, vp,
                                       ctypes.POINTER(Join), vp, vp, i32, vp]),
    ("ifq_conv_split_workspace_bytes", size_t, [ctypes.POINTER(ConvDesc), i32, i32]),
    ("ifq_conv_forward_split", i32, [ctypes.POINTER(ConvDesc), vp, vp, vp, vp, vp, i32, i32,
                                     vp, size_t, vp]),
    ("ifq_conv_forward", i32, [ctypes.POINTER(ConvDesc), vp, vp, vp,
                               ctypes.POINTER(Join), vp, vp, vp, size_t, vp]),
    ("ifq_conv_forward_fp4", i32, [ctypes.POINTER(ConvDesc), vp, vp, vp,
                                   ctypes.POINTER(Join), vp, vp]),
    ("ifq_conv_fp4_kernel_name", ctypes.c_char_p, [ctypes.POINTER(ConvDesc),
                                                   ctypes.POINTER(Join)]),
    ("ifq_packed_weight_bytes_fp4", size_t, [ctypes.POINTER(ConvDesc)]),
    ("ifq_pack_weights_fp4", i32, [ctypes.POINTER(ConvDesc), vp, vp, size_t]),
    ("ifq_conv_pool_forward_fp4", i32, [ctypes.POINTER(ConvDesc), ctypes.POINTER(PoolDesc),
                                        vp, vp, vp, vp, vp]),
    ("ifq_conv_pool_fp4_kernel_name", ctypes.c_char_p, [ctypes.POINTER(ConvDesc),
                                                        ctypes.POINTER(PoolDesc)]),
    ("ifq_conv_pool_forward", i32, [ctypes.POINTER(ConvDesc), ctypes.POINTER(PoolDesc),
                                    vp, vp, vp, vp, vp]),
    ("ifq_conv_pool_kernel_name", ctypes.c_char_p, [ctypes.POINTER(ConvDesc),
                                                    ctypes.POINTER(PoolDesc)]),
    ("ifq_maxpool_codes", i32, [ctypes.POINTER(PoolDesc), vp, vp, vp]),
    ("ifq_convert_codes", i32, [i64, i64, i64, i32, i32, i32, vp, vp, vp]),
    ("ifq_stack_workspace_bytes", size_t, [ctypes.POINTER(Stack)]),
    ("ifq_stack_slot_info", i32, [ctypes.POINTER(Stack), i32,
                                  ctypes.POINTER(size_t), ctypes.POINTER(size_t)]),
    ("ifq_run_stack", i32, [ctypes.POINTER(Stack), vp, vp, vp, size_t, vp]),
    ("ifq_run_stack_static", i32, [ctypes.POINTER(Stack), vp, vp, vp]),
    ("ifq_static_workspace_bytes", size_t, []),
]

_lib = None


def load():
    """Load libifq.so once; raise ImportError if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            "libifq.so is not built (expected at %s); run "
            "`python paper_1911_08076_amd/build.py` or "
            "`python -c 'import __graft_entry__; __graft_entry__.build()'`"
            % LIB_PATH)
    # torch ships its own HIP runtime under the soname libamdhip64.so.7.
    # Importing torch first makes the dynamic loader bind libifq.so to that
    # same copy, so the process holds one HIP runtime and torch's streams and
    # device pointers are valid in the library. Loaded the other way round,
    # two runtimes end up in the process and the library's launches fail.
    import torch  # noqa: F401
    lib = ctypes.CDLL(LIB_PATH)
    for name, res, args in SIGNATURES:
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib
