"""GPU parity of every variant of the register-blocked 3x3 kernels, conv_w2,
the persistent conv_wp and the wave-independent conv_wv
(ifq_conv_forward_variant), int8 and fp4 instances: int32 sums and output
codes (thresholds of Eq. 7/8, the identity residual join, or the join with
a 1x1 downsample computed in the kernel) must equal the oracle's bit for
bit on the same seeded inputs, on small ragged layers that span several
tiles and on the ResNet-18-shaped stack's full-size layers."""
import zlib

import numpy as np
import pytest

from gpu_util import (B64, U2, gpu_layer, oracle_layer, expect_layout, make_layer,
                      params_for, codes_for)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1911_08076_amd as P
    return P


# (name, n, h, w, cin, cout, stride)
SMALL = [
    ("r13x11_64_128", 2, 13, 11, 64, 128, 1),
    ("s2_15_64_128", 2, 15, 15, 64, 128, 2),
    ("r28_64_64", 1, 28, 28, 64, 64, 1),
    ("r14_256_256", 2, 14, 14, 256, 256, 1),
    ("r7_512_512", 3, 7, 7, 512, 512, 1),
    ("s2_14_128_256", 5, 14, 14, 128, 256, 2),
    ("r9_192_64", 1, 9, 9, 192, 64, 1),
    ("r5_128_96", 3, 5, 6, 128, 96, 1),
    # fewer half units than waves, units across images, ragged tails
    ("r5x7_64_64", 3, 5, 7, 64, 64, 1),
    ("r9_64_64", 5, 9, 9, 64, 64, 1),
    ("r17x23_64_64", 3, 17, 23, 64, 64, 1),
]

FULL = [
    ("l1", 64, 56, 56, 64, 64, 1),
    # more tiles than two workgroups per CU take at once: the persistent
    # kernel runs 3 (ragged: the last workgroup's one tile is partial) and 4
    # tiles per workgroup through its double buffers
    ("l1_n97", 97, 56, 56, 64, 64, 1),
    ("l1_n160", 160, 56, 56, 64, 64, 1),
    ("l2", 64, 28, 28, 128, 128, 1),
    ("l3", 64, 14, 14, 256, 256, 1),
    ("l4", 64, 7, 7, 512, 512, 1),
    ("l3.0.conv1_s2", 64, 28, 28, 128, 256, 2),
]


NVAR = 17   # conv_w2's ten, then conv_wp's two, conv_wv's four and conv_wvh's one
NW2 = 10    # conv_w2's variants


def _nvar(P):
    return P.ifq_conv_variant_count()


def _host_lib():
    """The library for host-side queries at collection (no GPU needed), or
    None where it is not built: then every combination is collected and the
    test itself skips the ones no variant takes."""
    try:
        import paper_1911_08076_amd as P
        P.ifq_conv_variant_count()
        return P
    except Exception:
        return None


def _thr_join(P, join, q=(0.25, 0.75, 1.25)):
    if not join:
        return None
    jn = P.make_join(P.IFQ_JOIN_IDENTITY, B64, None, None, list(q))
    jn.table = 0x1000
    return jn


def _combos(cases, full=False):
    """(case, join, variant) for the variants that take the layer (the planner's
    host-side answer), identity joins only on shape-preserving layers, and the
    multi-tile batches only on the persistent kernel."""
    P = _host_lib()
    out = []
    for c in cases:
        name, n, h, w, cin, cout, st = c
        for join in (False, True):
            if join and (st != 1 or cin != cout):
                continue
            for v in range(NVAR):
                if full and name in ("l1_n97", "l1_n160") and v < NW2:
                    continue   # one tile per workgroup: the batch-64 case covers it
                if P is not None:
                    ob = B64 if cout % 64 == 0 else U2
                    d = P.conv_desc(n, h, w, cin, cout, 3, st, 1, 2, 2, B64, ob)
                    if not P.ifq_conv_variant_name(d, _thr_join(P, join), v):
                        continue
                out.append(pytest.param(c, join, v, id="%s-%s-v%d" % (
                    name, "idj" if join else "thr", v)))
    return out


def _check(P, case, variant, join, out_layout=None):
    name, n, h, w, cin, cout, st = case
    if out_layout is None:
        out_layout = B64 if cout % 64 == 0 else U2
    L = make_layer(name, h, w, cin, cout, 3, st, 1, 2, 2,
                   ("identity", "x") if join else None)
    if join and (st != 1 or cin != cout):
        pytest.skip("an identity join needs the block input's shape")
    seed = zlib.crc32((name + str(join)).encode()) % 997
    p = params_for(seed, L)
    x = codes_for(seed, (n, h, w, cin), 2)
    d = P.conv_desc(n, h, w, cin, cout, 3, st, 1, 2, 2, B64, out_layout)
    jn = _thr_join(P, join, p["q_thr"])
    if not P.ifq_conv_variant_name(d, jn, variant):
        pytest.skip("variant %d does not take %s" % (variant, name))
    sc = x if join else None
    want_acc, want = oracle_layer(L, x, p, shortcut=sc)
    acc, got = gpu_layer(P, L, n, x, p, in_layout=B64, out_layout=out_layout, shortcut=sc,
                         sc_layout=B64, variant=variant)
    assert np.array_equal(acc, want_acc), (name, variant)
    assert np.array_equal(got, expect_layout(want, out_layout)), (name, variant)
    assert len(np.unique(want)) > 1


def test_variant_count(P):
    assert _nvar(P) == NVAR


@pytest.mark.parametrize("case,join,variant", _combos(SMALL))
def test_variant_small_bit_exact(P, case, join, variant):
    _check(P, case, variant, join)


@pytest.mark.parametrize("case,join,variant", _combos(FULL, full=True))
def test_variant_full_size_bit_exact(P, case, join, variant):
    _check(P, case, variant, join)


def test_variant_u2_output(P):
    # the NHWC packed output layout through the same tile copy-out
    _check(P, SMALL[0], 0, False, out_layout=U2)


@pytest.mark.parametrize("variant", range(NW2 + 2, NVAR), ids=lambda v: "v%d" % v)
@pytest.mark.parametrize("join", [False, True], ids=["thr", "idj"])
def test_wave_kernel_nhwc_packed_layouts(P, variant, join):
    # the wave-independent kernel's own stores and shortcut loads in the NHWC
    # packed layout (output, and the identity join's shortcut), on a ragged
    # multi-image layer: 64 channels, or 256 for the 32-channel instance
    # (which writes and reads half of each 64-channel cell)
    for case in (("r17x23_64_64", 3, 17, 23, 64, 64, 1), ("r9x13_256_256", 3, 9, 13, 256, 256, 1)):
        name, n, h, w, cin, cout, st = case
        d = P.conv_desc(n, h, w, cin, cout, 3, st, 1, 2, 2, B64, U2)
        jn = _thr_join(P, join)
        if jn is not None:
            jn.layout = U2
        if P.ifq_conv_variant_name(d, jn, variant):
            break
    L = make_layer(name, h, w, cin, cout, 3, st, 1, 2, 2, ("identity", "x") if join else None)
    seed = zlib.crc32((name + "u2" + str(join)).encode()) % 997
    p = params_for(seed, L)
    x = codes_for(seed, (n, h, w, cin), 2)
    sc = codes_for(seed + 1, (n, h, w, cin), 2) if join else None
    jn = _thr_join(P, join, p["q_thr"])
    if jn is not None:
        jn.layout = U2
    name_v = P.ifq_conv_variant_name(d, jn, variant)
    assert name_v.startswith(("conv_wv<", "conv_wvh<")), name_v
    want_acc, want = oracle_layer(L, x, p, shortcut=sc)
    acc, got = gpu_layer(P, L, n, x, p, in_layout=B64, out_layout=U2, shortcut=sc,
                         sc_layout=U2, variant=variant)
    assert np.array_equal(acc, want_acc), variant
    assert np.array_equal(got, expect_layout(want, U2)), variant
    assert len(np.unique(want)) > 1


# downsampling blocks' second conv with the 1x1 stride-2 downsample fused:
# (n, h_in, c_in, c_out); ragged, small and the full ResNet-18 shapes
FUSED = [(2, 56, 64, 128), (3, 28, 128, 256), (2, 14, 256, 512), (5, 13, 64, 128),
         (64, 56, 64, 128), (64, 28, 128, 256), (64, 14, 256, 512)]


def _fused_join(P, shape):
    n, hin, cin, cout = shape
    ho = (hin - 1) // 2 + 1
    d = P.conv_desc(n, ho, ho, cout, cout, 3, 1, 1, 2, 2, B64, B64)
    dd = P.conv_desc(n, hin, hin, cin, cout, 1, 2, 0, 2, 0, B64, P.IFQ_LAYOUT_I32_NHWC)
    jn = P.make_join(P.IFQ_JOIN_CONV_FUSED, B64, None, None, [0.25, 0.75, 1.25], down=dd)
    jn.coef = 0x1000
    jn.down_w = 0x1000
    return d, jn


def _fused_combos():
    P = _host_lib()
    out = []
    for f in FUSED:
        for v in range(NVAR):
            if P is not None:
                d, jn = _fused_join(P, f)
                if not P.ifq_conv_variant_name(d, jn, v):
                    continue
            out.append(pytest.param(f, v, id="%s-v%d" % ("x".join(map(str, f)), v)))
    return out


@pytest.mark.parametrize("shape,variant", _fused_combos())
def test_variant_fused_downsample_bit_exact(P, shape, variant):
    n, hin, cin, cout = shape
    D = make_layer("down", hin, hin, cin, cout, 1, 2, 0, 2, 0)
    ho = (hin - 1) // 2 + 1
    L = make_layer("conv2", ho, ho, cout, cout, 3, 1, 1, join=("conv", "d", "down"))
    d, jn = _fused_join(P, shape)
    if not P.ifq_conv_variant_name(d, jn, variant):
        pytest.skip("variant %d does not take %s" % (variant, shape))
    seed = 31 + hin + n
    pd = params_for(seed, D)
    p = params_for(seed + 1, L)
    xin = codes_for(seed, (n, hin, hin, cin), 2)
    x = codes_for(seed + 1, (n, ho, ho, cout), 2)
    want_d, _ = oracle_layer(D, xin, pd)
    want_acc, want = oracle_layer(L, x, p, shortcut=want_d, down=pd)
    acc, got = gpu_layer(P, L, n, x, p, in_layout=B64, out_layout=B64, down=pd,
                         fused_down=(D, xin), variant=variant)
    assert np.array_equal(acc, want_acc), (shape, variant)
    assert np.array_equal(got, expect_layout(want, B64)), (shape, variant)
    assert len(np.unique(want)) > 1
