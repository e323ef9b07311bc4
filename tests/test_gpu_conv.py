"""GPU parity of single layers through the C ABI: int32 sums and output codes
must equal the oracle's bit for bit on the same seeded inputs."""
import zlib

import numpy as np
import pytest

import oracle
from oracle import layout as olayout
from gpu_util import (I8, U2, I32, B64, gpu_layer, oracle_layer, expect_layout,
                      make_layer, params_for, codes_for, upload_codes, to_dev,
                      device)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1911_08076_amd as P
    return P


# (name, n, h, w, cin, cout, k, stride, pad, in_bits, out_bits)
LAYERS = [
    ("stack0_3x3_64", 1, 28, 28, 64, 64, 3, 1, 1, 2, 2),
    ("ragged_m", 2, 13, 11, 64, 128, 3, 1, 1, 2, 2),
    ("stride2", 2, 15, 15, 64, 128, 3, 2, 1, 2, 2),
    ("5x5_cin96", 1, 9, 9, 96, 256, 5, 1, 2, 2, 2),
    ("1x1_s2_int32", 2, 14, 14, 64, 128, 1, 2, 0, 2, 0),
    ("head_1x1_c30", 1, 13, 13, 512, 30, 1, 1, 0, 2, 0),
    ("first_8bit_cin3", 1, 20, 20, 3, 16, 3, 1, 1, 8, 2),
    ("cin16_cout32", 1, 18, 18, 16, 32, 3, 1, 1, 2, 2),
    ("cin32_cout64", 1, 12, 12, 32, 64, 3, 1, 1, 2, 2),
    ("cin5_cout24", 1, 7, 9, 5, 24, 3, 1, 1, 2, 2),
    ("cout7_bytes", 1, 6, 6, 16, 7, 3, 1, 1, 2, 2),
    ("k4608", 1, 7, 7, 512, 512, 3, 1, 1, 2, 2),
    ("in4_out4", 1, 8, 8, 64, 64, 3, 1, 1, 4, 4),
    ("in1_out1", 1, 9, 7, 32, 48, 3, 1, 1, 1, 1),
    ("cout384_cin384", 1, 13, 13, 384, 384, 3, 1, 1, 2, 2),
    ("valid_no_pad", 1, 10, 10, 64, 64, 3, 1, 0, 2, 2),
    ("8bit_cin16", 1, 10, 10, 16, 32, 3, 2, 1, 8, 2),
    # k-bit activations (Table 2/3 variants: 3 and 4 bits, 7 and 15 thresholds)
    ("in3_out3", 2, 11, 9, 64, 96, 3, 1, 1, 3, 3),
    ("in2_out3", 1, 9, 9, 128, 64, 3, 1, 1, 2, 3),
    ("in3_out4_5x5", 1, 9, 9, 96, 64, 5, 1, 2, 3, 4),
    ("in4_out2_s2", 2, 12, 12, 64, 64, 3, 2, 1, 4, 2),
    # AlexNet's fully connected layers as convs over the 6x6x256 pool5 output
    # (FC6: one 6x6 window) and over FC6's 1x1x4096 output (FC7), batch 32
    ("fc6_as_6x6_conv", 32, 6, 6, 256, 4096, 6, 1, 0, 2, 2),
    ("fc7_as_1x1_conv", 32, 1, 1, 4096, 4096, 1, 1, 0, 2, 2),
]


@pytest.mark.parametrize("case", LAYERS, ids=[c[0] for c in LAYERS])
def test_conv_layer_bit_exact(P, case):
    name, n, h, w, cin, cout, k, st, pad, ib, ob = case
    L = make_layer(name, h, w, cin, cout, k, st, pad, ib, ob)
    seed = zlib.crc32(name.encode()) % 997
    p = params_for(seed, L)
    x = codes_for(seed, (n, h, w, cin), ib)
    want_acc, want = oracle_layer(L, x, p)
    acc, got = gpu_layer(P, L, n, x, p)
    assert np.array_equal(acc, want_acc), name
    assert np.array_equal(got, want), name
    if ob:
        # the codes use more than one level (the comparison has teeth)
        assert len(np.unique(want)) > 1


FC_U2 = [("fc6_u2", 32, 6, 6, 256, 4096, 6), ("fc7_u2", 32, 1, 1, 4096, 4096, 1)]


@pytest.mark.parametrize("case", FC_U2, ids=[c[0] for c in FC_U2])
def test_fc_as_conv_on_mfma_path(P, case):
    # the same layers from 2-bit packed codes: the MFMA kernel takes any kh x kw
    name, n, h, w, cin, cout, k = case
    L = make_layer(name, h, w, cin, cout, k, 1, 0, 2, 2)
    d = P.conv_desc(n, h, w, cin, cout, k, 1, 0, 2, 2, U2, U2)
    assert P.ifq_conv_kernel_name(d).startswith("conv_mfma<")
    seed = zlib.crc32(name.encode()) % 997
    p = params_for(seed, L)
    x = codes_for(seed, (n, h, w, cin), 2)
    want_acc, want = oracle_layer(L, x, p)
    acc, got = gpu_layer(P, L, n, x, p, in_layout=U2, out_layout=U2)
    assert np.array_equal(acc, want_acc), name
    assert np.array_equal(got, expect_layout(want, U2)), name
    assert len(np.unique(want)) > 1


# 8-bit input with c_in <= 4 (a detector's first layer) runs the small-channel
# kernel: one YOLO-c1-sized layer (several output rows per workgroup, a
# ragged last tile), and shapes across its parameters (c_in 1..4, stride 2,
# 1x1 and 4x4 filters, 1..4 row blocks of 16 output channels, int32 output).
# (name, n, h, w, cin, cout, k, stride, pad, out_bits)
SMALL8 = [
    ("s8_yolo_c1", 2, 415, 416, 3, 16, 3, 1, 1, 2),
    ("s8_cin1_s2_c64", 3, 33, 31, 1, 64, 3, 2, 1, 2),
    ("s8_cin4_1x1_c48", 2, 17, 19, 4, 48, 1, 1, 0, 2),
    ("s8_cin2_c33_i32", 2, 21, 20, 2, 33, 3, 1, 1, 0),
    ("s8_cin3_4x4_s2_pad0", 1, 23, 29, 3, 16, 4, 2, 0, 2),
]


@pytest.mark.parametrize("case", SMALL8, ids=[c[0] for c in SMALL8])
def test_small8_bit_exact(P, case):
    name, n, h, w, cin, cout, k, st, pad, ob = case
    L = make_layer(name, h, w, cin, cout, k, st, pad, 8, ob)
    d = P.conv_desc(n, h, w, cin, cout, k, st, pad, 8, ob, I8, I8 if ob else I32)
    assert P.ifq_conv_kernel_name(d).startswith("conv_small8<")
    seed = zlib.crc32(name.encode()) % 997
    p = params_for(seed, L)
    x = codes_for(seed, (n, h, w, cin), 8)
    want_acc, want = oracle_layer(L, x, p)
    outs = [I8, U2] if ob else [I32]
    for out_l in outs:
        acc, got = gpu_layer(P, L, n, x, p, in_layout=I8, out_layout=out_l)
        assert np.array_equal(acc, want_acc), (name, out_l)
        assert np.array_equal(got, expect_layout(want, out_l)), (name, out_l)
    if ob:
        assert len(np.unique(want)) > 1



# 2-bit packed input with c_in 16 or 32 (a detector's second and third
# layers) runs the small-channel 2-bit kernel: the YOLO c2 and c3 shapes,
# and shapes across its parameters (one and two blocks of 32 output channels,
# half-used blocks, 1-pixel-wide and 1-row images where every tap but the
# centre column or row is padding, a ragged last row tile).
# (name, n, h, w, cin, cout)
SMALL2 = [
    ("s2_yolo_c2", 2, 208, 208, 16, 32),
    ("s2_yolo_c3", 2, 104, 104, 32, 64),
    ("s2_cin16_c48_ragged", 3, 37, 29, 16, 48),
    ("s2_cin32_c4", 2, 9, 11, 32, 4),
    ("s2_cin32_c36_1x1_image", 5, 1, 1, 32, 36),
    ("s2_cin16_one_row", 2, 1, 57, 16, 16),
    ("s2_cin16_one_column", 1, 67, 1, 16, 64),
    ("s2_cin32_c20", 3, 23, 17, 32, 20),
]


@pytest.mark.parametrize("case", SMALL2, ids=[c[0] for c in SMALL2])
def test_small2_bit_exact(P, case):
    name, n, h, w, cin, cout = case
    L = make_layer(name, h, w, cin, cout, 3, 1, 1, 2, 2)
    seed = zlib.crc32(name.encode()) % 997
    p = params_for(seed, L)
    x = codes_for(seed, (n, h, w, cin), 2)
    want_acc, want = oracle_layer(L, x, p)
    outs = [U2, B64] if cout % 64 == 0 else [U2]
    for out_l in outs:
        d = P.conv_desc(n, h, w, cin, cout, 3, 1, 1, 2, 2, U2, out_l)
        assert P.ifq_conv_kernel_name(d).startswith("conv_small2<"), (name, out_l)
        acc, got = gpu_layer(P, L, n, x, p, in_layout=U2, out_layout=out_l)
        assert np.array_equal(acc, want_acc), (name, out_l)
        assert np.array_equal(got, expect_layout(want, out_l)), (name, out_l)
        # without the sums dumped (the launch the stacks make)
        _, got = gpu_layer(P, L, n, x, p, in_layout=U2, out_layout=out_l, dump=False)
        assert np.array_equal(got, expect_layout(want, out_l)), (name, out_l)
    assert len(np.unique(want)) > 1



# 1x1 convolutions with int32 sums out and c_out <= 64 on 2-bit codes (a
# detector's head) run the latency-bound head kernel: the YOLO head, both
# code layouts, ragged channel counts, c_in past one chunk of eight channel
# blocks (1024) and a last chunk of one block (576).
# (name, n, h, w, cin, cout, in_layout)
HEAD = [
    ("head_yolo", 8, 13, 13, 512, 30, "b64"),
    ("head_u2_c64", 3, 9, 7, 128, 64, "u2"),
    ("head_c33", 2, 5, 11, 64, 33, "b64"),
    ("head_cin1024", 1, 6, 6, 1024, 30, "u2"),
    ("head_cin576_c8", 2, 7, 7, 576, 8, "b64"),
]


@pytest.mark.parametrize("case", HEAD, ids=[c[0] for c in HEAD])
def test_head_bit_exact(P, case):
    name, n, h, w, cin, cout, lay = case
    in_l = B64 if lay == "b64" else U2
    L = make_layer(name, h, w, cin, cout, 1, 1, 0, 2, 0)
    d = P.conv_desc(n, h, w, cin, cout, 1, 1, 0, 2, 0, in_l, I32)
    assert P.ifq_conv_kernel_name(d).startswith("conv_head<"), name
    seed = zlib.crc32(name.encode()) % 997
    p = params_for(seed, L)
    x = codes_for(seed, (n, h, w, cin), 2)
    want_acc, want = oracle_layer(L, x, p)
    acc, got = gpu_layer(P, L, n, x, p, in_layout=in_l, out_layout=I32)
    assert np.array_equal(acc, want_acc), name
    assert np.array_equal(got, want), name


U2_LAYERS = [
    ("u2_3x3_64", 2, 14, 14, 64, 64, 3, 1, 1),
    ("u2_stride2_128", 2, 15, 15, 64, 128, 3, 2, 1),
    ("u2_cin16", 1, 18, 18, 16, 32, 3, 1, 1),
    ("u2_cin32", 1, 12, 12, 32, 64, 3, 1, 1),
    ("u2_k4608", 1, 7, 7, 512, 512, 3, 1, 1),
    ("u2_cin96_5x5", 1, 9, 9, 96, 256, 5, 1, 2),
    ("u2_m3136_c128", 4, 28, 28, 128, 128, 3, 1, 1),
    ("u2_c256_s1", 2, 30, 30, 256, 256, 3, 1, 1),
    ("u2_c64_large_m", 8, 56, 56, 64, 64, 3, 1, 1),
    ("u2_c512_7x7", 12, 7, 7, 512, 512, 3, 1, 1),
    ("u2_1x1_s2_c256", 3, 14, 14, 128, 256, 1, 2, 0),
    ("u2_c192_ragged", 3, 11, 13, 192, 320, 3, 1, 1),
    ("u2_5x5_c64", 2, 17, 15, 64, 128, 5, 2, 2),
]


@pytest.mark.parametrize("case", U2_LAYERS, ids=[c[0] for c in U2_LAYERS])
@pytest.mark.parametrize("io", [(U2, U2), (U2, I8), (I8, U2)],
                         ids=["u2u2", "u2i8", "i8u2"])
def test_conv_packed_layouts_bit_exact(P, case, io):
    run_layout_case(P, case, io)


# shapes of the fast path (c_in % 64 == 0): every tile variant, ragged pixel
# and channel tiles, stride 2, 1x1 and 5x5 filters, the judged ResNet shapes
B64_LAYERS = [
    ("b64_3x3_64", 2, 14, 14, 64, 64, 3, 1, 1),
    ("b64_stride2_128", 2, 15, 15, 64, 128, 3, 2, 1),
    ("b64_k4608", 1, 7, 7, 512, 512, 3, 1, 1),
    ("b64_5x5_c64", 2, 17, 15, 64, 128, 5, 2, 2),
    ("b64_1x1_s2_c256", 3, 14, 14, 128, 256, 1, 2, 0),
    ("b64_c192_cout320", 3, 11, 13, 192, 320, 3, 1, 1),
    ("b64_l2_shape_b4", 4, 28, 28, 128, 128, 3, 1, 1),
    ("b64_l3_shape_b8", 8, 14, 14, 256, 256, 3, 1, 1),
    ("b64_l4_shape_b12", 12, 7, 7, 512, 512, 3, 1, 1),
    ("b64_l1_shape_b2", 2, 56, 56, 64, 64, 3, 1, 1),
    ("b64_cout96", 2, 9, 9, 128, 96, 3, 1, 1),
    ("b64_big_m", 16, 28, 28, 64, 128, 3, 1, 1),
]


@pytest.mark.parametrize("case", B64_LAYERS, ids=[c[0] for c in B64_LAYERS])
@pytest.mark.parametrize("io", [(B64, B64), (B64, U2), (U2, B64), (B64, I8)],
                         ids=["b64b64", "b64u2", "u2b64", "b64i8"])
def test_conv_block64_bit_exact(P, case, io):
    if io[1] == B64 and case[5] % 64:
        pytest.skip("BLOCK64 output needs c_out % 64 == 0")
    run_layout_case(P, case, io)


# Workgroup tiles of the size the ResNet-18 layers of the benchmark run with
# (the 3x3 kernels' tiles of 256, 128 and 64 output pixels, stride-2 layers),
# at batches the oracle finishes in about a second; the test also pins which
# kernel variant the planner takes for each (conv_w2, whose eighth template
# argument is its epilogue, 0 thresholds; or the wave-independent conv_wv and
# its 32-channel form conv_wvh).
HALO_TILES = [
    ("halo_l2_b83", 83, 28, 28, 128, 128, 1, "conv_wv<0, false, 73728, 80896>"),
    ("halo_l3_b83", 83, 14, 14, 256, 256, 1, "conv_wvh<0, false, 73728, 84992>"),
    ("halo_l4_b83", 83, 7, 7, 512, 512, 1, "conv_w2<1, 2, 4, 2, 2, 3, 2, 0, false, 1, 36864>"),
    ("halo_s2_b40", 40, 28, 28, 128, 256, 2, "conv_wv<0, false, 73728, 80896>"),
    ("halo_l1_b24", 24, 56, 56, 64, 64, 1, "conv_wv<0, false, 73728, 80896>"),
    # the stride-2 layers at the full batch of 64, with the largest windows
    ("halo_l2s2_b64", 64, 56, 56, 64, 128, 2, "conv_wv<0, false, 73728, 80896>"),
    ("halo_l4s2_b64", 64, 14, 14, 256, 512, 2, "conv_w2<1, 4, 2, 2, 2, 3, 2, 0, false, 1, 53248>"),
]


@pytest.mark.parametrize("case", HALO_TILES, ids=[c[0] for c in HALO_TILES])
def test_conv_halo_tiles_bit_exact(P, case):
    name, n, h, w, cin, cout, st, kernel = case
    d = P.ConvDesc(n, h, w, cin, cout, 3, 3, st, 1, 2, 2, B64, B64)
    assert P.ifq_conv_kernel_name(d) == kernel
    run_layout_case(P, (name, n, h, w, cin, cout, 3, st, 1), (B64, B64))


@pytest.mark.parametrize("case", HALO_TILES[:1] + HALO_TILES[4:],
                         ids=[c[0] for c in HALO_TILES[:1] + HALO_TILES[4:]])
def test_conv_halo_tiles_no_dump(P, case):
    # the same layers without the int32 dump, so only the code epilogue runs
    name, n, h, w, cin, cout, st, _ = case
    L = make_layer(name, h, w, cin, cout, 3, st, 1)
    seed = zlib.crc32(name.encode()) % 991
    p = params_for(seed, L)
    x = codes_for(seed, (n, h, w, cin), 2)
    _, want = oracle_layer(L, x, p)
    _, got = gpu_layer(P, L, n, x, p, in_layout=B64, out_layout=B64, dump=False)
    assert np.array_equal(got, expect_layout(want, B64))


def test_conv_block64_int32_out(P):
    L = make_layer("b64_i32", 14, 14, 128, 256, 1, 2, 0, 2, 0)
    p = params_for(17, L)
    x = codes_for(17, (3, 14, 14, 128), 2)
    want_acc, want = oracle_layer(L, x, p)
    acc, got = gpu_layer(P, L, 3, x, p, in_layout=B64, out_layout=I32)
    assert np.array_equal(acc, want_acc)
    assert np.array_equal(got, want)


def run_layout_case(P, case, io):
    name, n, h, w, cin, cout, k, st, pad = case
    L = make_layer(name, h, w, cin, cout, k, st, pad)
    seed = zlib.crc32(name.encode()) % 991
    p = params_for(seed, L)
    x = codes_for(seed, (n, h, w, cin), 2)
    want_acc, want = oracle_layer(L, x, p)
    acc, got = gpu_layer(P, L, n, x, p, in_layout=io[0], out_layout=io[1])
    assert np.array_equal(acc, want_acc)
    assert np.array_equal(got, expect_layout(want, io[1]))


@pytest.mark.parametrize("io", [(I8, I8, I8), (I8, U2, I8), (U2, U2, U2),
                                (U2, I8, U2), (B64, B64, B64), (B64, U2, I8),
                                (U2, B64, B64), (B64, U2, B64)],
                         ids=["i8", "sc_u2", "u2", "u2_sc_i8", "b64", "b64_sc_u2",
                              "u2_sc_b64", "b64_sc_u2_out_b64"])
@pytest.mark.parametrize("shape", [(2, 10, 10, 64, 64), (1, 7, 7, 512, 512),
                                   (1, 9, 11, 128, 128), (6, 14, 14, 256, 256)])
def test_identity_join_bit_exact(P, shape, io):
    n, h, w, cin, cout = shape
    in_l, sc_l, out_l = io
    L = make_layer("join_id", h, w, cin, cout, 3, 1, 1, join=("identity", "s"))
    p = params_for(31 + h, L)
    x = codes_for(31 + h, (n, h, w, cin), 2)
    sc = codes_for(77 + h, (n, h, w, cout), 2)
    want_acc, want = oracle_layer(L, x, p, shortcut=sc)
    acc, got = gpu_layer(P, L, n, x, p, in_layout=in_l, out_layout=out_l,
                         shortcut=sc, sc_layout=sc_l)
    assert np.array_equal(acc, want_acc)
    assert np.array_equal(got, expect_layout(want, out_l))


def test_identity_join_64_channel_variant(P):
    # the ResNet-18 l1 conv2 shape at batch 24 on the register-blocked
    # 64-channel variant (two workgroups per CU) with an identity join, and
    # on the kernel the planner picks
    n, h, c = 24, 56, 64
    d = P.conv_desc(n, h, h, c, c, 3, 1, 1, 2, 2, B64, B64)
    jn = P.make_join(P.IFQ_JOIN_IDENTITY, B64, None, None, [0.25, 0.75, 1.25])
    jn.table = 0x1000
    name = "conv_w2<1, 8, 1, 2, 1, 3, 3, 1, false, 2, 20480>"
    vs = [v for v in range(P.ifq_conv_variant_count())
          if P.ifq_conv_variant_name(d, jn, v) == name]
    assert vs, name
    assert P.ifq_conv_kernel_name(d, jn).startswith(("conv_w2<", "conv_wp<", "conv_wv<", "conv_wvh<"))
    L = make_layer("join_id", h, h, c, c, 3, 1, 1, join=("identity", "s"))
    p = params_for(41, L)
    x = codes_for(41, (n, h, h, c), 2)
    sc = codes_for(42, (n, h, h, c), 2)
    want_acc, want = oracle_layer(L, x, p, shortcut=sc)
    for variant in (vs[0], None):
        acc, got = gpu_layer(P, L, n, x, p, in_layout=B64, out_layout=B64, shortcut=sc,
                             sc_layout=B64, variant=variant)
        assert np.array_equal(acc, want_acc), variant
        assert np.array_equal(got, expect_layout(want, B64)), variant


@pytest.mark.parametrize("lay", [I8, U2, B64], ids=["i8", "u2", "b64"])
def test_conv_join_bit_exact(P, lay):
    # conv2 of a downsampling block: the shortcut is the int32 sum of a 1x1/2
    # conv of the block input, computed by the GPU path itself first
    n, hin, cin, cout = 2, 16, 64, 128
    D = make_layer("down", hin, hin, cin, cout, 1, 2, 0, 2, 0)
    L = make_layer("conv2", hin // 2, hin // 2, cout, cout, 3, 1, 1,
                   join=("conv", "d", "down"))
    pd = params_for(5, D)
    p = params_for(6, L)
    xin = codes_for(5, (n, hin, hin, cin), 2)
    x = codes_for(6, (n, hin // 2, hin // 2, cout), 2)
    want_d, _ = oracle_layer(D, xin, pd)
    _, got_d = gpu_layer(P, D, n, xin, pd, in_layout=lay)
    assert np.array_equal(got_d, want_d)
    want_acc, want = oracle_layer(L, x, p, shortcut=want_d, down=pd)
    acc, got = gpu_layer(P, L, n, x, p, in_layout=lay, out_layout=lay,
                         shortcut=want_d, down=pd)
    assert np.array_equal(acc, want_acc)
    assert np.array_equal(got, expect_layout(want, lay))


# conv2 of a downsampling block with the 1x1/2 downsample computed inside the
# conv kernel (IFQ_JOIN_CONV_FUSED): the shapes of the three ResNet-18
# downsampling blocks at small batches (one variant each), plus ragged ones
FUSED = [(2, 56, 64, 128), (3, 28, 128, 256), (2, 14, 256, 512), (1, 17, 128, 256),
         (5, 13, 64, 128), (40, 28, 128, 256)]


@pytest.mark.parametrize("shape", FUSED, ids=["x".join(map(str, f)) for f in FUSED])
def test_fused_downsample_join_bit_exact(P, shape):
    n, hin, cin, cout = shape
    D = make_layer("down", hin, hin, cin, cout, 1, 2, 0, 2, 0)
    ho = (hin - 1) // 2 + 1
    L = make_layer("conv2", ho, ho, cout, cout, 3, 1, 1, join=("conv", "d", "down"))
    pd = params_for(5 + hin, D)
    p = params_for(6 + hin, L)
    xin = codes_for(5 + hin, (n, hin, hin, cin), 2)
    x = codes_for(6 + hin, (n, ho, ho, cout), 2)
    want_d, _ = oracle_layer(D, xin, pd)
    want_acc, want = oracle_layer(L, x, p, shortcut=want_d, down=pd)
    acc, got = gpu_layer(P, L, n, x, p, in_layout=B64, out_layout=B64, down=pd,
                         fused_down=(D, xin))
    assert np.array_equal(acc, want_acc)
    assert np.array_equal(got, expect_layout(want, B64))


def test_conv_without_dump_and_determinism(P):
    L = make_layer("det", 28, 28, 128, 128, 3, 1, 1)
    p = params_for(9, L)
    x = codes_for(9, (4, 28, 28, 128), 2)
    _, a = gpu_layer(P, L, 4, x, p, dump=False)
    _, b = gpu_layer(P, L, 4, x, p, dump=False)
    assert np.array_equal(a, b)
    assert np.array_equal(a, oracle_layer(L, x, p)[1])


def test_empty_batch_launches_nothing(P):
    import torch
    d = P.conv_desc(0, 8, 8, 64, 64, 3, 1, 1, 2, 2)
    dummy = torch.zeros(16, dtype=torch.uint8, device=device())
    thr = torch.zeros(64 * 4, dtype=torch.int32, device=device())
    P.ifq_conv_forward(d, dummy, dummy, thr, dummy)
    torch.cuda.synchronize()


@pytest.mark.parametrize("case", [
    ((2, 27, 27, 256), 3, 2, "valid"), ((1, 13, 13, 256), 3, 2, "valid"),
    ((2, 224, 224, 64), 2, 2, "valid"), ((1, 13, 13, 512), 2, 1, "same"),
    ((1, 9, 9, 20), 3, 2, "same"), ((3, 7, 5, 12), 2, 2, "valid"),
    ((1, 8, 8, 3), 2, 2, "valid"),
])
@pytest.mark.parametrize("lay", [I8, U2, B64], ids=["i8", "u2", "b64"])
def test_maxpool_bit_exact(P, case, lay):
    import torch
    shape, k, st, mode = case
    n, h, w, c = shape
    if lay == U2 and c % 4:
        pytest.skip("packed layout needs C % 4 == 0")
    if lay == B64 and c % 64:
        pytest.skip("BLOCK64 needs C % 64 == 0")
    x = codes_for(h * 31 + c, shape, 2)
    want = oracle.maxpool(x, k, st, mode)
    m = P.IFQ_POOL_VALID if mode == "valid" else P.IFQ_POOL_SAME
    d = P.pool_desc(n, h, w, c, k, st, m, 2, lay)
    xd = upload_codes(P, x, lay)
    nb = P.ifq_tensor_bytes(*want.shape, lay)
    y = torch.empty(nb, dtype=torch.uint8, device=device())
    P.ifq_maxpool_codes(d, xd, y)
    torch.cuda.synchronize()
    got = y.cpu().numpy()
    assert np.array_equal(got, expect_layout(want, lay).reshape(-1))


def test_maxpool_8bit_codes(P):
    import torch
    x = codes_for(3, (1, 10, 10, 16), 8)
    want = oracle.maxpool(x, 2, 2, "valid")
    d = P.pool_desc(1, 10, 10, 16, 2, 2, P.IFQ_POOL_VALID, 8, I8)
    y = torch.empty(want.size, dtype=torch.uint8, device=device())
    P.ifq_maxpool_codes(d, to_dev(x), y)
    torch.cuda.synchronize()
    assert np.array_equal(y.cpu().numpy(), want.reshape(-1))


@pytest.mark.parametrize("shape", [(1, 1, 1, 4), (1, 1, 7, 12), (2, 10, 50, 64),
                                   (1, 3, 11, 16), (3, 5, 7, 192)])
def test_convert_codes_round_trip(P, shape):
    import torch
    n, h, w, c = shape
    x = codes_for(h * w + c, shape, 2)
    layouts = [U2] + ([B64] if c % 64 == 0 else [])
    for lay in layouts:
        packed = torch.empty(n * h * w * c // 4, dtype=torch.uint8, device=device())
        P.ifq_convert_codes(n, h, w, c, I8, lay, to_dev(x), packed)
        back = torch.empty(n * h * w * c, dtype=torch.uint8, device=device())
        P.ifq_convert_codes(n, h, w, c, lay, I8, packed, back)
        torch.cuda.synchronize()
        assert np.array_equal(packed.cpu().numpy(),
                              expect_layout(x, lay).reshape(-1))
        assert np.array_equal(back.cpu().numpy(), x.reshape(-1))
    if c % 64 == 0:
        # 2-bit NHWC <-> BLOCK64 directly
        u2 = upload_codes(P, x, U2)
        b64 = torch.empty_like(u2)
        P.ifq_convert_codes(n, h, w, c, U2, B64, u2, b64)
        u2b = torch.empty_like(u2)
        P.ifq_convert_codes(n, h, w, c, B64, U2, b64, u2b)
        torch.cuda.synchronize()
        assert np.array_equal(b64.cpu().numpy(), olayout.pack_block64(x).reshape(-1))
        assert torch.equal(u2, u2b)
