"""GPU parity of the fused conv + max-pool (ifq_conv_pool_forward): the
pooled codes must equal the oracle's conv -> thresholds -> max-pool on codes
(Eq. 1, Eq. 7-8, Eq. 4) bit for bit, for the two kernels that fuse the pool
(the small-channel 8-bit first layer, the small-channel 2-bit kernel for
c_in 16 and 32, and the windowed 3x3 kernel on BLOCK64 input), every code layout they write, pool sizes 2..4, tiles that span
images, and channels with a negative BN scale (the calibrated parameters
flip about a tenth of them)."""
import zlib

import numpy as np
import pytest

import oracle
from gpu_util import (I8, U2, B64, oracle_layer, expect_layout, make_layer, params_for,
                      codes_for, upload_codes, to_dev, device)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1911_08076_amd as P
    return P


def gpu_conv_pool(P, L, n, x, p, k, in_layout, out_layout, st=None, mode="valid"):
    import torch
    d = P.conv_desc(n, L.h, L.w, L.cin, L.cout, L.k, L.stride, L.pad,
                    L.in_bits, L.out_bits, in_layout, out_layout)
    ho, wo = P.ifq_conv_output_dims(d)
    st = k if st is None else st
    pm = P.IFQ_POOL_VALID if mode == "valid" else P.IFQ_POOL_SAME
    pd = P.pool_desc(n, ho, wo, L.cout, k, st, pm, L.out_bits, out_layout)
    name = P.ifq_conv_pool_kernel_name(d, pd)
    wd = to_dev(P.ifq_pack_weights(d, p["w"]))
    thr = P.ifq_fold_thresholds(L.cout, L.in_bits, L.out_bits, L.k * L.k * L.cin,
                                p["alpha"], p["beta_in"], p["q_thr"], bias=p["bias"],
                                mean=p["mean"], var=p["var"], gamma=p["gamma"],
                                bn_beta=p["bn_beta"], eps=p["eps"])
    td = to_dev(thr)
    xd = upload_codes(P, x, in_layout)
    if mode == "valid":
        pho, pwo = (ho - k) // st + 1, (wo - k) // st + 1
    else:
        pho, pwo = -(-ho // st), -(-wo // st)
    ob = P.ifq_tensor_bytes(n, pho, pwo, L.cout, out_layout)
    # poisoned output: every byte the kernel leaves alone shows up
    y = torch.full((ob,), 0xA5, dtype=torch.uint8, device=device())
    P.ifq_conv_pool_forward(d, pd, xd, wd, td, y)
    torch.cuda.synchronize()
    out = y.cpu().numpy()
    if out_layout == U2:
        out = out.reshape(n, pho, pwo, L.cout // 4)
    elif out_layout == B64:
        out = out.reshape(n, L.cout // 64, pho, pwo, 16)
    else:
        out = out.reshape(n, pho, pwo, L.cout)
    return name, out


def check(P, name, L, n, k, in_layout, outs, family, st=None, mode="valid"):
    seed = zlib.crc32(name.encode()) % 997
    p = params_for(seed, L)
    x = codes_for(seed, (n, L.h, L.w, L.cin), L.in_bits)
    _, codes = oracle_layer(L, x, p)
    want = oracle.maxpool(codes, k, k if st is None else st, mode)
    assert len(np.unique(want)) > 1
    for out_l in outs:
        kname, got = gpu_conv_pool(P, L, n, x, p, k, in_layout, out_l, st, mode)
        assert kname.startswith(family), (name, out_l, kname)
        assert np.array_equal(got, expect_layout(want, out_l)), (name, out_l, kname)


# name, n, h, w, c_in, c_out, pool k
SMALL8_POOL = [
    ("s8p_yolo_c1", 2, 416, 416, 3, 16, 2),
    ("s8p_c32_ragged_rows", 3, 50, 38, 3, 32, 2),
    ("s8p_c64_cin4", 1, 36, 44, 4, 64, 2),
    ("s8p_pool3", 2, 39, 45, 3, 16, 3),
    # 4 rows per workgroup with a last tile of 2, and a ragged last group of
    # pooled columns (pwo = 11) in the register pool
    ("s8p_rows4_ragged_tile", 8, 290, 22, 3, 16, 2),
]


@pytest.mark.parametrize("case", SMALL8_POOL, ids=[c[0] for c in SMALL8_POOL])
def test_small8_conv_pool_bit_exact(P, case):
    name, n, h, w, cin, cout, k = case
    L = make_layer(name, h, w, cin, cout, 3, 1, 1, 8, 2)
    check(P, name, L, n, k, I8, [I8, U2], "conv_small8<")



# name, n, h, w, c_in, c_out, pool k, output layouts
SMALL2_POOL = [
    ("s2p_yolo_c2", 2, 208, 208, 16, 32, 2, [U2]),
    ("s2p_yolo_c3", 2, 104, 104, 32, 64, 2, [B64, U2]),
    ("s2p_c48_ragged_rows", 3, 37, 29, 16, 48, 2, [U2]),
    ("s2p_pool3_c16", 2, 33, 27, 32, 16, 3, [U2]),
    ("s2p_pool4_c64", 1, 40, 44, 16, 64, 4, [B64]),
    # the register pool (2x2/2, c_out <= 32): a ragged last group of pooled
    # columns, and 4 rows per workgroup with a last tile of 2
    ("s2p_rp_c16_cin32_ragged", 3, 38, 42, 32, 16, 2, [U2]),
    ("s2p_rp_rows4_ragged_tile", 8, 290, 14, 16, 32, 2, [U2]),
]


@pytest.mark.parametrize("case", SMALL2_POOL, ids=[c[0] for c in SMALL2_POOL])
def test_small2_conv_pool_bit_exact(P, case):
    name, n, h, w, cin, cout, k, outs = case
    L = make_layer(name, h, w, cin, cout, 3, 1, 1, 2, 2)
    check(P, name, L, n, k, U2, outs, "conv_small2<")


# name, n, h, w, c_in, c_out, pool k, output layouts
HALO_POOL = [
    ("hp_yolo_c4", 2, 52, 52, 64, 128, 2, [B64, U2, I8]),
    ("hp_yolo_c5", 2, 26, 26, 128, 256, 2, [B64]),
    ("hp_vgg_conv2_2", 1, 112, 112, 128, 128, 2, [B64]),
    ("hp_vgg_conv4_3", 2, 28, 28, 512, 512, 2, [B64, U2]),
    ("hp_vgg_conv5_3_spans_images", 3, 14, 14, 512, 512, 2, [B64]),
    ("hp_c64_out64", 4, 56, 56, 64, 64, 2, [B64, I8]),
    ("hp_pool4", 2, 24, 24, 128, 128, 4, [B64]),
]


@pytest.mark.parametrize("case", HALO_POOL, ids=[c[0] for c in HALO_POOL])
def test_halo_conv_pool_bit_exact(P, case):
    name, n, h, w, cin, cout, k, outs = case
    L = make_layer(name, h, w, cin, cout, 3, 1, 1, 2, 2)
    check(P, name, L, n, k, B64, outs, "conv_halo<")


# windows that overlap, run in SAME mode or do not tile the output: each tile
# holds whole images (name, n, h, c_in, c_out, k, stride, mode, layouts)
WHOLE_IMAGE = [
    ("hp_alexnet_conv5_pool3s2", 3, 13, 384, 256, 3, 2, "valid", [B64, U2]),
    ("hp_yolo_c6_pool2s1_same", 2, 13, 256, 512, 2, 1, "same", [B64]),
    ("hp_odd_size_pool2", 2, 13, 128, 128, 2, 2, "valid", [B64, I8]),
    ("hp_pool3s3_same", 4, 10, 64, 128, 3, 3, "same", [B64]),
]


@pytest.mark.parametrize("case", WHOLE_IMAGE, ids=[c[0] for c in WHOLE_IMAGE])
def test_halo_conv_pool_whole_images(P, case):
    name, n, h, cin, cout, k, st, mode, outs = case
    L = make_layer(name, h, h, cin, cout, 3, 1, 1, 2, 2)
    check(P, name, L, n, k, B64, outs, "conv_halo<", st, mode)


def test_small8_conv_pool_whole_images(P):
    L = make_layer("s8p_pool3s2", 31, 29, 3, 16, 3, 1, 1, 8, 2)
    check(P, "s8p_pool3s2", L, 2, 3, I8, [I8, U2], "conv_small8<", 2, "valid")


def test_small2_conv_pool_whole_images(P):
    # overlapping 3/2 windows and a SAME pool: each workgroup holds whole images
    L = make_layer("s2p_pool3s2", 31, 29, 32, 32, 3, 1, 1, 2, 2)
    check(P, "s2p_pool3s2", L, 2, 3, U2, [U2], "conv_small2<", 2, "valid")
    L = make_layer("s2p_pool2s1_same", 13, 13, 16, 64, 3, 1, 1, 2, 2)
    check(P, "s2p_pool2s1_same", L, 3, 2, U2, [B64, U2], "conv_small2<", 1, "same")
