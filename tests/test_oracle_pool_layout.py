"""Pins of the oracle's max-pool on codes (Eq. 4) and the 2-bit code layout."""
import json
import os

import numpy as np
import pytest

import oracle
from oracle import brute, layout
from workloads import get_stack, layer_params

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.mark.parametrize("shape,k,st,mode", [
    ((2, 7, 7, 5), 3, 2, "valid"),
    ((1, 8, 6, 3), 2, 2, "valid"),
    ((1, 5, 5, 4), 2, 1, "same"),
    ((1, 6, 7, 2), 2, 1, "same"),
    ((2, 9, 9, 3), 3, 2, "same"),
    ((1, 13, 13, 2), 3, 2, "valid"),
    ((1, 4, 4, 1), 1, 1, "valid"),
])
def test_maxpool_matches_brute_force(shape, k, st, mode, rng):
    x = rng.integers(0, 4, size=shape, dtype=np.uint8)
    got = oracle.maxpool(x, k, st, mode)
    want = np.array(brute.maxpool(x.tolist(), k, st, mode), dtype=np.uint8)
    assert np.array_equal(got, want)


def test_maxpool_output_sizes_of_the_stacks():
    # AlexNet 27->13->6 (3/2), VGG/YOLO halving (2/2), YOLO 13->13 (2/1 same)
    for h, k, st, mode, want in [(27, 3, 2, "valid", 13), (13, 3, 2, "valid", 6),
                                 (224, 2, 2, "valid", 112), (13, 2, 1, "same", 13),
                                 (26, 2, 2, "valid", 13)]:
        y = oracle.maxpool(np.zeros((1, h, h, 1), np.uint8), k, st, mode)
        assert y.shape[1] == want


def test_maxpool_commutes_with_monotone_codes(rng):
    # for channels with s = +1 the code map is non-decreasing, so pooling the
    # int32 sums then quantizing equals quantizing then pooling the codes
    L = get_stack(0).layers[0]
    p = layer_params(0, 0, L, "calibrated")
    s, t = oracle.fold(p["alpha"], p["beta_in"], p["mean"], p["var"],
                       p["gamma"], p["bn_beta"], p["eps"], p["q_thr"], 576, 2)
    acc = rng.integers(-400, 400, size=(2, 8, 8, L.cout)).astype(np.int32)
    pooled_acc = acc.reshape(2, 4, 2, 4, 2, L.cout).max(axis=(2, 4))
    a = oracle.codes(np.ascontiguousarray(pooled_acc), s, t)
    b = oracle.maxpool(oracle.codes(acc, s, t), 2, 2, "valid")
    pos = s > 0
    assert np.array_equal(a[..., pos], b[..., pos])
    # for s = -1 the paper's order (pool before BN) would give the minimum code
    neg = s < 0
    pooled_min = acc.reshape(2, 4, 2, 4, 2, L.cout).min(axis=(2, 4))
    c = oracle.codes(np.ascontiguousarray(pooled_min), s, t)
    assert np.array_equal(c[..., neg], b[..., neg])


def test_pack2_round_trip(rng):
    codes = rng.integers(0, 4, size=(2, 5, 3, 16), dtype=np.uint8)
    packed = layout.pack2(codes)
    assert packed.shape == (2, 5, 3, 4)
    assert np.array_equal(layout.unpack2(packed, 16), codes)
    # channel c sits in bits 2*(c%4) of byte c//4
    one = np.zeros((1, 1, 1, 8), np.uint8)
    one[..., 6] = 3
    assert layout.pack2(one).tolist() == [[[[0, 3 << 4]]]]


def test_feature_map_memory_matches_table4():
    g = json.load(open(os.path.join(GOLDEN, "table4_feature_map_memory.json")))
    mbit = {}
    for e in g["entries"]:
        bits = layout.tensor_bits((e["h"], e["w"], e["c"]), e["bits"])
        mbit[e["name"]] = bits / 1e6
        # within one unit of the last printed digit
        assert abs(bits / 1e6 - e["mbit_printed"]) <= 0.1 + 1e-12, e
    # the 2-bit tensor of conv1 is 72,600 bytes
    assert layout.tensor_bits((55, 55, 96), 2) // 8 == 72600
    assert layout.pack2(np.zeros((55, 55, 96), np.uint8)).nbytes == 72600
    for r in g["savings_printed"]:
        # the printed ratios are those of the printed values
        num = [e for e in g["entries"] if e["name"] == r["num"]][0]["mbit_printed"]
        den = [e for e in g["entries"] if e["name"] == r["den"]][0]["mbit_printed"]
        assert round(num / den, 1) == r["ratio"]


def test_alexnet_parameter_count_supports_dense_convs():
    g = json.load(open(os.path.join(GOLDEN, "alexnet_parameter_count.json")))
    total = sum(L["cout"] * L["cin"] * L["k"] ** 2 for L in g["layers"])
    assert round(total / 1e6, 1) == g["million_params_printed"]
    # the AlexNet-shaped stack's conv2..conv5 have exactly these shapes
    convs = [L for L in get_stack(1).layers if hasattr(L, "cin")]
    shapes = [(L.cout, L.cin, L.k) for L in convs]
    want = [(L["cout"], L["cin"], L["k"]) for L in g["layers"][1:5]]
    assert shapes == want


@pytest.mark.parametrize("shape", [(2, 3, 5, 128), (1, 4, 2, 64), (3, 2, 3, 192)])
def test_pack_block64_places_every_code_by_the_layout_formula(shape):
    # IFQ_LAYOUT_U2_BLOCK64 (the k-bit feature maps of Table 4 at 2 bits,
    # regrouped in 64-channel blocks): code (n, y, x, c) sits in byte
    # (((n*C/64 + c/64)*H + y)*W + x)*16 + (c%64)/4, bits 2*(c%4) .. +1.
    # Every position is checked from that formula with explicit loops, on
    # codes that differ between any two axes, so a swapped axis of the
    # packer's transpose fails.
    n, h, w, c = shape
    idx = np.indices(shape)
    codes = ((idx[0] * 7 + idx[1] * 5 + idx[2] * 3 + idx[3] + idx[3] // 64) % 4).astype(np.uint8)
    flat = layout.pack_block64(codes).reshape(-1)
    assert flat.size == n * h * w * c // 4
    for ni in range(n):
        for y in range(h):
            for x in range(w):
                for ch in range(c):
                    byte = (((ni * (c // 64) + ch // 64) * h + y) * w + x) * 16 + (ch % 64) // 4
                    got = (int(flat[byte]) >> (2 * (ch % 4))) & 3
                    assert got == codes[ni, y, x, ch], (ni, y, x, ch)


def test_pack_block64_one_hot_cells():
    # a single nonzero code lands in exactly one byte, at the formula's place
    n, h, w, c = 2, 3, 4, 128
    for (ni, y, x, ch) in [(0, 0, 0, 0), (1, 2, 3, 127), (0, 1, 2, 64), (1, 0, 3, 5),
                           (0, 2, 0, 70)]:
        codes = np.zeros((n, h, w, c), np.uint8)
        codes[ni, y, x, ch] = 2
        flat = layout.pack_block64(codes).reshape(-1)
        byte = (((ni * (c // 64) + ch // 64) * h + y) * w + x) * 16 + (ch % 64) // 4
        assert np.flatnonzero(flat).tolist() == [byte]
        assert flat[byte] == 2 << (2 * (ch % 4))


def test_block64_round_trip(rng):
    codes = rng.integers(0, 4, size=(2, 3, 5, 192), dtype=np.uint8)
    packed = layout.pack_block64(codes)
    assert packed.shape == (2, 3, 3, 5, 16)
    assert np.array_equal(layout.unpack_block64(packed, 192), codes)
