"""Pins of the oracle's integer convolution (the integer part of Eq. 1)."""
import itertools

import numpy as np
import pytest
import torch

import oracle
from oracle import brute


def _rand_layer(rng, n, h, w, cin, cout, k, in_bits):
    x = rng.integers(0, 1 << in_bits, size=(n, h, w, cin), dtype=np.uint8)
    wt = (rng.integers(0, 2, size=(cout, cin, k, k)) * 2 - 1).astype(np.int8)
    return x, wt


CASES = [
    # (n, h, w, cin, cout, k, stride, pad, in_bits)
    (1, 5, 6, 3, 2, 3, 1, 1, 2),
    (2, 7, 5, 4, 3, 3, 2, 1, 2),
    (1, 6, 6, 2, 4, 5, 1, 2, 2),
    (1, 9, 7, 5, 2, 5, 2, 2, 2),
    (2, 4, 4, 8, 8, 1, 1, 0, 2),
    (1, 7, 7, 6, 5, 1, 2, 0, 2),
    (1, 6, 5, 3, 4, 3, 1, 1, 8),
    (1, 8, 8, 3, 2, 3, 2, 0, 8),
    (1, 5, 5, 1, 1, 3, 1, 0, 2),
    (1, 4, 6, 7, 3, 3, 1, 2, 2),
]


@pytest.mark.parametrize("case", CASES)
def test_acc_matches_brute_force(case, rng):
    n, h, w, cin, cout, k, st, pad, bits = case
    x, wt = _rand_layer(rng, n, h, w, cin, cout, k, bits)
    got = oracle.conv_acc(x, wt, st, pad, bits)
    want = np.array(brute.conv_acc(x.tolist(), wt.tolist(), st, pad), dtype=np.int64)
    assert got.shape == want.shape
    assert np.array_equal(got.astype(np.int64), want)


@pytest.mark.parametrize("case", [
    (2, 13, 11, 16, 24, 3, 1, 1, 2),
    (1, 14, 14, 32, 16, 3, 2, 1, 2),
    (2, 9, 9, 24, 8, 5, 1, 2, 2),
    (1, 10, 12, 64, 32, 1, 2, 0, 2),
    (1, 20, 20, 3, 16, 3, 1, 1, 8),
])
def test_acc_matches_float64_conv2d(case, rng):
    # integer-valued float64 tensors: every partial sum is an exact integer
    # far below 2^53, so torch's conv2d must agree exactly
    n, h, w, cin, cout, k, st, pad, bits = case
    x, wt = _rand_layer(rng, n, h, w, cin, cout, k, bits)
    got = oracle.conv_acc(x, wt, st, pad, bits)
    xt = torch.from_numpy(x.astype(np.float64)).permute(0, 3, 1, 2)
    wtt = torch.from_numpy(wt.astype(np.float64))
    want = torch.nn.functional.conv2d(xt, wtt, stride=st, padding=pad)
    want = want.permute(0, 2, 3, 1).numpy()
    assert np.array_equal(got.astype(np.float64), want)


@pytest.mark.parametrize("k,pad,c", [(3, 1, 2), (5, 2, 3), (3, 0, 1), (1, 0, 3)])
def test_acc_closed_form_constant_codes(k, pad, c):
    # all +1 weights on a constant code c: acc = c * Cin * (#taps inside)
    n, h, w, cin, cout = 1, 7, 6, 5, 2
    x = np.full((n, h, w, cin), c, dtype=np.uint8)
    wt = np.ones((cout, cin, k, k), dtype=np.int8)
    acc = oracle.conv_acc(x, wt, 1, pad, 2)
    ho, wo = acc.shape[1:3]
    for oy in range(ho):
        for ox in range(wo):
            rows = sum(1 for i in range(k) if 0 <= oy - pad + i < h)
            cols = sum(1 for j in range(k) if 0 <= ox - pad + j < w)
            assert (acc[0, oy, ox] == c * cin * rows * cols).all()
    # interior value is K * c with K = k*k*Cin
    if ho > 2 * pad and wo > 2 * pad:
        assert acc[0, pad, pad, 0] == k * k * cin * c


def test_acc_closed_form_1x1_single_channel(rng):
    x = rng.integers(0, 4, size=(2, 5, 5, 1), dtype=np.uint8)
    wt = np.array([[[[1]]], [[[-1]]]], dtype=np.int8)
    acc = oracle.conv_acc(x, wt, 1, 0, 2)
    assert np.array_equal(acc[..., 0], x[..., 0].astype(np.int32))
    assert np.array_equal(acc[..., 1], -x[..., 0].astype(np.int32))


def test_acc_zero_codes():
    x = np.zeros((1, 6, 6, 8), dtype=np.uint8)
    wt = -np.ones((4, 8, 3, 3), dtype=np.int8)
    assert not oracle.conv_acc(x, wt, 1, 1, 2).any()


def test_acc_reaches_bound_exactly():
    # all +1 weights on the top code: the interior sum is exactly K*(2^k-1)
    for bits in (2, 8):
        x = np.full((1, 3, 3, 4), (1 << bits) - 1, dtype=np.uint8)
        wt = np.ones((1, 4, 3, 3), dtype=np.int8)
        acc = oracle.conv_acc(x, wt, 1, 0, bits)
        assert acc[0, 0, 0, 0] == 36 * ((1 << bits) - 1)


def test_acc_flags_codes_beyond_their_bits():
    # a code of 4 in a 2-bit tensor breaks the bound and must be reported
    x = np.full((1, 3, 3, 2), 4, dtype=np.uint8)
    wt = np.ones((1, 2, 3, 3), dtype=np.int8)
    with pytest.raises(ValueError):
        oracle.conv_acc(x, wt, 1, 0, 2)
