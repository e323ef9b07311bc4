"""Pins of the pooling order (Eq. 4): pooling the integer sums with the sign
rule and thresholding once equals max-pooling the codes, for the window
shapes of the configs (2x2/2 valid, 3x3/2 valid overlapping, 2x2/1 same);
the literal float order (max of the conv output for every channel) agrees on
channels with a positive BN scale and not on the flipped ones."""
import numpy as np
import pytest

from oracle import core, pool_order
from workloads import Conv, layer_params, stack_input

WINDOWS = [(2, 2, "valid"), (3, 2, "valid"), (2, 1, "same"), (3, 3, "valid")]


def _layer(seed, h=13, w=12, cin=16, cout=40):
    L = Conv("po", "x", "y", h, w, cin, cout, 3, 1, 1, 2, 2, None)
    p = layer_params(3000 + seed, 0, L, "calibrated")
    x = stack_input(3000 + seed, (2, h, w, cin), 2)
    acc = core.conv_acc(x, p["w"], 1, 1, 2)
    s, t = core.fold(p["alpha"], p["beta_in"], p["mean"], p["var"], p["gamma"], p["bn_beta"],
                     p["eps"], p["q_thr"], 9 * cin, 2, bias=p["bias"])
    return L, p, x, acc, s, t


def test_pool_values_brute_force():
    # the window helper against explicit loops, clipped windows included
    rng = np.random.default_rng(1)
    v = rng.integers(-50, 50, size=(1, 5, 7, 3)).astype(np.int32)
    for k, st, mode in WINDOWS:
        got = pool_order.pool_values(v, k, st, mode, [True, False, True])
        ho, wo = got.shape[1:3]
        for oy in range(ho):
            for ox in range(wo):
                win = [v[0, y, x] for y in range(oy * st, oy * st + k)
                       for x in range(ox * st, ox * st + k) if y < 5 and x < 7]
                win = np.array(win)
                assert got[0, oy, ox, 0] == win[:, 0].max()
                assert got[0, oy, ox, 1] == win[:, 1].min()
                assert got[0, oy, ox, 2] == win[:, 2].max()


@pytest.mark.parametrize("k,st,mode", WINDOWS)
@pytest.mark.parametrize("seed", [0, 7])
def test_paper_order_on_sums_equals_pooling_codes(seed, k, st, mode):
    L, p, x, acc, s, t = _layer(seed)
    assert (s < 0).any() and (s > 0).any()
    want = core.maxpool(core.codes(acc, s, t), k, st, mode)
    got = pool_order.pooled_sums_then_codes(acc, s, t, k, st, mode)
    assert np.array_equal(got, want)
    assert len(np.unique(want)) > 1


def test_max_for_every_channel_breaks_the_flipped_ones():
    # the sign rule matters: max over the sums of a flipped channel picks
    # its lowest code
    L, p, x, acc, s, t = _layer(3)
    want = core.maxpool(core.codes(acc, s, t), 2, 2, "valid")
    wrong = core.codes(pool_order.pool_values(acc, 2, 2, "valid", True), s, t)
    flipped = np.asarray(s) < 0
    assert np.array_equal(wrong[..., ~flipped], want[..., ~flipped])
    assert (wrong[..., flipped] != want[..., flipped]).any()


def test_literal_float_order():
    # float max before BN: equal to pooling codes where gamma > 0 (outside the
    # float band), different somewhere on the gamma < 0 channels
    L, p, x, acc, s, t = _layer(5)
    want = core.maxpool(core.codes(acc, s, t), 2, 2, "valid")
    lit, margin = pool_order.float_max_then_quantize(x, p, 1, 1, 2, 2, "valid")
    pos = np.asarray(p["gamma"]) > 0
    keep = margin[..., pos] > 1e-9
    assert keep.mean() > 0.999
    assert np.array_equal(lit[..., pos][keep], want[..., pos][keep])
    assert (lit[..., ~pos] != want[..., ~pos]).any()
