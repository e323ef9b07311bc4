"""Pins of the separated fixed-point conversion (Sec. 2.2, Eq. 5), the
baseline of Table 2, against the float chain of the same substructure."""
import numpy as np
import pytest

from oracle import core, float_chain, separated
from workloads import Conv, layer_params, stack_input


def _layer(seed, cin=16, cout=32, h=9, w=11):
    L = Conv("sep", "x", "y", h, w, cin, cout, 3, 1, 1, 2, 2, None)
    return (L, layer_params(2000 + seed, 0, L, "calibrated"),
            stack_input(2000 + seed, (2, h, w, cin), 2))


def test_exact_parameters_make_flooring_lossless():
    # every parameter a multiple of 2^-8 (and sd = 1, so theta = mean and
    # sigma = +-1 exactly): Eq. 5's floors change nothing at m = 8, and the
    # separated codes are the float chain's
    L, p, x = _layer(3)
    rng = np.random.default_rng(7)
    co = L.cout
    p = dict(p)
    p["alpha"] = rng.integers(3, 26, size=co) / 256.0
    p["eps"] = 2.0 ** -20
    p["var"] = np.full(co, 1.0 - p["eps"])
    p["mean"] = rng.integers(-512, 512, size=co) / 256.0
    p["bn_beta"] = np.zeros(co)
    p["gamma"] = np.where(rng.random(co) < 0.2, -1.0, 1.0)
    p["bias"] = rng.integers(-2048, 2048, size=co) / 65536.0
    sp = separated.separated_params(p, 8)
    assert np.array_equal(sp["a"] / 256.0, p["alpha"])
    assert np.array_equal(sp["theta"], p["mean"])
    assert np.array_equal(sp["bias"] / 65536.0, p["bias"])
    acc = core.conv_acc(x, p["w"], 1, 1, 2)
    got = separated.codes_from_sums(acc, sp)
    want, margin = float_chain.substructure(x, p, 1, 1)
    assert np.array_equal(got[margin > 1e-9], want[margin > 1e-9])
    assert len(np.unique(want)) > 1


def test_flooring_loses_codes_and_more_bits_lose_fewer():
    # the general case: a coarse Q_m changes codes, a fine one almost none,
    # and the integrated conversion none outside the float chain's band
    L, p, x = _layer(11)
    r = separated.compare(x, p, 1, 1, 2, ms=(4, 8, 12, 30))
    assert r[4] > r[8] > r[12] >= r[30]
    assert r[4] > 0.02
    assert r[30] < 1e-3
    assert r["integrated"] == 0.0


@pytest.mark.parametrize("seed", [2, 9])
def test_fine_q_agrees_outside_a_narrow_band(seed):
    # (Y - theta) / sigma is the float chain's BN output exactly, so at
    # Q = 2^40 the floors move it by far less than 1e-6: every code whose
    # BN output lies further than that from a threshold must agree; a
    # nonzero bias exercises Eq. 5's floor(b Q^2) term
    L, p, x = _layer(seed)
    p = dict(p)
    p["bias"] = np.random.default_rng(seed).normal(0.0, 0.3, size=L.cout)
    acc = core.conv_acc(x, p["w"], 1, 1, 2)
    got = separated.codes_from_sums(acc, separated.separated_params(p, 40))
    want, margin = float_chain.substructure(x, p, 1, 1)
    keep = margin > 1e-6
    assert keep.mean() > 0.999
    assert np.array_equal(got[keep], want[keep])
    # and the coarse Q_m of Table 2 does lose codes on the same layer
    coarse = separated.codes_from_sums(acc, separated.separated_params(p, 8))
    assert np.mean(coarse != want) > 1e-3


@pytest.mark.parametrize("gamma_sign", [1.0, -1.0])
def test_sigma_sign_flips_the_comparison(gamma_sign):
    # one channel, negative gamma: sigma < 0, and the separated codes at a
    # fine Q_m still follow the float chain (the division flips the order)
    L, p, x = _layer(5, cout=4)
    p = dict(p)
    p["gamma"] = np.abs(p["gamma"]) * gamma_sign
    r = separated.compare(x, p, 1, 1, 2, ms=(40,))
    assert r[40] <= r["band"]
