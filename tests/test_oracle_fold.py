"""Pins of the oracle's threshold fold and integer codes (Eq. 6 -> Eq. 7/8).

The fold is checked exhaustively: for every channel and every integer sum a
the layer can produce (|a| <= B = K*(2^k_in - 1)), the code from the folded
integer thresholds must equal the code from evaluating the composed float
inequality of Eq. (6) directly, except where the float value lies within
1e-9 of a quantizer threshold.
"""
from fractions import Fraction
import math

import numpy as np
import pytest

import oracle
from oracle import brute
from workloads import get_stack, layer_params, quant_thresholds

BAND = 1e-9


def eq6_codes(a, p):
    """Eq. (6) evaluated in fp64 for a column of integer sums a (broadcast)."""
    y = p["alpha"] * p["beta_in"] * a + p["bias"]
    ybn = p["gamma"] * (y - p["mean"]) / np.sqrt(p["var"] + p["eps"]) + p["bn_beta"]
    code = np.zeros(ybn.shape, dtype=np.int64)
    margin = np.full(ybn.shape, np.inf)
    for q in p["q_thr"]:
        code += ybn > q
        margin = np.minimum(margin, np.abs(ybn - q))
    return code, margin


def fold_codes(a, p, k, in_bits, flags=0):
    s, t = oracle.fold(p["alpha"], p["beta_in"], p["mean"], p["var"],
                       p["gamma"], p["bn_beta"], p["eps"], p["q_thr"], k,
                       in_bits, bias=p["bias"], flags=flags)
    acc = np.ascontiguousarray(np.broadcast_to(a, (a.shape[0], s.shape[0])),
                               dtype=np.int32)
    return oracle.codes(acc, s, t).astype(np.int64), s, t


def exhaustive(p, k, in_bits, flags=0):
    bound = k * ((1 << in_bits) - 1)
    a = np.arange(-bound, bound + 1, dtype=np.int64)[:, None]
    got, s, t = fold_codes(a, p, k, in_bits, flags)
    want, margin = eq6_codes(a.astype(np.float64), p)
    clear = margin > BAND
    return got, want, clear, s, t


LAYERS = [(0, 0), (1, 0), (1, 3), (3, 17), (4, 0), (4, 10), (2, 14)]


@pytest.mark.parametrize("variant", ["plain", "calibrated"])
@pytest.mark.parametrize("cfg,li", LAYERS)
def test_fold_exhaustive_against_eq6(cfg, li, variant):
    L = get_stack(cfg).layers[li]
    p = layer_params(cfg, li, L, variant)
    k = L.k * L.k * L.cin
    got, want, clear, s, t = exhaustive(p, k, L.in_bits)
    assert np.array_equal(got[clear], want[clear])
    # the band is essentially never hit with random parameters
    assert (~clear).sum() <= 2
    # flipped channels are exactly the negative-gamma ones
    assert np.array_equal(s < 0, p["gamma"] < 0)
    assert (s < 0).sum() == round(0.1 * L.cout)
    # thresholds are non-decreasing in i and within [-B-1, B]
    bound = k * ((1 << L.in_bits) - 1)
    assert (np.diff(t, axis=1) >= 0).all()
    assert t.min() >= -bound - 1 and t.max() <= bound


def test_mutation_without_flip_fails():
    # planting the paper's "sigma > 0" assumption (no flip) must be caught
    L = get_stack(3).layers[17]
    p = layer_params(3, 17, L, "calibrated")
    k = L.k * L.k * L.cin
    got, want, clear, s, t = exhaustive(p, k, L.in_bits, flags=oracle.MUTATE_NO_FLIP)
    neg = p["gamma"] < 0
    bad_cols = (got != want) & clear
    assert bad_cols[:, neg].any(axis=0).all()       # every flipped channel fails
    assert not bad_cols[:, ~neg].any()              # the others are untouched


def _params(co, **kw):
    p = dict(alpha=np.full(co, 0.5), bias=np.zeros(co), mean=np.zeros(co),
             var=np.ones(co), gamma=np.ones(co), bn_beta=np.zeros(co), eps=0.0,
             beta_in=0.5, q_thr=quant_thresholds(2))
    for key, v in kw.items():
        p[key] = np.asarray(v, dtype=np.float64) if isinstance(v, list) else v
    return p


def _exact_code(a, p, c):
    # Eq. (6) in exact rational arithmetic (sd must be exactly representable)
    sd = Fraction(math.sqrt(p["var"][c] + p["eps"]))
    assert sd * sd == Fraction(p["var"][c]) + Fraction(p["eps"])
    y = Fraction(p["alpha"][c]) * Fraction(p["beta_in"]) * a + Fraction(p["bias"][c])
    ybn = Fraction(p["gamma"][c]) * (y - Fraction(p["mean"][c])) / sd + Fraction(p["bn_beta"][c])
    return sum(1 for q in p["q_thr"] if ybn > Fraction(q))


def test_thresholds_on_integers_ties_go_low():
    # alpha*beta = 0.25 puts every new threshold on an integer (t = 1, 3, 5 and
    # -1, -3, -5 for negative gamma); equality must give the lower code (Eq. 3)
    p = _params(4, alpha=[0.5, 0.5, 0.5, 0.5], gamma=[1.0, -1.0, 2.0, -0.5],
                mean=[0.0, 0.0, 0.5, -0.25])
    a = np.arange(-40, 41)[:, None]
    got, s, t = fold_codes(a, p, 16, 2)
    for c in range(4):
        for ai, g in zip(a[:, 0], got[:, c]):
            assert g == _exact_code(int(ai), p, c), (c, ai)
    assert list(t[0]) == [1, 3, 5]
    assert list(s) == [1, -1, 1, -1]
    assert list(t[1]) == [1, 3, 5]


def test_gamma_zero_gives_constant_code():
    p = _params(4, gamma=[0.0] * 4, bn_beta=[-1.0, 0.5, 1.0, 3.0])
    a = np.arange(-30, 31)[:, None]
    got, s, t = fold_codes(a, p, 10, 2)
    for c, want in enumerate([0, 1, 2, 3]):
        assert (got[:, c] == want).all()


def test_zero_codes_give_count_of_negative_thresholds(rng):
    L = get_stack(0).layers[0]
    p = layer_params(0, 0, L, "plain")
    s, t = oracle.fold(p["alpha"], p["beta_in"], p["mean"], p["var"],
                       p["gamma"], p["bn_beta"], p["eps"], p["q_thr"], 576, 2)
    acc = np.zeros((3, L.cout), dtype=np.int32)
    c = oracle.codes(acc, s, t)
    assert np.array_equal(c[0], (t < 0).sum(axis=1).astype(np.uint8))


def test_extreme_alpha_and_saturation():
    # tiny and large alpha, huge |mean| (thresholds beyond the bound get
    # clamped), nonzero bias: codes must still follow Eq. (6)
    co = 6
    p = _params(co, alpha=[0.01, 0.1, 0.01, 0.1, 0.05, 0.05],
                mean=[0.0, 0.0, 1e6, -1e6, 3.0, -3.0],
                gamma=[1.0, -1.3, 0.7, -0.7, 1.2, -1.2],
                bias=[0.0, 0.1, 0.0, 0.0, -0.2, 0.3],
                var=[0.5, 2.0, 1.0, 1.0, 0.7, 1.9], eps=1e-5)
    k = 9 * 8
    got, want, clear, s, t = exhaustive(p, k, 2)
    assert np.array_equal(got[clear], want[clear])
    assert (got[:, 2] == 0).all() and (got[:, 3] == 0).all()
    bound = k * 3
    assert t[2].tolist() == [bound] * 3


def test_brute_force_eq6_matches_vectorised_eq6(rng):
    # the two float evaluations of Eq. (6) used by the tests agree
    L = get_stack(0).layers[0]
    p = layer_params(0, 0, L, "calibrated")
    a = rng.integers(-1700, 1700, size=64)
    want, margin = eq6_codes(a[:, None].astype(np.float64), p)
    for r, ai in enumerate(a):
        for c in range(0, L.cout, 7):
            code, m = brute.code_eq6(int(ai), p["alpha"][c], p["beta_in"],
                                     p["bias"][c], p["mean"][c], p["var"][c],
                                     p["gamma"][c], p["bn_beta"][c], p["eps"],
                                     p["q_thr"])
            assert code == want[r, c]


@pytest.mark.parametrize("bad", ["alpha", "var", "q", "nan", "beta"])
def test_fold_rejects_invalid(bad):
    p = _params(3)
    kw = {}
    if bad == "alpha":
        p["alpha"] = np.array([0.5, 0.0, 0.5])
    elif bad == "var":
        p["var"] = np.array([1.0, -1.0, 1.0])
    elif bad == "q":
        p["q_thr"] = np.array([0.25, 0.25, 1.25])
    elif bad == "nan":
        p["mean"] = np.array([0.0, np.nan, 0.0])
    elif bad == "beta":
        p["beta_in"] = 0.0
    with pytest.raises(ValueError):
        oracle.fold(p["alpha"], p["beta_in"], p["mean"], p["var"], p["gamma"],
                    p["bn_beta"], p["eps"], p["q_thr"], 9, 2)


@pytest.mark.parametrize("out_bits", [1, 3, 4])
def test_fold_k_bit_generalisation(out_bits):
    # Eq. (8): 2^k - 1 thresholds; uniform thresholds i*base + offset
    L = get_stack(0).layers[0]
    p = layer_params(0, 0, L, "calibrated")
    p["q_thr"] = quant_thresholds(out_bits)
    got, want, clear, s, t = exhaustive(p, 576, 2)
    assert t.shape[1] == (1 << out_bits) - 1
    assert np.array_equal(got[clear], want[clear])
