"""Pins of the compact thresholds (Sec. 3.2, Eq. 8): a hand-worked channel
for each sign of gamma and for gamma = 0, exact agreement with the table fold
where the arithmetic is exact, the true floor of the exact rational t_i away
from integers, and the float chain's codes on seeded k-bit layers."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import compact, core, float_chain
from workloads import Conv, layer_params, stack_input
from workloads.gen import STEP


def _p(gamma, bn_beta=0.0):
    return {"alpha": np.array([0.25]), "beta_in": 0.5, "bias": np.array([0.0]),
            "mean": np.array([1.0]), "var": np.array([1.0]), "eps": 0.0,
            "gamma": np.array([gamma]), "bn_beta": np.array([bn_beta])}


def test_hand_worked_channels():
    # alpha*beta = 1/8, sd = 1, q = 0.25, 0.75, 1.25 (base 0.5, offset -0.25)
    r = compact.fold_compact(_p(2.0), 0.5, -0.25, 2)
    assert r["base"][0] == 2.0 and r["offset"][0] == 7.0 and r["s"][0] == 1
    s, T = compact.expand(r, 2, 1000.0)
    assert list(T[0]) == [9, 11, 13] and s[0] == 1
    # gamma = -2: Y_bn = 2 - a/4; t_i = 9 - 2i; thresholds on -a
    r = compact.fold_compact(_p(-2.0), 0.5, -0.25, 2)
    assert r["base"][0] == -2.0 and r["offset"][0] == 9.0
    s, T = compact.expand(r, 2, 1000.0)
    assert s[0] == -1 and list(T[0]) == [-7, -5, -3]
    for a in range(-20, 21):
        ybn = 2.0 - a / 4.0
        want = sum(ybn > q for q in (0.25, 0.75, 1.25))
        assert sum(-a > t for t in T[0]) == want
    # gamma = 0: the constant code #{i : 0.8 > q_i} = 2
    r = compact.fold_compact(_p(0.0, 0.8), 0.5, -0.25, 2)
    assert r["s"][0] == 0 and r["cstar"][0] == 2
    s, T = compact.expand(r, 2, 50.0)
    assert s[0] == 1 and list(T[0]) == [-51, -51, 50]


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_equals_table_fold_on_exact_parameters(bits):
    # dyadic parameters, alpha and gamma powers of two: every step of both
    # folds is exact, so the records agree
    rng = np.random.default_rng(bits)
    c = 48
    p = {"alpha": 2.0 ** -rng.integers(2, 8, c).astype(np.float64), "beta_in": 0.5,
         "bias": rng.integers(-64, 64, c) / 256.0, "mean": rng.integers(-512, 512, c) / 64.0,
         "var": np.ones(c), "eps": 0.0, "gamma": rng.choice([-4.0, -1.0, -0.5, 0.0, 0.5, 2.0], c),
         "bn_beta": rng.integers(-8, 8, c) / 8.0}
    nq = (1 << bits) - 1
    q = np.array([i * STEP - STEP / 2 for i in range(1, nq + 1)])
    k = 576
    bound = float(k * 3)
    s1, T1 = core.fold(p["alpha"], p["beta_in"], p["mean"], p["var"], p["gamma"], p["bn_beta"],
                       p["eps"], q, k, 2, bias=p["bias"])
    s2, T2 = compact.expand(compact.fold_compact(p, STEP, -STEP / 2, bits), bits, bound)
    assert np.array_equal(s1, s2) and np.array_equal(T1, T2)


def _layer(bits, seed):
    L = Conv("cp", "x", "y", 9, 10, 64, 48, 3, 1, 1, 2, bits, None)
    return L, layer_params(4000 + seed, 0, L, "calibrated")


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_true_floor_of_the_exact_threshold(bits):
    # against exact rational arithmetic on the same float inputs: T_i is the
    # floor of s * t_i wherever t_i is not within 1e-9 of an integer
    L, p = _layer(bits, 1)
    r = compact.fold_compact(p, STEP, -STEP / 2, bits)
    bound = 1e9
    s, T = compact.expand(r, bits, bound)
    checked = 0
    for c in range(L.cout):
        ga = Fraction(float(p["gamma"][c]))
        if ga == 0:
            continue
        sd = Fraction(float(np.sqrt(p["var"][c] + p["eps"])))
        ab = Fraction(float(p["alpha"][c])) * Fraction(float(p["beta_in"]))
        for i in range(1, (1 << bits)):
            q = i * Fraction(STEP) - Fraction(STEP) / 2
            t = ((q - Fraction(float(p["bn_beta"][c]))) * sd / ga + Fraction(float(p["mean"][c]))
                 - Fraction(float(p["bias"][c]))) / ab
            st = t if ga > 0 else -t
            fl = st.numerator // st.denominator
            if abs(st - round(st)) > Fraction(1, 10 ** 9):
                assert T[c, i - 1] == fl, (c, i)
                checked += 1
    assert checked > 100


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_codes_equal_the_float_chain(bits):
    # the paper's claim for the compact form: the same codes as the float
    # network, outside the band where the float chain's own rounding decides
    L, p = _layer(bits, 2)
    x = stack_input(4000 + bits, (2, L.h, L.w, L.cin), 2)
    acc = core.conv_acc(x, p["w"], 1, 1, 2)
    s, T = compact.expand(compact.fold_compact(p, STEP, -STEP / 2, bits), bits,
                          float(9 * L.cin * 3))
    got = core.codes(acc, s, T)
    want, margin = float_chain.substructure(x, p, 1, 1)
    keep = margin > 1e-9
    assert keep.mean() > 0.999
    assert np.array_equal(got[keep], want[keep])
    assert len(np.unique(want)) > 2
