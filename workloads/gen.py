"""Seeded random draws for the synthetic stacks.

Every array comes from NumPy's PCG64 seeded with
SeedSequence([SEED_ROOT, config, layer, kind, *extra]); the path under test and
the oracle consume the same arrays.

Distributions (one rule for every layer of every stack):
  input codes      uniform on {0 .. 2^bits - 1}, drawn image by image so that a
                   smaller batch is a prefix of the full one
  weights          +1 / -1 with probability 1/2, PyTorch OIHW int8
  alpha            uniform [0.01, 0.1] per output channel
  BN mean          normal, variance 4 (std 2)
  BN var           uniform [0.5, 2]
  BN gamma         uniform [0.5, 1.5], negated on exactly round(0.1 * Cout)
                   channels chosen uniformly without replacement
  BN beta          standard normal
  BN eps           1e-5
  bias             0
  input step beta  0.5 for 2-bit codes, 1/255 for 8-bit codes
  quantizer        levels {0, D, 2D, ...} with step D = 0.5 and mid-point
                   thresholds (i - 1/2) * D, i = 1 .. 2^k - 1

The "calibrated" variant replaces the BN mean and variance by draws scaled to
the spread a sum of K products of random +-1 weights with uniform codes has
(variance K * E[x^2]), so that output codes use all levels rather than
saturating. It is for test power only; timing uses the plain variant.
"""
import enum
import numpy as np

SEED_ROOT = 1911080760
STEP = 0.5          # quantizer step of every hidden layer
EPS = 1e-5


class Kind(enum.IntEnum):
    INPUT = 0
    WEIGHT = 1
    ALPHA = 2
    MEAN = 3
    VAR = 4
    GAMMA = 5
    GAMMA_FLIP = 6
    BN_BETA = 7


def _rng(config, layer, kind, *extra):
    ss = np.random.SeedSequence([SEED_ROOT, int(config), int(layer), int(kind)]
                                + [int(e) for e in extra])
    return np.random.Generator(np.random.PCG64(ss))


def input_step(bits):
    """Step between consecutive input code levels."""
    return 1.0 / 255.0 if bits == 8 else STEP


def quant_thresholds(bits):
    """Mid-point thresholds of the uniform k-bit quantizer with step 0.5."""
    n = (1 << bits) - 1
    return np.array([(i - 0.5) * STEP for i in range(1, n + 1)], dtype=np.float64)


def stack_input(config, shape, bits):
    """Input codes, NHWC uint8, drawn one image at a time."""
    n, h, w, c = shape
    hi = 1 << bits
    out = np.empty(shape, dtype=np.uint8)
    for i in range(n):
        out[i] = _rng(config, 0, Kind.INPUT, i).integers(0, hi, size=(h, w, c),
                                                        dtype=np.uint8)
    return out


def layer_params(config, layer_index, layer, variant="plain"):
    """Weights and float parameters of one conv layer.

    Returns a dict with: w (int8 OIHW +-1), alpha, bias, mean, var, gamma,
    bn_beta (float64 per output channel), eps, beta_in, q_thr (float64).
    """
    co, ci, k = layer.cout, layer.cin, layer.k
    li = layer_index + 1
    w = _rng(config, li, Kind.WEIGHT).integers(0, 2, size=(co, ci, k, k),
                                               dtype=np.int8)
    w = (w * 2 - 1).astype(np.int8)
    alpha = _rng(config, li, Kind.ALPHA).uniform(0.01, 0.1, size=co)
    beta_in = input_step(layer.in_bits)
    if variant == "plain":
        mean = _rng(config, li, Kind.MEAN).normal(0.0, 2.0, size=co)
        var = _rng(config, li, Kind.VAR).uniform(0.5, 2.0, size=co)
    elif variant == "calibrated":
        levels = (1 << layer.in_bits) - 1
        ex2 = float(np.mean(np.arange(levels + 1, dtype=np.float64) ** 2))
        spread = alpha * beta_in * np.sqrt(k * k * ci * ex2)
        mean = _rng(config, li, Kind.MEAN).normal(0.0, 0.5, size=co) * spread
        var = _rng(config, li, Kind.VAR).uniform(0.5, 2.0, size=co) * spread ** 2
    else:
        raise ValueError("unknown variant %r" % variant)
    gamma = _rng(config, li, Kind.GAMMA).uniform(0.5, 1.5, size=co)
    n_flip = int(round(0.1 * co))
    flip = _rng(config, li, Kind.GAMMA_FLIP).choice(co, size=n_flip, replace=False)
    gamma[flip] = -gamma[flip]
    bn_beta = _rng(config, li, Kind.BN_BETA).normal(0.0, 1.0, size=co)
    out_bits = layer.out_bits if layer.out_bits > 0 else 2
    return dict(w=w, alpha=alpha, bias=np.zeros(co), mean=mean, var=var,
                gamma=gamma, bn_beta=bn_beta, eps=EPS, beta_in=beta_in,
                q_thr=quant_thresholds(out_bits))
