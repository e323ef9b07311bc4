"""Separated fixed-point conversion of one substructure (Sec. 2.2, Eq. 5),
the baseline the integrated conversion (Sec. 3.2) is measured against in
Table 2. Test infrastructure, host only.

Every floating-point parameter is scaled by Q_m = 2^m and floored on its own:
the conv's alpha and beta (and the bias at Q_m^2), as Eq. 5 writes it, and
likewise the BN parameters theta, sigma and the quantizer thresholds. The
paper leaves the arithmetic after Eq. 5 open; the reading used here (each
step exact on the floored values, so that the only loss is the flooring):

  Y     = (floor(alpha Q) floor(beta Q) S + floor(b Q^2)) / Q^2   S = W_b (x) X_q
  theta = floor(theta Q) / Q,  sigma = floor(sigma Q) / Q
  thr_i = floor(thr_i Q) / Q
  code  = #{ i : (Y - theta) / sigma > thr_i }

with Eq. 2's two BN parameters taken from the BN affine as
theta = mean - bn_beta * sd / gamma and sigma = sd / gamma (sd =
sqrt(var + eps); sigma < 0 where gamma < 0, and the division then flips
the comparison as the float chain does). The integer sums S come from the
C oracle; everything after them is float64 on exactly representable
rationals.
"""
import numpy as np

from . import core
from . import float_chain


def separated_params(p, m):
    """The floored parameters of one layer at Q_m = 2^m (per channel)."""
    q = float(2 ** m)
    alpha = np.asarray(p["alpha"], np.float64)
    sd = np.sqrt(np.asarray(p["var"], np.float64) + p["eps"])
    gamma = np.asarray(p["gamma"], np.float64)
    theta = np.asarray(p["mean"], np.float64) - np.asarray(p["bn_beta"], np.float64) * sd / gamma
    sigma = sd / gamma
    bias = np.broadcast_to(np.asarray(p["bias"], np.float64), alpha.shape)
    return {
        "a": np.floor(alpha * q),                      # floor(alpha Q)
        "b": np.floor(float(p["beta_in"]) * q),         # floor(beta Q)
        "bias": np.floor(bias * q * q),                 # floor(b Q^2)
        "theta": np.floor(theta * q) / q,
        "sigma": np.floor(sigma * q) / q,
        "thr": np.floor(np.asarray(p["q_thr"], np.float64) * q) / q,
        "q": q,
    }


def codes_from_sums(acc, sp):
    """Eq. 5 then BN and the quantizer on the floored parameters."""
    q = sp["q"]
    y = (sp["a"] * sp["b"] * acc.astype(np.float64) + sp["bias"]) / (q * q)
    with np.errstate(divide="ignore", invalid="ignore"):
        z = (y - sp["theta"]) / sp["sigma"]
    code = np.zeros(acc.shape, dtype=np.uint8)
    for t in sp["thr"]:
        code += (z > t).astype(np.uint8)
    return code


def compare(x, p, stride, pad, in_bits, ms, band=1e-9):
    """Code mismatch rates against the float chain (O_float) on one layer.

    Returns {m: fraction of output codes that differ} for the separated
    conversion at each m, plus "integrated": the integer-threshold codes
    (O_int), counted outside the band around the float thresholds where
    the float chain's own rounding decides, and "band": the fraction of
    elements inside it."""
    acc = core.conv_acc(x, p["w"], stride, pad, in_bits)
    want, margin = float_chain.substructure(x, p, stride, pad)
    out = {}
    for m in ms:
        got = codes_from_sums(acc, separated_params(p, m))
        out[m] = float(np.mean(got != want))
    k = int(np.prod(p["w"].shape[1:]))
    s, t = core.fold(p["alpha"], p["beta_in"], p["mean"], p["var"], p["gamma"], p["bn_beta"],
                     p["eps"], p["q_thr"], k, in_bits, bias=p["bias"])
    integ = core.codes(acc, s, t)
    outside = margin > band
    out["integrated"] = float(np.mean((integ != want) & outside))
    out["band"] = float(np.mean(~outside))
    return out


def table(ms=(8, 9, 10, 12)):
    """The synthetic analogue of Table 2 on seeded layers of the configs:
    per layer, the separated conversion's code mismatch rate against the
    float chain at each m, and the integrated conversion's (outside the
    band)."""
    from workloads import gen, stacks
    rows = []
    for cfg, names, n in ((0, ("conv",), 1), (1, ("conv3", "conv4"), 2),
                          (3, ("l2.1.conv1", "l3.1.conv1"), 2)):
        st = stacks.get_stack(cfg)
        for li, L in enumerate(st.layers):
            if getattr(L, "name", None) not in names:
                continue
            for variant in ("plain", "calibrated"):
                p = gen.layer_params(cfg, li, L, variant)
                x = gen.stack_input(cfg + 100 * li, (n, L.h, L.w, L.cin), L.in_bits)
                r = compare(x, p, L.stride, L.pad, L.in_bits, ms)
                rows.append((st.name, L.name, variant, r))
    return rows


if __name__ == "__main__":
    ms = (8, 9, 10, 12)
    print("| stack | layer | BN params | " + " | ".join("separated m=%d" % m for m in ms) +
          " | integrated | in band |")
    print("|---" * (len(ms) + 5) + "|")
    for stack, layer, variant, r in table(ms):
        print("| %s | %s | %s | " % (stack, layer, variant) +
              " | ".join("%.4f" % r[m] for m in ms) +
              " | %.4f | %.1e |" % (r["integrated"], r["band"]))
