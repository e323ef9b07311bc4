"""O_int: a synthetic layer stack run through the C oracle, layer by layer.

Per conv layer: integer sums (Eq. 1), then either the int32 sums themselves
(layers without a quantizer), the residual join, or the folded integer
thresholds (Eq. 7). Pool layers take the max over code windows (Eq. 4 applied
to codes). Test infrastructure.
"""
import numpy as np

from workloads import get_stack, layer_params, stack_input, Conv, Pool
from . import core


def find_layer(layers, name):
    for i, L in enumerate(layers):
        if L.name == name:
            return i, L
    raise KeyError(name)


def conv_layer(L, x, p, shortcut=None, down=None):
    """One quantized substructure. Returns (output, acc).

    output: uint8 codes, or the int32 sums when L.out_bits == 0.
    shortcut: for a join, the shortcut tensor (codes or int32 sums);
    down: the downsample conv's params dict for a conv shortcut.
    """
    a = core.conv_acc(x, p["w"], L.stride, L.pad, L.in_bits)
    if L.out_bits == 0:
        return a, a
    if L.join is not None:
        kind = L.join[0]
        if kind == "identity":
            coef = core.join_coeffs("identity", p, p["beta_in"], p["beta_in"])
        else:
            coef = core.join_coeffs("conv", p, p["beta_in"], down["beta_in"],
                                    down=down)
        return core.join_codes(a, shortcut.astype(np.int32), coef,
                               p["q_thr"]), a
    k = L.k * L.k * L.cin
    s, t = core.fold(p["alpha"], p["beta_in"], p["mean"], p["var"],
                     p["gamma"], p["bn_beta"], p["eps"], p["q_thr"], k,
                     L.in_bits, bias=p["bias"])
    return core.codes(a, s, t), a


def stack_params(config, variant="plain"):
    cfg = get_stack(config)
    return [layer_params(config, i, L, variant) if isinstance(L, Conv) else None
            for i, L in enumerate(cfg.layers)]


def stack_x(config, batch=None):
    cfg = get_stack(config)
    n = cfg.batch if batch is None else batch
    L0 = cfg.layers[0]
    return stack_input(config, (n, L0.h, L0.w, L0.cin), L0.in_bits)


def run_stack(config, batch=None, variant="plain", x=None, params=None,
              keep_acc=False):
    """Run a whole stack. Returns dict slot -> tensor.

    With keep_acc, also "in:<layer>", "out:<layer>", "acc:<layer>" (int32
    sums) and "sc:<layer>" (join shortcut) for every layer, since slots are
    reused along the stack.
    """
    cfg = get_stack(config)
    layers = cfg.layers
    if x is None:
        x = stack_x(config, batch)
    if params is None:
        params = stack_params(config, variant)
    slots = {"x": x}
    for i, L in enumerate(layers):
        if keep_acc:
            slots["in:" + L.name] = slots[L.src]
        if isinstance(L, Pool):
            slots[L.dst] = core.maxpool(slots[L.src], L.k, L.stride, L.mode)
            if keep_acc:
                slots["out:" + L.name] = slots[L.dst]
            continue
        sc = down = None
        if L.join is not None:
            sc = slots[L.join[1]]
            if L.join[0] == "conv":
                j, _ = find_layer(layers, L.join[2])
                down = params[j]
        out, a = conv_layer(L, slots[L.src], params[i], sc, down)
        slots[L.dst] = out
        if keep_acc:
            slots["acc:" + L.name] = a
            slots["out:" + L.name] = out
            if sc is not None:
                slots["sc:" + L.name] = sc
    return slots
