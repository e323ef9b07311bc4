"""The paper's defining invariant on every conv layer of the five stacks.

Table 2 reports that the integrated conversion gives exactly the float
network's outputs. Here: O_int codes (integer sums + folded thresholds, or the
fp64 residual join) equal O_float codes (the float chain conv -> BN ->
quantizer) for every element whose float value is farther than 1e-9 from a
quantizer threshold. Each layer is fed the same O_int input; batch is reduced
to keep the CPU time small, all channel and spatial sizes are the stacks' own.
"""
import numpy as np
import pytest

from oracle import stack, float_chain
from workloads import get_stack, Conv

BAND = 1e-9
BATCH = {0: 1, 1: 2, 2: 1, 3: 2, 4: 1}


def _check_config(cfg, variant):
    layers = get_stack(cfg).layers
    params = stack.stack_params(cfg, variant)
    slots = stack.run_stack(cfg, batch=BATCH[cfg], params=params, keep_acc=True)
    n_band = 0
    n_checked = 0
    for i, L in enumerate(layers):
        if not isinstance(L, Conv):
            continue
        p = params[i]
        x = slots["in:" + L.name]
        if L.out_bits == 0:
            # int32 output: the float conv must equal alpha*beta*acc + b
            y = float_chain.conv(x, p["beta_in"], p["w"], p["alpha"], p["bias"],
                                 L.stride, L.pad)
            a = slots["acc:" + L.name].astype(np.float64)
            ref = p["alpha"] * p["beta_in"] * a + p["bias"]
            assert np.allclose(y, ref, rtol=0, atol=1e-9)
            continue
        if L.join is None:
            code, margin = float_chain.substructure(x, p, L.stride, L.pad)
        elif L.join[0] == "identity":
            sc = p["beta_in"] * slots["sc:" + L.name].astype(np.float64)
            code, margin = float_chain.joined(x, p, L.stride, L.pad, sc)
        else:
            j, D = stack.find_layer(layers, L.join[2])
            pd = params[j]
            sc = float_chain.downsample_value(slots["in:" + D.name], pd, D.stride, D.pad)
            code, margin = float_chain.joined(x, p, L.stride, L.pad, sc)
        got = slots["out:" + L.name]
        clear = margin > BAND
        assert got.shape == code.shape, L.name
        mism = (got != code) & clear
        assert not mism.any(), (L.name, int(mism.sum()))
        n_band += int((~clear).sum())
        n_checked += got.size
    return n_band, n_checked


@pytest.mark.parametrize("variant", ["plain", "calibrated"])
@pytest.mark.parametrize("cfg", [0, 1, 2, 3, 4])
def test_integer_codes_equal_float_chain(cfg, variant):
    n_band, n_checked = _check_config(cfg, variant)
    assert n_checked > 0
    assert n_band <= 1e-6 * n_checked + 2


def test_stack_shapes_chain():
    # each layer's output shape (derived by the oracle) is the next reader's
    # listed input shape
    for cfg in range(5):
        layers = get_stack(cfg).layers
        slots = stack.run_stack(cfg, batch=1, keep_acc=True)
        for L in layers:
            x = slots["in:" + L.name]
            c = L.cin if isinstance(L, Conv) else L.c
            assert x.shape[1:] == (L.h, L.w, c), (cfg, L.name)
