"""GPU parity of whole stacks through ifq_run_stack: every tensor the stack
leaves in its workspace and its output must equal the oracle's bit for bit.

Small cases use a reduced batch; the full cases run each stack at its own
batch size in the launch configuration the benchmark times, and compare every
output element against the oracle run on the host cores.
"""
import numpy as np
import pytest

from oracle import stack as ostack
from oracle import layout as olayout
from workloads import get_stack

pytestmark = pytest.mark.gpu

_ORACLE = {}


def oracle_run(cfg, batch, variant):
    key = (cfg, batch, variant)
    if key not in _ORACLE:
        params = ostack.stack_params(cfg, variant)
        x = ostack.stack_x(cfg, batch)
        _ORACLE.clear()
        _ORACLE[key] = (params, x, ostack.run_stack(cfg, x=x, params=params))
    return _ORACLE[key]


@pytest.fixture(scope="module")
def P():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1911_08076_amd as P
    return P


def check_stack(P, cfg, batch, layout, variant):
    import torch
    params, x, want = oracle_run(cfg, batch, variant)
    layers = get_stack(cfg).layers
    # "b64f": downsamples inside their joins; "...p": pools inside the convs
    # that feed them, where a fused kernel covers the pair
    fuse = layout in ("b64f", "b64p", "b64pa", "b64fp4", "b64pfp4")
    fpool = "all" if layout.endswith("pa") else (layout.endswith("p") or layout == "b64pfp4")
    fp4 = layout.endswith("fp4")
    base = {"b64f": "b64", "b64p": "b64", "b64pa": "b64", "i8p": "i8",
            "b64fp4": "b64", "b64pfp4": "b64"}.get(layout, layout)
    dev = P.DeviceStack(layers, params, batch, code_layout=base, fuse_down=fuse,
                        fuse_pool=fpool, fp4=fp4)
    if fp4 and base == "b64" and cfg == 3:
        # the 3x3 layers of the ResNet-shaped stack are on fp4 (at full batch
        # all but the 64-channel ones), the fused downsample joins included
        covered = {L.name for L in layers if hasattr(L, "cin") and
                   (L.join is None or L.join[0] == "identity" or L.name in dev.fused)}
        assert dev.fp4_layers and set(dev.fp4_layers) <= covered
    if fuse:
        # every downsample of a ResNet-shaped stack is folded into its join
        assert len(dev.fused) == sum(1 for L in layers if L.name.endswith(".down"))
    if fpool:
        names = dev.layer_kernel_names()
        for i, L in enumerate(dev.layers):
            if L.name in dev.fused_pool:
                assert dev._layers[i].kind in (P.IFQ_LAYER_CONV_POOL,
                                               P.IFQ_LAYER_CONV_POOL_FP4) and names[i]
    xd = dev.upload_input(x)
    y = dev.alloc_output()
    dev.run(xd, y)
    torch.cuda.synchronize()
    got = dev.download_output(y)
    assert got.shape == want["y"].shape
    assert np.array_equal(got, want["y"]), "stack output differs"
    checked = 1
    # the oracle keeps the last tensor written under each slot name; a slot
    # is compared where the same layer wrote it last on both sides (fusions
    # leave some names to other writers, or move a tensor to a slot of its own)
    last_writer = {L.dst: L.name for L in layers}
    for name, (shape, lay, bits) in dev.tensor_info.items():
        if name in ("x", "y"):
            continue
        orig, writer = dev.slot_origin[name]
        if last_writer.get(orig) != writer:
            continue
        g = dev.read_slot(name)
        w = want[orig]
        if lay == P.IFQ_LAYOUT_U2_NHWC_PACKED:
            w = olayout.pack2(w)
        elif lay == P.IFQ_LAYOUT_U2_BLOCK64:
            w = olayout.pack_block64(w)
        assert np.array_equal(g, w), "slot %s differs" % name
        checked += 1
    # running again gives the same bytes (no state carried between runs)
    y2 = dev.alloc_output()
    dev.run(xd, y2)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)
    return checked


SMALL = [(0, 1), (1, 2), (2, 1), (3, 2), (4, 1)]


@pytest.mark.parametrize("layout", ["i8", "u2", "b64", "b64f", "b64p", "b64pa", "i8p",
                                    "b64fp4", "b64pfp4"])
@pytest.mark.parametrize("cfg,batch", SMALL)
def test_stack_small_batch(P, cfg, batch, layout):
    for variant in ("calibrated", "plain"):
        assert check_stack(P, cfg, batch, layout, variant) >= 1


@pytest.mark.slow
@pytest.mark.parametrize("layout", ["b64", "u2", "i8"])
@pytest.mark.parametrize("cfg", [0, 1, 3, 4, 2])
def test_stack_full_size(P, cfg, layout):
    batch = get_stack(cfg).batch
    check_stack(P, cfg, batch, layout, "plain")


@pytest.mark.slow
@pytest.mark.parametrize("cfg", [4, 2])
def test_stack_full_size_fused_pools(P, cfg):
    # the benchmark's configuration of the stacks with pools: BLOCK64 codes,
    # the 2x2/2 pools inside the convs that feed them
    check_stack(P, cfg, get_stack(cfg).batch, "b64p", "plain")


@pytest.mark.slow
def test_stack_full_size_fp4(P):
    # the ResNet-18 body at batch 64 with its threshold layers on fp4
    check_stack(P, 3, get_stack(3).batch, "b64fp4", "plain")


@pytest.mark.slow
def test_stack_full_size_fused_downsample(P):
    # the benchmark's configuration: ResNet-18 body, batch 64, BLOCK64 codes,
    # downsample convs inside their joins
    check_stack(P, 3, get_stack(3).batch, "b64f", "plain")


@pytest.mark.parametrize("bits", [3, 4])
def test_kbit_alexnet_body(P, bits):
    # the AlexNet body with k-bit activations (the k = 3, 4 networks of
    # Tables 2-3): every conv takes and gives k-bit codes (one byte each), the
    # pools run on them; the generic path and the k-bit folds, end to end
    import dataclasses
    import torch
    from oracle import core
    from oracle.stack import conv_layer
    from workloads import Conv, layer_params, stack_input
    cfg = get_stack(1)
    layers = [dataclasses.replace(L, in_bits=bits, out_bits=bits) if isinstance(L, Conv)
              else dataclasses.replace(L, bits=bits) for L in cfg.layers]
    batch = 2
    params = [layer_params(1, i, L, "calibrated") if isinstance(L, Conv) else None
              for i, L in enumerate(layers)]
    L0 = layers[0]
    x = stack_input(1, (batch, L0.h, L0.w, L0.cin), bits)
    slots = {"x": x}
    for i, L in enumerate(layers):
        if isinstance(L, Conv):
            slots[L.dst], _ = conv_layer(L, slots[L.src], params[i])
        else:
            slots[L.dst] = core.maxpool(slots[L.src], L.k, L.stride, L.mode)
    dev = P.DeviceStack(layers, params, batch, code_layout="i8")
    xd = dev.upload_input(x)
    y = dev.alloc_output()
    dev.run(xd, y)
    torch.cuda.synchronize()
    got = dev.download_output(y)
    assert np.array_equal(got, slots["y"])
    assert got.max() > 3   # codes beyond the 2-bit range occur
