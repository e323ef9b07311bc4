"""GPU parity of the contraction of Eq. (1) split over K across workgroups
(the register-blocked 3x3 kernel's partial tiles added by the last
workgroup of each tile, then the threshold epilogue of Eq. 7/8; run through
ifq_conv_forward_split, the planner prices it above every unsplit launch of
the benchmark layers): int32 sums and codes must equal the oracle's bit for
bit for splits of 2 and 4 on every int8 variant that takes them, at the
ResNet-18 l4 and the Tiny-YOLOv2 c7 shapes and on ragged and stride-2
layers; the workspace's counters must be left at zero, so one workspace
serves repeated calls and other layers."""
import zlib

import numpy as np
import pytest

from gpu_util import (B64, gpu_layer, oracle_layer, expect_layout, make_layer, params_for,
                      codes_for, device)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1911_08076_amd as P
    return P


def _setup(name, n, h, w, cin, cout, st=1):
    L = make_layer(name, h, w, cin, cout, 3, st, 1, 2, 2)
    seed = zlib.crc32(name.encode()) % 997
    p = params_for(seed, L)
    x = codes_for(seed, (n, h, w, cin), 2)
    want_acc, want = oracle_layer(L, x, p)
    assert len(np.unique(want)) > 1
    return L, p, x, want_acc, want


# (name, n, h, w, c_in, c_out, stride)
FORCED = [("l4", 64, 7, 7, 512, 512, 1), ("yolo_c7", 8, 13, 13, 512, 512, 1),
          ("r9x11_256_128", 3, 9, 11, 256, 128, 1),
          ("s2_15_256_256", 2, 15, 15, 256, 256, 2)]


def _int8_w2(P):
    # conv_w2's int8 variants (the first ten; the persistent kernels follow)
    return [v for v in range(10) if P.ifq_conv_variant_fp4(v) == 0]


@pytest.mark.parametrize("case", FORCED, ids=[c[0] for c in FORCED])
def test_forced_split_bit_exact(P, case):
    import torch
    name, n, h, w, cin, cout, st = case
    L, p, x, want_acc, want = _setup(name, n, h, w, cin, cout, st)
    d = P.conv_desc(n, h, w, cin, cout, 3, st, 1, 2, 2, B64, B64)
    runs = 0
    for v in _int8_w2(P):
        for ks in (2, 4):
            nb = P.ifq_conv_split_workspace_bytes(d, v, ks)
            if not nb:
                continue
            ws = torch.zeros(nb, dtype=torch.uint8, device=device())
            print("split: %s variant %d x%d" % (name, v, ks), flush=True)
            for rep in range(2):   # the same workspace twice: counters back at zero
                acc, got = gpu_layer(P, L, n, x, p, in_layout=B64, out_layout=B64,
                                     split=(v, ks, ws))
                assert np.array_equal(acc, want_acc), (name, v, ks, rep)
                assert np.array_equal(got, expect_layout(want, B64)), (name, v, ks, rep)
            assert int(ws[:64 << 10].to(torch.int32).abs().sum()) == 0
            runs += 1
    assert runs >= 2, name


def test_one_workspace_serves_several_layers(P):
    # two layers of different tiles and splits, then the first again, all on
    # one workspace sized for the largest
    import torch
    c7 = _setup("ws_c7", 8, 13, 13, 512, 512)
    l4 = _setup("ws_l4", 16, 7, 7, 512, 512)
    d7 = P.conv_desc(8, 13, 13, 512, 512, 3, 1, 1, 2, 2, B64, B64)
    d4 = P.conv_desc(16, 7, 7, 512, 512, 3, 1, 1, 2, 2, B64, B64)
    nb = max(P.ifq_conv_split_workspace_bytes(d7, 2, 2), P.ifq_conv_split_workspace_bytes(d4, 0, 4))
    assert P.ifq_conv_split_workspace_bytes(d7, 2, 2) and P.ifq_conv_split_workspace_bytes(d4, 0, 4)
    ws = torch.zeros(nb, dtype=torch.uint8, device=device())
    for which, n, split in (("c7", 8, (2, 2, ws)), ("l4", 16, (0, 4, ws)), ("c7", 8, (2, 2, ws))):
        L, p, x, want_acc, want = c7 if which == "c7" else l4
        acc, got = gpu_layer(P, L, n, x, p, in_layout=B64, out_layout=B64, split=split)
        assert np.array_equal(acc, want_acc), which
        assert np.array_equal(got, expect_layout(want, B64)), which
    assert int(ws[:64 << 10].to(torch.int32).abs().sum()) == 0
