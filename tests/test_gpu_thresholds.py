"""GPU parity of the compact thresholds (Sec. 3.2, Eq. 8): records expanded
on the device equal the oracle's expansion, and a conv that reads them gives
the oracle's codes, for 2-, 3- and 4-bit outputs (the 2-bit case on the
windowed kernel, BLOCK64 codes; the others on the generic path)."""
import numpy as np
import pytest

from oracle import compact, core
from gpu_util import I8, B64, expect_layout, make_layer, params_for, codes_for, upload_codes, \
    to_dev, device
from workloads.gen import STEP

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1911_08076_amd as P
    return P


@pytest.mark.parametrize("bits,layout,n,h,cin,cout", [
    (2, B64, 2, 14, 64, 128), (3, I8, 2, 11, 64, 96), (4, I8, 1, 9, 32, 200)])
def test_expanded_thresholds_drive_the_conv(P, bits, layout, n, h, cin, cout):
    import torch
    L = make_layer("cx%d" % bits, h, h, cin, cout, 3, 1, 1, 2, bits)
    p = dict(params_for(50 + bits, L))
    p["gamma"] = np.array(p["gamma"], dtype=np.float64)
    p["gamma"][3] = 0.0
    k = 9 * cin
    recs = P.ifq_fold_thresholds_compact(cout, 2, bits, k, p["alpha"], p["beta_in"], STEP,
                                         -STEP / 2, bias=p["bias"], mean=p["mean"],
                                         var=p["var"], gamma=p["gamma"], bn_beta=p["bn_beta"],
                                         eps=p["eps"])
    recs_d = to_dev(recs.view(np.uint8))
    thr_d = torch.full((cout, 1 << bits), 0x5A5A5A5A, dtype=torch.int32, device=device())
    P.ifq_expand_thresholds(recs_d, cout, 2, k, bits, thr_d)
    torch.cuda.synchronize()
    s, T = compact.expand(compact.fold_compact(p, STEP, -STEP / 2, bits), bits, float(k * 3))
    got = thr_d.cpu().numpy()
    assert np.array_equal(got[:, 0], s) and np.array_equal(got[:, 1:], T)
    assert (s == -1).any()

    x = codes_for(60 + bits, (n, h, h, cin), 2)
    want = core.codes(core.conv_acc(x, p["w"], 1, 1, 2), s, T)
    d = P.conv_desc(n, h, h, cin, cout, 3, 1, 1, 2, bits, layout, layout)
    wd = to_dev(P.ifq_pack_weights(d, p["w"]))
    xd = upload_codes(P, x, layout)
    ob = P.ifq_tensor_bytes(n, h, h, cout, layout)
    y = torch.empty(ob, dtype=torch.uint8, device=device())
    P.ifq_conv_forward(d, xd, wd, thr_d, y)
    torch.cuda.synchronize()
    out = y.cpu().numpy()
    out = out.reshape(n, cout // 64, h, h, 16) if layout == B64 else out.reshape(n, h, h, cout)
    assert np.array_equal(out, expect_layout(want, layout))
    assert len(np.unique(want)) > 2


def _saturating_records(cout, bound, rng):
    """{s, T1, T2, T3} records at and near the ends of [-bound-1, bound]."""
    pats = [[-bound - 1] * 3, [bound] * 3, [-bound - 1, 0, bound], [-bound - 1, -bound - 1, bound],
            [-bound, bound - 1, bound]]
    rec = np.zeros((cout, 4), dtype=np.int32)
    for c in range(cout):
        rec[c, 0] = 1 if (c // 4) % 2 == 0 else -1
        if c % 8 < len(pats):
            rec[c, 1:] = pats[c % 8]
        else:
            rec[c, 1:] = np.sort(rng.integers(-bound - 1, bound + 1, 3))
    return rec


def test_saturated_thresholds_on_a_wide_layer(P):
    # c_in = 1024: |sum| and |T| reach 3*9*1024 = 27648, so T' - sum spans
    # twice the int16 range the packed 2-bit epilogues compare in; sums at
    # both ends (all-3 codes against all +1 / all -1 filters) meet thresholds
    # at both ends, for both signs s
    import torch
    n, h, cin, cout = 2, 6, 1024, 64
    bound = 3 * 9 * cin
    rng = np.random.default_rng(1024)
    w = rng.choice(np.array([-1, 1], dtype=np.int8), size=(cout, cin, 3, 3))
    w[0::4] = 1
    w[1::4] = -1
    x = codes_for(77, (n, h, h, cin), 2)
    x[0] = 3
    rec = _saturating_records(cout, bound, rng)
    acc = core.conv_acc(x, w, 1, 1, 2)
    assert acc.max() == bound and acc.min() == -bound
    want = core.codes(acc, np.ascontiguousarray(rec[:, 0]), np.ascontiguousarray(rec[:, 1:]))
    assert len(np.unique(want)) == 4
    d = P.conv_desc(n, h, h, cin, cout, 3, 1, 1, 2, 2, B64, B64)
    xd = upload_codes(P, x, B64)
    thr_d = to_dev(rec)
    ob = P.ifq_tensor_bytes(n, h, h, cout, B64)
    runs = [("auto", None)] + [(P.ifq_conv_variant_name(d, None, v), v)
                               for v in range(P.ifq_conv_variant_count())
                               if P.ifq_conv_variant_name(d, None, v)]
    assert len(runs) > 1
    for name, v in runs:
        fp4 = v is not None and P.ifq_conv_variant_fp4(v) == 1
        wd = to_dev(P.ifq_pack_weights_fp4(d, w) if fp4 else P.ifq_pack_weights(d, w))
        y = torch.full((ob,), 0x5A, dtype=torch.uint8, device=device())
        print("saturated thresholds:", name, P.ifq_conv_kernel_name(d) if v is None else "",
              flush=True)
        if v is None:
            P.ifq_conv_forward(d, xd, wd, thr_d, y)
        else:
            P.ifq_conv_forward_variant(d, xd, wd, thr_d, y, v)
        torch.cuda.synchronize()
        out = y.cpu().numpy().reshape(n, cout // 64, h, h, 16)
        assert np.array_equal(out, expect_layout(want, B64)), name
