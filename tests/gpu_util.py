"""Helpers for the GPU parity tests: run one layer through the C ABI and the
same layer through the oracle, on the same seeded inputs."""
import numpy as np

import oracle
from oracle import layout as olayout
from workloads import Conv, layer_params, stack_input

I8, U2, I32, B64 = 0, 1, 2, 3


def device():
    import torch
    return torch.device("cuda:0")


def to_dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a).reshape(-1)).to(device())


def upload_codes(P, codes, layout):
    """Host NHWC codes -> device tensor in `layout` (library converter)."""
    import torch
    src = to_dev(codes.astype(np.uint8))
    if layout == I8:
        return src
    n, h, w, c = codes.shape
    out = torch.empty(n * h * w * c // 4, dtype=torch.uint8, device=device())
    P.ifq_convert_codes(n, h, w, c, I8, layout, src, out)
    return out


def oracle_layer(L, x, p, shortcut=None, down=None):
    """Expected (acc, output) of one layer from the oracle."""
    acc = oracle.conv_acc(x, p["w"], L.stride, L.pad, L.in_bits)
    if L.out_bits == 0:
        return acc, acc
    if L.join is not None:
        if L.join[0] == "identity":
            coef = oracle.join_coeffs("identity", p, p["beta_in"], p["beta_in"])
        else:
            coef = oracle.join_coeffs("conv", p, p["beta_in"], down["beta_in"],
                                      down=down)
        return acc, oracle.join_codes(acc, shortcut.astype(np.int32), coef,
                                      p["q_thr"])
    s, t = oracle.fold(p["alpha"], p["beta_in"], p["mean"], p["var"],
                       p["gamma"], p["bn_beta"], p["eps"], p["q_thr"],
                       L.k * L.k * L.cin, L.in_bits, bias=p["bias"])
    return acc, oracle.codes(acc, s, t)


def gpu_layer(P, L, n, x, p, in_layout=I8, out_layout=None, shortcut=None,
              sc_layout=I8, down=None, dump=True, fused_down=None, variant=None,
              split=None):
    """Run one conv through ifq_conv_forward; returns (acc or None, output).

    output is uint8 codes NHWC (packed [..., c/4] for U2, [n][c/64][h][w][16]
    for B64) or int32 sums. fused_down = (D, xin): a conv join whose 1x1
    downsample layer D (params down) runs inside the kernel on the BLOCK64
    codes xin (IFQ_JOIN_CONV_FUSED) instead of reading its sums. variant:
    run that variant of the register-blocked 3x3 kernel
    (ifq_conv_forward_variant) instead of the kernel ifq_conv_forward picks.
    split = (variant, ksplit, ws): that int8 variant with its contraction
    split over ksplit workgroups (ifq_conv_forward_split) on workspace ws
    (None: a fresh zero-filled one)."""
    import torch
    if out_layout is None:
        out_layout = I32 if L.out_bits == 0 else I8
    d = P.conv_desc(n, L.h, L.w, L.cin, L.cout, L.k, L.stride, L.pad,
                    L.in_bits, L.out_bits, in_layout, out_layout)
    ho, wo = P.ifq_conv_output_dims(d)
    fp4 = variant is not None and P.ifq_conv_variant_fp4(variant) == 1
    blob = P.ifq_pack_weights_fp4(d, p["w"]) if fp4 else P.ifq_pack_weights(d, p["w"])
    wd = to_dev(blob)
    td = None
    join = None
    if L.out_bits != 0 and L.join is None:
        thr = P.ifq_fold_thresholds(L.cout, L.in_bits, L.out_bits,
                                    L.k * L.k * L.cin, p["alpha"], p["beta_in"],
                                    p["q_thr"], bias=p["bias"], mean=p["mean"],
                                    var=p["var"], gamma=p["gamma"],
                                    bn_beta=p["bn_beta"], eps=p["eps"])
        td = to_dev(thr)
    keep = []
    if L.join is not None:
        if L.join[0] == "identity":
            table = P.ifq_fold_join_table(p, p["beta_in"], L.in_bits,
                                          L.k * L.k * L.cin, L.out_bits, p["q_thr"])
            scd = upload_codes(P, shortcut, sc_layout)
            td_ = to_dev(table)
            keep += [scd, td_]
            join = P.make_join(P.IFQ_JOIN_IDENTITY, sc_layout, scd, None,
                               p["q_thr"], table=td_)
        elif fused_down is not None:
            D, xin = fused_down
            coef = P.ifq_fold_join(P.IFQ_JOIN_CONV, p, down["beta_in"], down=down)
            dd = P.conv_desc(n, D.h, D.w, D.cin, D.cout, D.k, D.stride, D.pad,
                             D.in_bits, 0, B64, I32)
            wdd = to_dev(P.ifq_pack_weights_fp4(dd, down["w"]) if fp4 else
                         P.ifq_pack_weights(dd, down["w"]))
            xind = upload_codes(P, xin, B64)
            cd = to_dev(coef)
            keep += [wdd, xind, cd]
            join = P.make_join(P.IFQ_JOIN_CONV_FUSED, B64, xind, cd, p["q_thr"],
                               down_w=wdd, down=dd)
            # the kernel name query sees the join: a fused kernel instance
            # (the windowed kernel's fused flag, or the register-blocked
            # kernel's epilogue mode 2)
            kn = P.ifq_conv_kernel_name(d, join)
            assert ", true, " in kn or (kn.startswith("conv_w2<") and
                                        kn[8:-1].split(", ")[7] == "2"), kn
        else:
            coef = P.ifq_fold_join(P.IFQ_JOIN_CONV, p, down["beta_in"], down=down)
            scd = to_dev(shortcut.astype(np.int32))
            cd = to_dev(coef)
            keep += [scd, cd]
            join = P.make_join(P.IFQ_JOIN_CONV, I32, scd, cd, p["q_thr"])
    xd = upload_codes(P, x, in_layout) if L.in_bits <= 8 else None
    ob = P.ifq_tensor_bytes(n, ho, wo, L.cout, out_layout)
    y = torch.empty(max(ob, 1), dtype=torch.uint8, device=device())
    acc = None
    if dump:
        acc = torch.empty(max(n * ho * wo * L.cout, 1), dtype=torch.int32,
                          device=device())
    if split is not None:
        sv, ks, ws = split
        if ws is None:
            ws = torch.zeros(P.ifq_conv_split_workspace_bytes(d, sv, ks), dtype=torch.uint8,
                             device=device())
        P.ifq_conv_forward_split(d, xd, wd, td, y, sv, ks, ws, acc_dump=acc)
    elif variant is None:
        # a K-split launch needs its workspace, zero-filled before first use
        wsb = P.ifq_conv_workspace_bytes(d)
        ws = torch.zeros(wsb, dtype=torch.uint8, device=device()) if wsb else None
        P.ifq_conv_forward(d, xd, wd, td, y, join=join, acc_dump=acc, ws=ws)
    else:
        name = P.ifq_conv_variant_name(d, join, variant)
        assert name.startswith(("conv_w2<", "conv_wp<", "conv_wv<", "conv_wvh<")), (variant, name)
        assert P.kernel_is_fp4(name) == fp4, (variant, name)
        print("variant %d: %s n=%d %dx%dx%d -> %d s%d" % (variant, name, n, L.h, L.w, L.cin,
                                                          L.cout, L.stride), flush=True)
        P.ifq_conv_forward_variant(d, xd, wd, td, y, variant, join=join, acc_dump=acc)
    torch.cuda.synchronize()
    shape = (n, ho, wo, L.cout)
    acc_h = None if acc is None else acc[:np.prod(shape)].cpu().numpy().reshape(shape)
    if out_layout == I32:
        out = y[:ob].view(torch.int32).cpu().numpy().reshape(shape)
    elif out_layout == U2:
        out = y[:ob].cpu().numpy().reshape(n, ho, wo, L.cout // 4)
    elif out_layout == B64:
        out = y[:ob].cpu().numpy().reshape(n, L.cout // 64, ho, wo, 16)
    else:
        out = y[:ob].cpu().numpy().reshape(shape)
    return acc_h, out


def expect_layout(codes, out_layout):
    """Oracle codes in the byte layout the GPU wrote."""
    if out_layout == U2:
        return olayout.pack2(codes)
    if out_layout == B64:
        return olayout.pack_block64(codes)
    return codes


def make_layer(name, h, w, cin, cout, k, stride, pad, in_bits=2, out_bits=2,
               join=None):
    return Conv(name, "x", "y", h, w, cin, cout, k, stride, pad, in_bits,
                out_bits, join)


def params_for(seed, L, variant="calibrated"):
    return layer_params(1000 + seed, 0, L, variant)


def codes_for(seed, shape, bits):
    return stack_input(1000 + seed, shape, bits)
