"""Host side of the C ABI, on the CPU: the library loads and exports every
entry point include/ifq.h declares, the weight packer writes the documented
layout, the threshold and join folds equal the oracle's bit for bit (two
separate implementations of the same fixed fp64 order of Sec. 3.2), and every
validation error is returned before anything is launched.

No test here launches a kernel: every device entry point is called only with
arguments its host-side validation rejects.
"""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import oracle
import paper_1911_08076_amd as P
from paper_1911_08076_amd import _ffi
from workloads import get_stack, layer_params, Conv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ifq.h")

OK = 0
EINVAL = -1
EUNSUP = -2
EBUF = -4
I8, U2, I32, B64 = 0, 1, 2, 3


def declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"IFQ_API\s+[\w\s\*]+?\b(ifq_\w+)\s*\(", text)))


def test_header_declares_the_entry_points():
    names = declared_symbols()
    for want in ("ifq_pack_weights", "ifq_fold_thresholds", "ifq_conv_forward",
                 "ifq_maxpool_codes", "ifq_run_stack"):
        assert want in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(_ffi.LIB_PATH)
    names = declared_symbols()
    out = subprocess.run(["nm", "-D", "--defined-only", _ffi.LIB_PATH],
                         capture_output=True, text=True, check=True).stdout
    exported = {l.split()[-1] for l in out.splitlines() if " T " in l}
    for n in names:
        assert n in exported, n
        assert getattr(lib, n) is not None
    # the binding wraps exactly the declared set
    assert sorted(s[0] for s in _ffi.SIGNATURES) == names
    # nothing else with the library's prefix leaks out
    assert {e for e in exported if e.startswith("ifq_")} == set(names)


def test_version_and_no_error_text():
    assert P.ifq_version().endswith("gfx950")
    P.ifq_tensor_bytes(1, 1, 1, 4, U2)


# --- tensor sizes -----------------------------------------------------------

def test_tensor_bytes_of_the_layouts():
    assert P.ifq_tensor_bytes(2, 3, 5, 8, I8) == 240
    assert P.ifq_tensor_bytes(2, 3, 5, 8, U2) == 60
    assert P.ifq_tensor_bytes(2, 3, 5, 8, I32) == 960
    assert P.ifq_tensor_bytes(2, 3, 5, 128, B64) == 960
    assert P.ifq_tensor_bytes(2, 3, 5, 96, B64) == 0    # C % 64 != 0
    assert P.ifq_tensor_bytes(1, 1, 1, 6, U2) == 0     # C % 4 != 0
    assert P.ifq_tensor_bytes(1, 1, 1, 4, 7) == 0      # unknown layout
    assert P.ifq_tensor_bytes(-1, 1, 1, 4, I8) == 0


def test_tensor_bytes_matches_table4_conv1_map():
    # Table 4: the conv1 feature map of IFQ-AlexNet, 55x55x96 at k = 2 bits,
    # is 0.58 Mbit (printed 0.6); the packed layout stores exactly that
    nb = P.ifq_tensor_bytes(1, 55, 55, 96, U2)
    assert nb == 72600
    assert abs(nb * 8 / 1e6 - 0.6) < 0.05


@pytest.mark.parametrize("h,k,s,p,want", [(28, 3, 1, 1, 28), (56, 3, 2, 1, 28),
                                         (56, 1, 2, 0, 28), (27, 5, 1, 2, 27),
                                         (416, 3, 1, 1, 416), (7, 7, 1, 0, 1)])
def test_conv_output_dims(h, k, s, p, want):
    d = P.conv_desc(1, h, h, 16, 16, k, s, p, 2, 2)
    assert P.ifq_conv_output_dims(d) == (want, want)


# --- weight packer ------------------------------------------------------------

def unpack_blob(blob, cout, cin, kh, kw, u2, mfma):
    """Reads W_b back out of a packed blob following the documented layout."""
    k = kh * kw * cin
    kpad = -(-k // 64) * 64
    cpad = -(-cout // (32 if mfma else 16)) * (32 if mfma else 16)
    rows = np.frombuffer(blob[:cpad * kpad].tobytes(), dtype=np.int8)
    rowsum = np.frombuffer(blob[cpad * kpad:cpad * kpad + 4 * cpad].tobytes(),
                           dtype=np.int32)
    w = np.zeros((cout, cin, kh, kw), dtype=np.int8)
    if mfma:
        # [row block of 32][K32 step][lane 32h + r][16 bytes]; byte 4q + i of
        # K32 step 2*kk + t is channel 64g + 32h + 16t + 4i + q of K64 step
        # kk = g*T + tap (T = kh*kw)
        G = cin // 64
        frag = rows.reshape(cpad // 32, kpad // 32, 2, 32, 4, 4)  # rb,k32,h,r,q,i
        for tap in range(kh * kw):
            for g in range(G):
                kk = g * kh * kw + tap
                for t in range(2):
                    blk = frag[:, 2 * kk + t]                     # rb,h,r,q,i
                    for h in range(2):
                        for i in range(4):
                            for q in range(4):
                                c = 64 * g + 32 * h + 16 * t + 4 * i + q
                                col = blk[:, h, :, q, i].reshape(-1)[:cout]
                                w[:, c, tap // kw, tap % kw] = col
        mat = frag.transpose(0, 3, 1, 2, 4, 5).reshape(cpad, -1)
    else:
        mat = rows.reshape(cpad, kpad)
        for r_ in range(kh):
            for s_ in range(kw):
                for c in range(cin):
                    cp = c
                    if u2:
                        base, i = c & ~15, c & 15
                        cp = base + (i & 3) * 4 + (i >> 2)
                    w[:, c, r_, s_] = mat[:cout, (r_ * kw + s_) * cin + cp]
    return w, mat, rowsum, k, cpad


@pytest.mark.parametrize("shape,layout", [
    ((64, 64, 3, 3), I8), ((64, 64, 3, 3), U2), ((30, 512, 1, 1), I8),
    ((16, 3, 3, 3), I8), ((256, 96, 5, 5), I8), ((128, 192, 3, 3), U2),
    ((48, 32, 3, 3), U2), ((7, 16, 3, 3), I8), ((96, 128, 3, 3), B64),
    ((40, 64, 1, 1), B64), ((64, 256, 5, 5), B64)])
def test_pack_weights_layout(shape, layout, rng):
    cout, cin, kh, kw = shape
    w = (rng.integers(0, 2, size=shape, dtype=np.int8) * 2 - 1).astype(np.int8)
    d = P.conv_desc(1, 9, 9, cin, cout, kh, 1, kh // 2, 2, 2, layout,
                    kw=kw)
    blob = P.ifq_pack_weights(d, w)
    assert blob.nbytes == P.ifq_packed_weight_bytes(d)
    mfma = layout in (U2, B64) and cin % 64 == 0
    back, mat, rowsum, k, cpad = unpack_blob(blob, cout, cin, kh, kw,
                                             layout == U2, mfma)
    assert np.array_equal(back, w)
    # every stored +-1 is one of the layer's weights; padding is zero
    assert np.count_nonzero(mat) == w.size
    assert np.array_equal(rowsum[:cout], w.reshape(cout, -1).sum(1))
    assert not rowsum[cout:].any()
    # the trailing zero block the kernels read for out-of-range fragments
    assert not blob[-1024:].any()


def test_pack_rejects_non_binary_weight_and_leaves_dst(rng):
    d = P.conv_desc(1, 8, 8, 16, 16, 3, 1, 1, 2, 2)
    w = np.ones((16, 16, 3, 3), dtype=np.int8)
    w[3, 2, 1, 0] = 0
    dst = np.full(P.ifq_packed_weight_bytes(d), 0x5A, dtype=np.uint8)
    with pytest.raises(P.IfqError) as e:
        P.ifq_pack_weights(d, w, dst)
    assert e.value.status == EINVAL
    assert (dst == 0x5A).all()


def test_pack_rejects_small_buffer():
    d = P.conv_desc(1, 8, 8, 16, 16, 3, 1, 1, 2, 2)
    w = np.ones((16, 16, 3, 3), dtype=np.int8)
    dst = np.zeros(P.ifq_packed_weight_bytes(d) - 1, dtype=np.uint8)
    with pytest.raises(P.IfqError) as e:
        P.ifq_pack_weights(d, w, dst)
    assert e.value.status == EBUF


# --- threshold fold: library vs oracle ---------------------------------------

def lib_fold(p, k, in_bits, out_bits=2):
    return P.ifq_fold_thresholds(len(p["alpha"]), in_bits, out_bits, k,
                                 p["alpha"], p["beta_in"], p["q_thr"],
                                 bias=p["bias"], mean=p["mean"], var=p["var"],
                                 gamma=p["gamma"], bn_beta=p["bn_beta"],
                                 eps=p["eps"])


def orc_fold(p, k, in_bits):
    return oracle.fold(p["alpha"], p["beta_in"], p["mean"], p["var"], p["gamma"],
                       p["bn_beta"], p["eps"], p["q_thr"], k, in_bits,
                       bias=p["bias"])


@pytest.mark.parametrize("cfg", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("variant", ["plain", "calibrated"])
def test_fold_equals_oracle_on_every_stack_layer(cfg, variant):
    layers = get_stack(cfg).layers
    n = 0
    for i, L in enumerate(layers):
        if not isinstance(L, Conv) or L.out_bits == 0:
            continue
        p = layer_params(cfg, i, L, variant)
        k = L.k * L.k * L.cin
        rec = lib_fold(p, k, L.in_bits, L.out_bits)
        s, t = orc_fold(p, k, L.in_bits)
        assert np.array_equal(rec[:, 0], s)
        assert np.array_equal(rec[:, 1:], t)
        n += 1
    assert n >= 1


def edge_params(rng, c=64):
    p = dict(alpha=rng.uniform(0.01, 0.1, c), bias=rng.normal(0, 0.3, c),
             mean=rng.normal(0, 2, c), var=rng.uniform(0.5, 2, c),
             gamma=rng.uniform(0.5, 1.5, c), bn_beta=rng.normal(0, 1, c),
             eps=1e-5, beta_in=0.5, q_thr=np.array([0.25, 0.75, 1.25]))
    p["gamma"][:8] *= -1          # flipped channels
    p["gamma"][8:10] = 0.0        # constant-code channels
    p["bn_beta"][8] = 1.0         # constant code 2
    p["bn_beta"][9] = -3.0        # constant code 0
    # channels whose thresholds land exactly on integers: with var+eps = 1,
    # gamma = 1, bn_beta = 0, alpha*beta = 1/4 and mean = m, t_i = 4*(q_i + m)
    for c_ in (10, 11):
        p["alpha"][c_] = 0.5
        p["var"][c_] = 1.0 - 1e-5
        p["gamma"][c_] = 1.0 if c_ == 10 else -1.0
        p["bn_beta"][c_] = 0.0
        p["mean"][c_] = 0.75
        p["bias"][c_] = 0.0
    p["alpha"][12] = 1e-6        # thresholds far outside the reachable sums
    return p


def test_fold_edge_cases_equal_oracle(rng):
    p = edge_params(rng)
    k = 576
    rec = lib_fold(p, k, 2)
    s, t = orc_fold(p, k, 2)
    assert np.array_equal(rec[:, 0], s)
    assert np.array_equal(rec[:, 1:], t)
    bound = k * 3
    # gamma == 0: the constant code #{i : bn_beta > q_i}
    acc = np.arange(-bound, bound + 1, dtype=np.int64)
    for c_, want in ((8, 2), (9, 0)):
        sv = rec[c_, 0] * acc
        code = sum((sv > rec[c_, i]).astype(int) for i in (1, 2, 3))
        assert (code == want).all()
    # integer-valued thresholds (t_i = 3 + 4 q_i for gamma = 1, 3 - 4 q_i for
    # gamma = -1): a sum that lands exactly on one makes Y_bn equal q_i, and
    # Eq. (3) sends that tie to the lower code in both directions
    assert list(rec[10, 1:]) == [4, 6, 8]
    assert list(rec[11, 1:]) == [-2, 0, 2]
    for c_, ties in ((10, (4, 6, 8)), (11, (2, 0, -2))):
        for i, a in enumerate(ties):
            sv = rec[c_, 0] * a
            code = sum(int(sv > rec[c_, j]) for j in (1, 2, 3))
            ybn = p["gamma"][c_] * (0.25 * a - 0.75)
            assert code == sum(int(ybn > q) for q in p["q_thr"])
            assert ybn == p["q_thr"][i]
    # clamped to [-B-1, B]
    assert rec[12, 1:].min() >= -bound - 1 and rec[12, 1:].max() <= bound


@pytest.mark.parametrize("field,value", [
    ("alpha", 0.0), ("alpha", -0.1), ("alpha", np.nan), ("var", -2.0),
    ("gamma", np.nan), ("mean", np.inf), ("bn_beta", np.nan)])
def test_fold_rejects_bad_channel(field, value, rng):
    p = edge_params(rng, 16)
    p[field] = p[field].copy()
    p[field][3] = value
    with pytest.raises(P.IfqError) as e:
        lib_fold(p, 576, 2)
    assert e.value.status == EINVAL


@pytest.mark.parametrize("q", [[0.25, 0.25, 1.25], [0.75, 0.25, 1.25],
                               [0.25, np.nan, 1.25]])
def test_fold_rejects_bad_quantizer(q, rng):
    p = edge_params(rng, 16)
    p["q_thr"] = np.array(q)
    with pytest.raises(P.IfqError):
        lib_fold(p, 576, 2)


def test_fold_rejects_bad_beta_and_bits(rng):
    p = edge_params(rng, 16)
    p["beta_in"] = 0.0
    with pytest.raises(P.IfqError):
        lib_fold(p, 576, 2)
    p = edge_params(rng, 16)
    with pytest.raises(P.IfqError):
        lib_fold(p, 576, 9)
    with pytest.raises(P.IfqError):
        lib_fold(p, 576, 2, out_bits=5)


# --- join fold: library vs oracle ----------------------------------------------

@pytest.mark.parametrize("variant", ["plain", "calibrated"])
def test_join_coefficients_equal_oracle(variant):
    layers = get_stack(3).layers
    names = {L.name: i for i, L in enumerate(layers)}
    n = 0
    for i, L in enumerate(layers):
        if not isinstance(L, Conv) or L.join is None:
            continue
        p = layer_params(3, i, L, variant)
        if L.join[0] == "identity":
            got = P.ifq_fold_join(P.IFQ_JOIN_IDENTITY, p, p["beta_in"])
            want = oracle.join_coeffs("identity", p, p["beta_in"], p["beta_in"])
        else:
            j = names[L.join[2]]
            pd = layer_params(3, j, layers[j], variant)
            got = P.ifq_fold_join(P.IFQ_JOIN_CONV, p, pd["beta_in"], down=pd)
            want = oracle.join_coeffs("conv", p, p["beta_in"], pd["beta_in"],
                                      down=pd)
        assert np.array_equal(got.view(np.uint64), want.view(np.uint64))
        n += 1
    assert n == 8


@pytest.mark.parametrize("variant", ["plain", "calibrated"])
def test_join_table_equals_oracle_fp64_join(variant):
    # the integer records reproduce the fp64 join for every reachable sum
    # and every shortcut code, on every identity join of the ResNet stack
    layers = get_stack(3).layers
    n = 0
    for i, L in enumerate(layers):
        if not isinstance(L, Conv) or L.join is None or L.join[0] != "identity":
            continue
        p = layer_params(3, i, L, variant)
        k = L.k * L.k * L.cin
        bound = k * 3
        table = P.ifq_fold_join_table(p, p["beta_in"], 2, k, 2, p["q_thr"])
        coef = oracle.join_coeffs("identity", p, p["beta_in"], p["beta_in"])
        a = np.arange(-bound, bound + 1, dtype=np.int64)
        for x in range(4):
            acc = np.ascontiguousarray(np.broadcast_to(a[:, None], (a.size, L.cout)),
                                       dtype=np.int32)
            sc = np.full(acc.shape, x, dtype=np.int32)
            want = oracle.join_codes(acc, sc, coef, p["q_thr"]).astype(np.int64)
            rec = table[:, x, :]
            got = ((rec[None, :, 0] * acc)[..., None] > rec[None, :, 1:]).sum(-1)
            assert np.array_equal(got, want), (L.name, x)
        n += 1
    assert n == 5


def test_join_table_edge_cases(rng):
    c = 8
    p = dict(alpha=rng.uniform(0.01, 0.1, c), bias=np.zeros(c),
             mean=rng.normal(0, 2, c), var=rng.uniform(0.5, 2, c),
             gamma=rng.uniform(0.5, 1.5, c), bn_beta=rng.normal(0, 1, c),
             eps=1e-5, beta_in=0.5)
    p["gamma"][0] = -0.7          # decreasing in a: s = -1
    p["gamma"][1] = 0.0           # constant in a
    p["bn_beta"][2] = 50.0        # always the top code
    p["bn_beta"][3] = -50.0       # always code 0
    q = np.array([0.25, 0.75, 1.25])
    k = 64
    table = P.ifq_fold_join_table(p, 0.5, 2, k, 2, q)
    coef = oracle.join_coeffs("identity", p, 0.5, 0.5)
    assert (table[0, :, 0] == -1).all() and (table[1:, :, 0] == 1).all()
    a = np.arange(-3 * k, 3 * k + 1, dtype=np.int32)
    for x in range(4):
        acc = np.ascontiguousarray(np.broadcast_to(a[:, None], (a.size, c)))
        want = oracle.join_codes(acc, np.full(acc.shape, x, np.int32), coef, q)
        rec = table[:, x, :]
        got = ((rec[None, :, 0] * acc)[..., None] > rec[None, :, 1:]).sum(-1)
        assert np.array_equal(got, want)
    assert (table[2, :, 1:] == -3 * k - 1).all() and (table[3, :, 1:] == 3 * k).all()
    with pytest.raises(P.IfqError):
        P.ifq_fold_join_table(p, 0.5, 2, k, 2, np.array([0.75, 0.25, 1.25]))
    with pytest.raises(P.IfqError):
        P.ifq_fold_join_table(p, 0.5, 2, 0, 2, q)


def test_join_rejects_bad_kind_and_alpha():
    L = get_stack(3).layers[1]
    p = layer_params(3, 1, L)
    with pytest.raises(P.IfqError):
        P.ifq_fold_join(7, p, 0.5)
    q = dict(p)
    q["alpha"] = p["alpha"].copy()
    q["alpha"][0] = -1.0
    with pytest.raises(P.IfqError):
        P.ifq_fold_join(P.IFQ_JOIN_IDENTITY, q, 0.5)


# --- validation of device entry points (nothing is launched) -------------------

def status_of(fn, *args):
    lib = _ffi.load()
    return getattr(lib, fn)(*args)


FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first


@pytest.mark.parametrize("desc,want", [
    (dict(n=-1), EINVAL), (dict(h=0), EINVAL), (dict(c_in=0), EINVAL),
    (dict(kh=0), EINVAL), (dict(stride=0), EINVAL), (dict(pad=-1), EINVAL),
    (dict(h=2, pad=0), EINVAL),                       # filter larger than input
    (dict(in_bits=9), EINVAL), (dict(out_bits=5), EINVAL),
    (dict(in_layout=U2, in_bits=8), EINVAL),
    (dict(in_layout=U2, c_in=6), EINVAL),
    (dict(in_layout=U2, c_in=20), EUNSUP),             # C % 16 for packed input
    (dict(in_layout=5), EINVAL),
    (dict(in_layout=B64, c_in=96), EINVAL),           # BLOCK64 needs C % 64
    (dict(in_layout=B64, in_bits=4), EINVAL),
    (dict(out_layout=B64, c_out=96), EINVAL),
    (dict(out_layout=B64, out_bits=4), EINVAL),
    (dict(out_bits=0, out_layout=I8), EINVAL),
    (dict(out_layout=U2, out_bits=4), EINVAL),
    (dict(out_layout=U2, c_out=30), EINVAL),
    (dict(out_layout=I32), EINVAL),
    (dict(n=100000, h=224, w=224, c_in=64), EUNSUP),    # 2^31-byte tensors
])
def test_conv_forward_rejects_bad_desc(desc, want):
    base = dict(n=1, h=8, w=8, c_in=64, c_out=64, kh=3, kw=3, stride=1, pad=1,
                in_bits=2, out_bits=2, in_layout=I8, out_layout=I8)
    base.update(desc)
    d = _ffi.ConvDesc(**base)
    st = status_of("ifq_conv_forward", ctypes.byref(d), FAKE, FAKE, FAKE, None,
                   FAKE, None, None, 0, None)
    assert st == want
    assert P.ifq_last_error() != ""
    assert P.ifq_packed_weight_bytes(d) == 0


def test_conv_forward_rejects_bad_pointers():
    d = P.conv_desc(1, 8, 8, 64, 64, 3, 1, 1, 2, 2)
    # thresholds required for a code output, forbidden for an int32 output
    st = status_of("ifq_conv_forward", ctypes.byref(d), FAKE, FAKE, None, None,
                   FAKE, None, None, 0, None)
    assert st == EINVAL
    d0 = P.conv_desc(1, 8, 8, 64, 64, 3, 1, 1, 2, 0)
    st = status_of("ifq_conv_forward", ctypes.byref(d0), FAKE, FAKE, FAKE, None,
                   FAKE, None, None, 0, None)
    assert st == EINVAL
    st = status_of("ifq_conv_forward", ctypes.byref(d), None, FAKE, FAKE, None,
                   FAKE, None, None, 0, None)
    assert st == EINVAL


def test_conv_forward_rejects_bad_join():
    d = P.conv_desc(1, 8, 8, 64, 64, 3, 1, 1, 2, 2)
    coef = np.zeros((64, 3))
    table = np.zeros((64, 4, 4), dtype=np.int32)
    # each join has what its kind needs, so it fails for the listed reason
    for kind, layout, q, want in [
            (9, I8, [0.25, 0.75, 1.25], EINVAL),
            (P.IFQ_JOIN_IDENTITY, I32, [0.25, 0.75, 1.25], EINVAL),
            (P.IFQ_JOIN_CONV, I8, [0.25, 0.75, 1.25], EINVAL),
            (P.IFQ_JOIN_IDENTITY, I8, [0.25, 0.75], EINVAL),
            (P.IFQ_JOIN_IDENTITY, I8, [0.75, 0.25, 1.25], EINVAL)]:
        j = P.make_join(kind, layout, None, coef, q, table=table)
        j.shortcut = 0x1000
        st = status_of("ifq_conv_forward", ctypes.byref(d), FAKE, FAKE, None,
                       ctypes.byref(j), FAKE, None, None, 0, None)
        assert st == want, (kind, layout, q)
    # a join with thresholds given as well
    j = P.make_join(P.IFQ_JOIN_IDENTITY, I8, None, None, [0.25, 0.75, 1.25],
                    table=table)
    j.shortcut = 0x1000
    st = status_of("ifq_conv_forward", ctypes.byref(d), FAKE, FAKE, FAKE,
                   ctypes.byref(j), FAKE, None, None, 0, None)
    assert st == EINVAL
    # an identity join without its table, a conv join without coefficients
    for kind, layout in ((P.IFQ_JOIN_IDENTITY, I8), (P.IFQ_JOIN_CONV, I32)):
        j = P.make_join(kind, layout, None, None, [0.25, 0.75, 1.25])
        j.shortcut = 0x1000
        st = status_of("ifq_conv_forward", ctypes.byref(d), FAKE, FAKE, None,
                       ctypes.byref(j), FAKE, None, None, 0, None)
        assert st == EINVAL


@pytest.mark.parametrize("pool,want", [
    (dict(k=0), EINVAL), (dict(stride=0), EINVAL), (dict(mode=3), EINVAL),
    (dict(k=9), EINVAL), (dict(layout=U2, c=6), EINVAL),
    (dict(layout=U2, bits=8), EINVAL), (dict(bits=0), EINVAL),
    (dict(layout=I32), EINVAL), (dict(layout=B64, c=32), EINVAL)])
def test_maxpool_rejects_bad_desc(pool, want):
    base = dict(n=1, h=8, w=8, c=16, k=2, stride=2, mode=0, bits=2, layout=I8)
    base.update(pool)
    d = _ffi.PoolDesc(**base)
    st = status_of("ifq_maxpool_codes", ctypes.byref(d), FAKE, FAKE, None)
    assert st == want


@pytest.mark.parametrize("pool,want", [
    (dict(h=18), EINVAL),                     # not the conv's output
    (dict(c=32), EINVAL),
    (dict(n=3), EINVAL),
    (dict(layout=U2), EINVAL),                # not the conv's layout
    (dict(bits=4), EINVAL),
    # windows that need whole images per tile, which 20x20 outputs
    # (400 pixels) do not fit: not covered
    (dict(k=3, stride=2), EUNSUP),            # overlapping windows
    (dict(mode=1), EUNSUP),                   # same mode
    (dict(k=3, stride=3), EUNSUP),            # 20 is no multiple of 3
    (dict(k=0), EINVAL)])
def test_conv_pool_rejects_inconsistent_pair(pool, want):
    d = P.conv_desc(2, 20, 20, 64, 64, 3, 1, 1, 2, 2, B64, B64)
    base = dict(n=2, h=20, w=20, c=64, k=2, stride=2, mode=0, bits=2, layout=B64)
    base.update(pool)
    pd = _ffi.PoolDesc(**base)
    assert P.ifq_conv_pool_kernel_name(d, pd) == ""
    st = status_of("ifq_conv_pool_forward", ctypes.byref(d), ctypes.byref(pd), FAKE,
                   FAKE, FAKE, FAKE, None)
    assert st == want


def test_conv_pool_kernel_choice():
    # the pair fuses in the windowed 3x3 kernel (BLOCK64 input) and in the
    # 8-bit first-layer kernel; other inputs have no fused kernel
    pd = lambda n, h, c, lay: _ffi.PoolDesc(n, h, h, c, 2, 2, 0, 2, lay)
    d = P.conv_desc(2, 28, 28, 256, 256, 3, 1, 1, 2, 2, B64, B64)
    assert P.ifq_conv_pool_kernel_name(d, pd(2, 28, 256, B64)).startswith("conv_halo<")
    d = P.conv_desc(2, 64, 64, 3, 16, 3, 1, 1, 8, 2, I8, U2)
    assert P.ifq_conv_pool_kernel_name(d, pd(2, 64, 16, U2)).startswith("conv_small8<")
    d = P.conv_desc(2, 28, 28, 256, 256, 3, 1, 1, 2, 2, U2, U2)
    assert P.ifq_conv_pool_kernel_name(d, pd(2, 28, 256, U2)) == ""
    assert status_of("ifq_conv_pool_forward", ctypes.byref(d),
                     ctypes.byref(pd(2, 28, 256, U2)), FAKE, FAKE, FAKE, FAKE, None) == EUNSUP
    # a tile cannot hold two rows of 224 pixels: not covered
    d = P.conv_desc(1, 224, 224, 64, 64, 3, 1, 1, 2, 2, B64, B64)
    assert P.ifq_conv_pool_kernel_name(d, pd(1, 224, 64, B64)) == ""
    # overlapping and SAME windows on 13x13 outputs: whole images per tile
    d = P.conv_desc(3, 13, 13, 384, 256, 3, 1, 1, 2, 2, B64, B64)
    p3 = _ffi.PoolDesc(3, 13, 13, 256, 3, 2, 0, 2, B64)
    assert P.ifq_conv_pool_kernel_name(d, p3).startswith("conv_halo<")
    d = P.conv_desc(2, 13, 13, 256, 512, 3, 1, 1, 2, 2, B64, B64)
    p2 = _ffi.PoolDesc(2, 13, 13, 512, 2, 1, 1, 2, B64)
    assert P.ifq_conv_pool_kernel_name(d, p2).startswith("conv_halo<")


def test_convert_rejects_bad_args():
    cv = lambda *a: status_of("ifq_convert_codes", *a)
    assert cv(1, 1, 10, 6, I8, U2, FAKE, FAKE, None) == EINVAL     # C % 4
    assert cv(1, 1, 10, 8, I8, I8, FAKE, FAKE, None) == EINVAL     # same layout
    assert cv(1, 1, 10, 8, I8, I32, FAKE, FAKE, None) == EINVAL    # not codes
    assert cv(1, 1, 10, 96, I8, B64, FAKE, FAKE, None) == EINVAL   # C % 64
    assert cv(1, 1, 10, 8, I8, U2, None, FAKE, None) == EINVAL
    assert cv(-1, 1, 10, 8, I8, U2, FAKE, FAKE, None) == EINVAL


# --- stack planning -------------------------------------------------------------

def make_stack(layers, batch=1, layout="i8"):
    """ifq_stack of fake device pointers (planning and validation only)."""
    slots = {"x": 0, "y": 1}
    lay_of = {}
    arr = (_ffi.Layer * len(layers))()
    for i, L in enumerate(layers):
        for s in (L.src, L.dst):
            slots.setdefault(s, len(slots))
        rec = arr[i]
        rec.src, rec.dst, rec.join_src = slots[L.src], slots[L.dst], -1
        lin = lay_of.get(L.src, U2 if layout == "u2" else I8)
        if isinstance(L, Conv):
            lout = I32 if L.out_bits == 0 else (U2 if layout == "u2" else I8)
            rec.kind = P.IFQ_LAYER_CONV
            rec.conv = P.conv_desc(batch, L.h, L.w, L.cin, L.cout, L.k, L.stride,
                                   L.pad, L.in_bits, L.out_bits, lin, lout)
            rec.w_packed = 0x1000
            if L.join is None and L.out_bits:
                rec.thr = 0x1000
            if L.join is not None:
                rec.join = P.make_join(
                    P.IFQ_JOIN_IDENTITY if L.join[0] == "identity" else P.IFQ_JOIN_CONV,
                    lay_of.get(L.join[1], lin) if L.join[0] == "identity" else I32,
                    None, None, L.out_bits and [0.25, 0.75, 1.25])
                rec.join.coef = 0x1000
                rec.join.table = 0x1000
                rec.join_src = slots[L.join[1]]
        else:
            lout = lin
            rec.kind = P.IFQ_LAYER_POOL
            rec.pool = P.pool_desc(batch, L.h, L.w, L.c, L.k, L.stride,
                                   0 if L.mode == "valid" else 1, L.bits, lin)
        lay_of[L.dst] = lout
    st = _ffi.Stack(len(layers), len(slots),
                    ctypes.cast(arr, ctypes.POINTER(_ffi.Layer)), None)
    st._keep = arr
    return st, slots


@pytest.mark.parametrize("cfg", [0, 1, 2, 3, 4])
def test_stack_workspace_covers_every_slot(cfg):
    layers = get_stack(cfg).layers
    for layout in ("i8", "u2"):
        st, slots = make_stack(layers, 2, "i8" if cfg == 4 else layout)
        total = P.ifq_stack_workspace_bytes(st)
        spans = []
        for name, k in slots.items():
            if k < 2:
                continue
            off, nb = P.ifq_stack_slot_info(st, k)
            assert off % 256 == 0 and off + nb <= total
            spans.append((off, off + nb))
        spans.sort()
        for (a0, a1), (b0, b1) in zip(spans, spans[1:]):
            assert a1 <= b0  # slots do not overlap


def test_stack_rejects_unwritten_slot_and_small_workspace():
    layers = list(get_stack(1).layers)
    st, _ = make_stack(layers)
    total = P.ifq_stack_workspace_bytes(st)
    assert total > 0
    lib = _ffi.load()
    assert lib.ifq_run_stack(ctypes.byref(st), FAKE, FAKE, FAKE, total - 1,
                             None) == EBUF
    # layer 2 reads a slot nobody wrote
    st.layers[2].src = st.n_slots - 1
    st.layers[1].dst = 3
    assert P.ifq_stack_workspace_bytes(st) == 0
    assert lib.ifq_run_stack(ctypes.byref(st), FAKE, FAKE, FAKE, 1 << 30,
                             None) == EINVAL


def test_stack_rejects_bad_layer_kind_and_slots():
    layers = list(get_stack(0).layers)
    st, _ = make_stack(layers)
    lib = _ffi.load()
    st.layers[0].kind = 5
    assert lib.ifq_run_stack(ctypes.byref(st), FAKE, FAKE, FAKE, 1 << 20,
                             None) == EINVAL
    st, _ = make_stack(layers)
    st.layers[0].dst = 0          # writing the input slot
    assert lib.ifq_run_stack(ctypes.byref(st), FAKE, FAKE, FAKE, 1 << 20,
                             None) == EINVAL


def test_identity_join_needs_2bit_shortcut_codes():
    # the identity join's table has 4 shortcut levels and the kernels read 2
    # bits per shortcut code: wider shortcut codes are refused, not misread
    d = P.conv_desc(1, 8, 8, 64, 64, 3, 1, 1, 2, 2)
    table = np.zeros((64, 4, 4), dtype=np.int32)
    for sc_bits, want in ((0, None), (2, None), (1, EUNSUP), (3, EUNSUP), (4, EUNSUP),
                          (8, EUNSUP)):
        j = P.make_join(P.IFQ_JOIN_IDENTITY, I8, None, None, [0.25, 0.75, 1.25], table=table)
        j.shortcut = 0x1000
        j.sc_bits = sc_bits
        name = P.ifq_conv_kernel_name(d, j)
        st = status_of("ifq_conv_forward", ctypes.byref(P.conv_desc(0, 8, 8, 64, 64, 3, 1, 1,
                                                                    2, 2)),
                       FAKE, FAKE, None, ctypes.byref(j), FAKE, None, None, 0, None)
        if want is None:
            assert st == 0 and name
        else:
            assert st == want, sc_bits


def test_stack_rejects_a_join_slot_smaller_than_the_join_reads():
    # s2 holds a 4x4 map (a stride-2 conv's output); the identity join of the
    # last layer reads an 8x8 map of the same channels from it
    layers = [Conv("a", "x", "s2", 8, 8, 64, 64, 3, 2, 1, 2, 2),
              Conv("b", "x", "s3", 8, 8, 64, 64, 3, 1, 1, 2, 2),
              Conv("c", "s3", "y", 8, 8, 64, 64, 3, 1, 1, 2, 2, ("identity", "s2"))]
    st, slots = make_stack(layers, 2)
    lib = _ffi.load()
    assert P.ifq_stack_workspace_bytes(st) == 0
    assert lib.ifq_run_stack(ctypes.byref(st), FAKE, FAKE, FAKE, 1 << 30, None) == EINVAL
    assert "join reads" in P.ifq_last_error()
    # the same stack with the join on the 8x8 map plans
    layers[2] = Conv("c", "s3", "y", 8, 8, 64, 64, 3, 1, 1, 2, 2, ("identity", "s3"))
    st, slots = make_stack(layers[1:], 2)
    assert P.ifq_stack_workspace_bytes(st) > 0


def test_stack_rejects_identity_shortcut_of_wider_codes():
    # s2 holds 3-bit codes (byte per code); an identity join reading it would
    # see only their low 2 bits, so the stack is refused
    def layers(bits):
        return [Conv("a", "x", "s2", 8, 8, 64, 64, 3, 1, 1, 2, bits),
                Conv("b", "s2", "s3", 8, 8, 64, 64, 3, 1, 1, bits, 2),
                Conv("c", "s3", "y", 8, 8, 64, 64, 3, 1, 1, 2, 2, ("identity", "s2"))]
    lib = _ffi.load()
    st, _ = make_stack(layers(2), 2)
    assert P.ifq_stack_workspace_bytes(st) > 0
    st, _ = make_stack(layers(3), 2)
    assert P.ifq_stack_workspace_bytes(st) == 0
    assert lib.ifq_run_stack(ctypes.byref(st), FAKE, FAKE, FAKE, 1 << 30, None) == EUNSUP
    assert "2-bit only" in P.ifq_last_error()


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_compact_fold_matches_oracle(bits):
    # the library's host fold of the compact records (Eq. 8) and the
    # oracle's, written separately, agree to the last bit
    from oracle import compact
    from workloads import Conv, layer_params
    from workloads.gen import STEP
    L = Conv("cf", "x", "y", 9, 9, 64, 96, 3, 1, 1, 2, bits, None)
    p = dict(layer_params(77, 0, L, "calibrated"))
    p["gamma"] = np.array(p["gamma"], dtype=np.float64)
    p["gamma"][5] = 0.0                      # the constant-code case
    got = P.ifq_fold_thresholds_compact(L.cout, 2, bits, 9 * L.cin, p["alpha"], p["beta_in"],
                                        STEP, -STEP / 2, bias=p["bias"], mean=p["mean"],
                                        var=p["var"], gamma=p["gamma"], bn_beta=p["bn_beta"],
                                        eps=p["eps"])
    want = compact.fold_compact(p, STEP, -STEP / 2, bits)
    for f in ("base", "offset", "s", "cstar"):
        assert np.array_equal(got[f], want[f]), f
    assert (got["s"] == -1).any() and got["s"][5] == 0


def test_compact_fold_rejects_bad_quantizer():
    a = np.ones(4)
    for base, offset in ((0.0, 0.0), (-0.5, 0.0), (float("nan"), 0.0), (0.5, float("inf"))):
        with pytest.raises(P.IfqError):
            P.ifq_fold_thresholds_compact(4, 2, 2, 9, a, 0.5, base, offset)
    st = status_of("ifq_expand_thresholds", FAKE, 0, 2, 9, 2, FAKE, None)
    assert st == EINVAL
    st = status_of("ifq_expand_thresholds", FAKE, 4, 2, 9, 5, FAKE, None)
    assert st == EINVAL


def test_fp4_entry_points_host_side():
    # the fp4 path covers the 3x3 kernels' 2-bit threshold and join layers
    # only (fp4 instances: the register-blocked kernel's ninth template
    # argument, the windowed kernel's last)
    d = P.conv_desc(2, 28, 28, 128, 128, 3, 1, 1, 2, 2, B64, B64)
    name = P.ifq_conv_fp4_kernel_name(d)
    assert name.startswith(("conv_w2<", "conv_wp<", "conv_wv<", "conv_wvh<")) and P.kernel_is_fp4(name), name
    k = 9 * 128
    assert P._ffi.load().ifq_packed_weight_bytes_fp4(ctypes.byref(d)) == (128 // 32) * (k // 64) * 1024 + 1024
    w = np.ones((128, 128, 3, 3), dtype=np.int8)
    blob = P.ifq_pack_weights_fp4(d, w)
    # +2.0 is the e2m1 nibble 0x4 in every used position, the zero block stays 0
    assert set(np.unique(blob[:-1024])) == {0x44} and not blob[-1024:].any()
    w[0, 0, 0, 0] = 3
    with pytest.raises(P.IfqError):
        P.ifq_pack_weights_fp4(d, w)
    # int32 output, byte-code input, 8-bit input: no fp4 kernel
    for dd in (P.conv_desc(2, 28, 28, 128, 128, 3, 1, 1, 2, 0, B64, I32),
               P.conv_desc(2, 28, 28, 128, 128, 3, 1, 1, 2, 2, I8, I8)):
        assert P.ifq_conv_fp4_kernel_name(dd) == ""
    d8 = P.conv_desc(2, 28, 28, 128, 128, 3, 1, 1, 2, 2, I8, I8)
    assert status_of("ifq_conv_forward_fp4", ctypes.byref(d8), FAKE, FAKE, FAKE, None, FAKE,
                     None) == EUNSUP


def test_new_entry_points_accept_an_empty_batch():
    # n = 0: validated, then nothing to launch (no tensor pointer is needed;
    # the thresholds are, as for ifq_conv_forward, and never dereferenced)
    d = P.conv_desc(0, 28, 28, 128, 128, 3, 1, 1, 2, 2, B64, B64)
    pd = _ffi.PoolDesc(0, 28, 28, 128, 2, 2, 0, 2, B64)
    assert status_of("ifq_conv_pool_forward", ctypes.byref(d), ctypes.byref(pd), None, None,
                     FAKE, None, None) == OK
    assert status_of("ifq_conv_forward_fp4", ctypes.byref(d), None, None, FAKE, None, None,
                     None) == OK
    # the pool must still describe the conv's output
    bad = _ffi.PoolDesc(0, 27, 28, 128, 2, 2, 0, 2, B64)
    assert status_of("ifq_conv_pool_forward", ctypes.byref(d), ctypes.byref(bad), None, None,
                     FAKE, None, None) == EINVAL


def test_run_stack_static_host_side():
    # the static-workspace driver validates before touching the GPU: a NULL
    # stack and a stack needing more than the static workspace are refused
    lib = _ffi.load()
    cap = P.ifq_static_workspace_bytes()
    assert cap == 64 << 20
    assert lib.ifq_run_stack_static(None, FAKE, FAKE, None) == EINVAL
    st, _ = make_stack(list(get_stack(3).layers), 64, "i8")
    assert P.ifq_stack_workspace_bytes(st) > cap
    assert lib.ifq_run_stack_static(ctypes.byref(st), FAKE, FAKE, None) == EBUF
    assert "static workspace" in P.ifq_last_error()


# ---------------------------------------------------------------------------
# K split across workgroups: workspace sizing and host-side checks (the
# launches themselves are GPU tests)
B64L = P.IFQ_LAYOUT_U2_BLOCK64


def test_split_workspace_sizes():
    # the planner prices a split with its measured cost (a device-scope
    # fence per workgroup), above the unsplit launch of every benchmark
    # layer, even the detector's 13x13 512->512 layers that fill 88 of 256
    # CUs: no workspace is asked for
    for shape in ((8, 13, 13, 512, 512), (64, 56, 56, 64, 64), (1, 13, 13, 512, 512)):
        d = P.conv_desc(*shape, 3, 1, 1, 2, 2, B64L, B64L)
        assert P.ifq_conv_workspace_bytes(d) == 0, shape
    # forced splits: 64 KiB of counters, then ksplit partial tiles of
    # BM x BN int32 per tile (variant 0: 128 x 256 tiles, one K group)
    l4 = P.conv_desc(64, 7, 7, 512, 512, 3, 1, 1, 2, 2, B64L, B64L)
    for s in (2, 4):
        b = P.ifq_conv_split_workspace_bytes(l4, 0, s)
        assert b > 64 << 10 and (b - (64 << 10)) % (s * 128 * 256 * 4) == 0
    assert P.ifq_conv_split_workspace_bytes(l4, 0, 1) == 0   # not a split
    assert P.ifq_conv_split_workspace_bytes(l4, 0, 3) == 0   # 3 does not divide 8 blocks
    assert P.ifq_conv_split_workspace_bytes(l4, 2, 4) == 0   # 4 K groups x 4 > 8 blocks
    fp4 = [v for v in range(P.ifq_conv_variant_count()) if P.ifq_conv_variant_fp4(v) == 1]
    assert fp4 and all(P.ifq_conv_split_workspace_bytes(l4, v, 2) == 0 for v in fp4)
    i32 = P.conv_desc(64, 7, 7, 512, 512, 3, 1, 1, 2, 0, B64L, P.IFQ_LAYOUT_I32_NHWC)
    assert P.ifq_conv_split_workspace_bytes(i32, 0, 2) == 0  # threshold epilogue only


def test_split_rejects_small_workspace():
    lib = _ffi.load()
    l4 = P.conv_desc(64, 7, 7, 512, 512, 3, 1, 1, 2, 2, B64L, B64L)
    need = P.ifq_conv_split_workspace_bytes(l4, 0, 2)
    assert lib.ifq_conv_forward_split(ctypes.byref(l4), FAKE, FAKE, FAKE, FAKE, None, 0, 2,
                                      FAKE, need - 1, None) == EBUF
    assert lib.ifq_conv_forward_split(ctypes.byref(l4), FAKE, FAKE, FAKE, FAKE, None, 0, 3,
                                      FAKE, 1 << 30, None) == EUNSUP


@pytest.mark.parametrize("cfg", [0, 3, 4])
def test_stack_slots_follow_the_counter_region(cfg):
    # every stack's conv workspace, with the split counters at offset 0,
    # comes first, so that no stack's slots land on another's counters
    st, slots = make_stack(get_stack(cfg).layers, 2, "i8" if cfg == 4 else "b64")
    for name, k in slots.items():
        if k >= 2:
            off, nb = P.ifq_stack_slot_info(st, k)
            assert off >= 64 << 10
