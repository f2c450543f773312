"""libquan's C ABI on the host: the library loads, exports every symbol that
include/quan.h declares, and rejects every invalid argument with its error
code and a message before it makes any HIP call (these run without a GPU:
the pointers below are never dereferenced)."""
import ctypes
import os
import re

import pytest

from paper_2509_05512_amd import quan

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "quan.h")

OK, E_NULL, E_SHAPE, E_DTYPE, E_ALIGN, E_ALIAS, E_UNSUP = 0, -1, -2, -3, -4, -5, -6


def declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"QUAN_API\s+[^;(]*?\b(quan_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(quan.LIB_PATH):
        pytest.skip("libquan.so not built")
    return quan.load_library()


def test_header_declares_expected_entry_points():
    syms = declared_symbols()
    for name in ["quan_qconv2d_forward", "quan_iqbn_forward", "quan_iqbn_relu_forward",
                 "quan_last_error", "quan_release", "quan_version"]:
        assert name in syms


def test_library_exports_every_declared_symbol(lib):
    for name in declared_symbols():
        assert hasattr(lib, name), f"libquan.so does not export {name}"
    assert set(quan.SIGNATURES) == set(declared_symbols())


def test_version(lib):
    assert "gfx950" in quan.quan_version()


# Fake, 256-byte-aligned, disjoint "device" addresses; never dereferenced.
X, WR, WI, WJ, WK, B, OUT = (0x10000000 * (i + 1) for i in range(7))
G, BE, MEAN, VAR = (0x90000000 + 0x100000 * i for i in range(4))


def conv(lib, fn="quan_qconv2d_forward", **kw):
    a = dict(x=X, wr=WR, wi=WI, wj=WJ, wk=WK, bias=B, sh=1, sw=1, ph=1, pw=1, dh=1, dw=1,
             out=OUT, n=2, cin=4, h=16, w=16, cout=4, kh=3, kw=3, dtype=1)
    a.update(kw)
    rc = getattr(lib, fn)(a["x"], a["wr"], a["wi"], a["wj"], a["wk"], a["bias"],
                          a["sh"], a["sw"], a["ph"], a["pw"], a["dh"], a["dw"], a["out"],
                          a["n"], a["cin"], a["h"], a["w"], a["cout"], a["kh"], a["kw"],
                          a["dtype"], None)
    return rc, lib.quan_last_error().decode()


def iqbn(lib, relu=False, fn_name=None, **kw):
    a = dict(x=X, g=G, b=BE, eps=1e-5, out=OUT, mean=MEAN, var=VAR, n=2, c=4, h=8, w=8, dtype=1)
    a.update(kw)
    fn = getattr(lib, fn_name) if fn_name else (lib.quan_iqbn_relu_forward if relu else lib.quan_iqbn_forward)
    rc = fn(a["x"], a["g"], a["b"], a["eps"], a["out"], a["mean"], a["var"], a["n"], a["c"],
            a["h"], a["w"], a["dtype"], None)
    return rc, lib.quan_last_error().decode()


CONV_ERRORS = [
    ("null x", dict(x=None), E_NULL),
    ("null w_j", dict(wj=None), E_NULL),
    ("null out", dict(out=None), E_NULL),
    ("bad dtype", dict(dtype=7), E_DTYPE),
    ("n = 0", dict(n=0), E_SHAPE),
    ("c_in = 0", dict(cin=0), E_SHAPE),
    ("c_out < 0", dict(cout=-3), E_SHAPE),
    ("k = 0", dict(kh=0), E_SHAPE),
    ("stride 0", dict(sh=0), E_SHAPE),
    ("dilation 0", dict(dw=0), E_SHAPE),
    ("negative pad", dict(pw=-1), E_SHAPE),
    ("kernel wider than input", dict(w=2, pw=0), E_SHAPE),
    ("dilated span too big", dict(h=5, ph=0, dh=3), E_SHAPE),
    ("x misaligned", dict(x=X + 8), E_ALIGN),
    ("out misaligned", dict(out=OUT + 4), E_ALIGN),
    ("bf16 weight odd address", dict(wr=WR + 1), E_ALIGN),
    ("fp32 bias 2-byte aligned", dict(bias=B + 2, dtype=0), E_ALIGN),
    ("out overlaps x", dict(out=X + 256), E_ALIAS),
    ("out overlaps weight", dict(out=WK - 256), E_ALIAS),
    ("out overlaps bias", dict(out=B), E_ALIAS),
    ("input too large", dict(n=1 << 16, h=256, w=256, cin=64), E_UNSUP),
    ("image beyond 32-bit tile offsets", dict(n=1, h=4096, w=4096, cin=16, dtype=0), E_UNSUP),
]


@pytest.mark.parametrize("fn", ["quan_qconv2d_forward", "quan_qconv2d_separable_forward"])
@pytest.mark.parametrize("name,kw,code", CONV_ERRORS, ids=[c[0] for c in CONV_ERRORS])
def test_qconv2d_rejects(lib, name, kw, code, fn):
    rc, msg = conv(lib, fn, **kw)
    assert rc == code, (name, rc, msg)
    assert msg, "an error must leave a message"


def fused(lib, **kw):
    a = dict(x=X, packed=WR, bias=B, sh=1, sw=1, ph=1, pw=1, dh=1, dw=1, g=G, b=BE, eps=1e-5, relu=0,
             stats=0, out=OUT, mean=MEAN, var=VAR, n=2, cin=4, h=16, w=16, cout=4, kh=3, kw=3, dtype=1)
    a.update(kw)
    rc = lib.quan_qconv2d_iqbn_forward(a["x"], a["packed"], a["bias"], a["sh"], a["sw"], a["ph"], a["pw"],
                                       a["dh"], a["dw"], a["g"], a["b"], a["eps"], a["relu"], a["stats"],
                                       a["out"],
                                       a["mean"], a["var"], a["n"], a["cin"], a["h"], a["w"], a["cout"],
                                       a["kh"], a["kw"], a["dtype"], None)
    return rc, lib.quan_last_error().decode()


FUSED_ERRORS = [
    ("null packed", dict(packed=None), E_NULL),
    ("null gamma", dict(g=None), E_NULL),
    ("null var", dict(var=None), E_NULL),
    ("bad dtype", dict(dtype=5), E_DTYPE),
    ("c_out = 0", dict(cout=0), E_SHAPE),
    ("eps = 0", dict(eps=0.0), E_SHAPE),
    ("relu = 2", dict(relu=2), E_SHAPE),
    ("stats mode 3", dict(stats=3), E_SHAPE),
    ("stats mode -1", dict(stats=-1), E_SHAPE),
    ("packed misaligned", dict(packed=WR + 8), E_ALIGN),
    ("mean misaligned", dict(mean=MEAN + 2), E_ALIGN),
    ("out overlaps packed", dict(out=WR), E_ALIAS),
    ("mean overlaps var", dict(var=MEAN + 4), E_ALIAS),
    ("mean inside out", dict(mean=OUT + 64), E_ALIAS),
]


@pytest.mark.parametrize("name,kw,code", FUSED_ERRORS, ids=[c[0] for c in FUSED_ERRORS])
def test_fused_conv_iqbn_rejects(lib, name, kw, code):
    rc, msg = fused(lib, **kw)
    assert rc == code, (name, rc, msg)
    assert msg


def infer(lib, **kw):
    a = dict(x=X, packed=WR, bias=B, sh=1, sw=1, ph=1, pw=1, dh=1, dw=1, m=MEAN, v=VAR, g=G, b=BE,
             eps=1e-5, relu=0, out=OUT, n=2, cin=4, h=16, w=16, cout=4, kh=3, kw=3, dtype=1)
    a.update(kw)
    rc = lib.quan_qconv2d_iqbn_inference(a["x"], a["packed"], a["bias"], a["sh"], a["sw"], a["ph"],
                                         a["pw"], a["dh"], a["dw"], a["m"], a["v"], a["g"], a["b"],
                                         a["eps"], a["relu"], a["out"], a["n"], a["cin"], a["h"], a["w"],
                                         a["cout"], a["kh"], a["kw"], a["dtype"], None)
    return rc, lib.quan_last_error().decode()


INFER_ERRORS = [
    ("null packed", dict(packed=None), E_NULL),
    ("null running mean", dict(m=None), E_NULL),
    ("null running var", dict(v=None), E_NULL),
    ("null beta", dict(b=None), E_NULL),
    ("bad dtype", dict(dtype=7), E_DTYPE),
    ("k = 0", dict(kh=0), E_SHAPE),
    ("eps = 0", dict(eps=0.0), E_SHAPE),
    ("eps nan", dict(eps=float("nan")), E_SHAPE),
    ("relu = -1", dict(relu=-1), E_SHAPE),
    ("packed misaligned", dict(packed=WR + 4), E_ALIGN),
    ("var misaligned", dict(v=VAR + 1), E_ALIGN),
    ("out overlaps packed", dict(out=WR), E_ALIAS),
    ("mean inside out", dict(m=OUT + 128), E_ALIAS),
    ("gamma inside out", dict(g=OUT + 4), E_ALIAS),
]


@pytest.mark.parametrize("name,kw,code", INFER_ERRORS, ids=[c[0] for c in INFER_ERRORS])
def test_inference_conv_iqbn_rejects(lib, name, kw, code):
    rc, msg = infer(lib, **kw)
    assert rc == code, (name, rc, msg)
    assert msg


POINCARE_ERRORS = [
    ("null rgb", dict(rgb=None), E_NULL),
    ("null out", dict(out=None), E_NULL),
    ("bad dtype", dict(dtype=2), E_DTYPE),
    ("h = 0", dict(h=0), E_SHAPE),
    ("n < 0", dict(n=-1), E_SHAPE),
    ("too large", dict(n=1 << 12, h=1024, w=1024), E_UNSUP),
    ("rgb misaligned", dict(rgb=X + 1), E_ALIGN),
    ("out misaligned", dict(out=OUT + 2), E_ALIGN),
    ("out overlaps rgb", dict(out=X + 64), E_ALIAS),
]


@pytest.mark.parametrize("name,kw,code", POINCARE_ERRORS, ids=[c[0] for c in POINCARE_ERRORS])
def test_poincare_rejects(lib, name, kw, code):
    a = dict(rgb=X, out=OUT, n=2, h=16, w=16, dtype=1)
    a.update(kw)
    rc = lib.quan_poincare_map(a["rgb"], a["out"], a["n"], a["h"], a["w"], a["dtype"], None)
    assert rc == code, (name, rc, lib.quan_last_error())
    assert lib.quan_last_error()


DX, DG, DB = 0xA0000000, 0xA8000000, 0xA8100000
DW0, DW1, DW2, DW3 = (0xB0000000 + 0x100000 * i for i in range(4))


def stem(lib, **kw):
    a = dict(rgb=X, packed=WR, bias=B, sh=2, sw=2, ph=1, pw=1, dh=1, dw=1, out=OUT, n=2, h=16, w=16, cout=16,
             kh=3, kw=3, dtype=1)
    a.update(kw)
    rc = lib.quan_qconv2d_poincare_forward(a["rgb"], a["packed"], a["bias"], a["sh"], a["sw"], a["ph"], a["pw"],
                                           a["dh"], a["dw"], a["out"], a["n"], a["h"], a["w"], a["cout"], a["kh"],
                                           a["kw"], a["dtype"], None)
    return rc, lib.quan_last_error().decode()


STEM_ERRORS = [
    ("null rgb", dict(rgb=None), E_NULL),
    ("null packed", dict(packed=None), E_NULL),
    ("bad dtype", dict(dtype=2), E_DTYPE),
    ("c_out = 0", dict(cout=0), E_SHAPE),
    ("empty output", dict(h=1, ph=0), E_SHAPE),
    ("rgb off its element", dict(rgb=X + 1), E_ALIGN),
    ("out misaligned", dict(out=OUT + 8), E_ALIGN),
    ("packed misaligned", dict(packed=WR + 8), E_ALIGN),
    ("out overlaps rgb", dict(out=X + 256), E_ALIAS),
    ("out overlaps packed", dict(out=WR - 256), E_ALIAS),
]


@pytest.mark.parametrize("name,kw,code", STEM_ERRORS, ids=[c[0] for c in STEM_ERRORS])
def test_poincare_stem_rejects(lib, name, kw, code):
    rc, msg = stem(lib, **kw)
    assert rc == code, (name, rc, msg)
    assert msg


def bwd_data(lib, fn="quan_qconv2d_backward_data", **kw):
    a = dict(dy=OUT, wr=WR, wi=WI, wj=WJ, wk=WK, sh=1, sw=1, ph=1, pw=1, dh=1, dw=1, dx=DX, n=2, cin=4, h=16, w=16,
             cout=4, kh=3, kw=3, dtype=1)
    a.update(kw)
    rc = getattr(lib, fn)(a["dy"], a["wr"], a["wi"], a["wj"], a["wk"], a["sh"], a["sw"], a["ph"],
                                        a["pw"], a["dh"], a["dw"], a["dx"], a["n"], a["cin"], a["h"], a["w"],
                                        a["cout"], a["kh"], a["kw"], a["dtype"], None)
    return rc, lib.quan_last_error().decode()


def bwd_weight(lib, fn="quan_qconv2d_backward_weight", **kw):
    a = dict(x=X, dy=OUT, sh=1, sw=1, ph=1, pw=1, dh=1, dw=1, d0=DW0, d1=DW1, d2=DW2, d3=DW3, db=DB, n=2, cin=4,
             h=16, w=16, cout=4, kh=3, kw=3, dtype=1)
    a.update(kw)
    rc = getattr(lib, fn)(a["x"], a["dy"], a["sh"], a["sw"], a["ph"], a["pw"], a["dh"], a["dw"],
                                          a["d0"], a["d1"], a["d2"], a["d3"], a["db"], a["n"], a["cin"], a["h"],
                                          a["w"], a["cout"], a["kh"], a["kw"], a["dtype"], None)
    return rc, lib.quan_last_error().decode()


BWD_DATA_ERRORS = [
    ("null dy", dict(dy=None), E_NULL),
    ("null w_k", dict(wk=None), E_NULL),
    ("null dx", dict(dx=None), E_NULL),
    ("bad dtype", dict(dtype=3), E_DTYPE),
    ("stride 0", dict(sh=0), E_SHAPE),
    ("pad beyond the kernel span", dict(ph=3), E_UNSUP),
    ("dx misaligned", dict(dx=DX + 2), E_ALIGN),
    ("weight misaligned", dict(wi=WI + 1), E_ALIGN),
    ("dx overlaps dy", dict(dx=OUT + 64), E_ALIAS),
    ("dx overlaps a kernel", dict(dx=WJ - 64), E_ALIAS),
]


@pytest.mark.parametrize("fn", ["quan_qconv2d_backward_data", "quan_qconv2d_separable_backward_data"])
@pytest.mark.parametrize("name,kw,code", BWD_DATA_ERRORS, ids=[c[0] for c in BWD_DATA_ERRORS])
def test_backward_data_rejects(lib, name, kw, code, fn):
    rc, msg = bwd_data(lib, fn=fn, **kw)
    assert rc == code, (name, rc, msg)
    assert msg


BWD_WEIGHT_ERRORS = [
    ("null x", dict(x=None), E_NULL),
    ("null dw_j", dict(d2=None), E_NULL),
    ("bad dtype", dict(dtype=-2), E_DTYPE),
    ("k = 0", dict(kw=0), E_SHAPE),
    ("dw misaligned", dict(d1=DW1 + 2), E_ALIGN),
    ("db misaligned", dict(db=DB + 1), E_ALIGN),
    ("dw overlaps x", dict(d0=X + 4), E_ALIAS),
    ("db overlaps dy", dict(db=OUT + 4), E_ALIAS),
    ("dw overlap each other", dict(d3=DW2 + 4), E_ALIAS),
]


@pytest.mark.parametrize("fn", ["quan_qconv2d_backward_weight", "quan_qconv2d_separable_backward_weight"])
@pytest.mark.parametrize("name,kw,code", BWD_WEIGHT_ERRORS, ids=[c[0] for c in BWD_WEIGHT_ERRORS])
def test_backward_weight_rejects(lib, name, kw, code, fn):
    rc, msg = bwd_weight(lib, fn=fn, **kw)
    assert rc == code, (name, rc, msg)
    assert msg


def iqbn_bwd(lib, **kw):
    a = dict(x=X, dout=OUT, y=B, m=MEAN, v=VAR, g=G, eps=1e-5, dx=DX, dg=DG, db=DB, n=2, c=4, h=8, w=8, dtype=1)
    a.update(kw)
    rc = lib.quan_iqbn_backward(a["x"], a["dout"], a["y"], a["m"], a["v"], a["g"], a["eps"], a["dx"], a["dg"],
                                a["db"], a["n"], a["c"], a["h"], a["w"], a["dtype"], None)
    return rc, lib.quan_last_error().decode()


IQBN_BWD_ERRORS = [
    ("null x", dict(x=None), E_NULL),
    ("null dout", dict(dout=None), E_NULL),
    ("null var", dict(v=None), E_NULL),
    ("null dgamma", dict(dg=None), E_NULL),
    ("bad dtype", dict(dtype=9), E_DTYPE),
    ("w = 0", dict(w=0), E_SHAPE),
    ("eps = 0", dict(eps=0.0), E_SHAPE),
    ("too large", dict(n=1 << 14, h=512, w=512), E_UNSUP),
    ("dout misaligned", dict(dout=OUT + 2), E_ALIGN),
    ("y misaligned", dict(y=B + 8), E_ALIGN),
    ("dbeta misaligned", dict(db=DB + 1), E_ALIGN),
    ("dx overlaps x", dict(dx=X + 32), E_ALIAS),
    ("dx partially overlaps dout", dict(dx=OUT + 16), E_ALIAS),
    ("dgamma inside dx", dict(dg=DX + 64), E_ALIAS),
    ("dgamma overlaps dbeta", dict(db=DG + 8), E_ALIAS),
]


@pytest.mark.parametrize("name,kw,code", IQBN_BWD_ERRORS, ids=[c[0] for c in IQBN_BWD_ERRORS])
def test_iqbn_backward_rejects(lib, name, kw, code):
    rc, msg = iqbn_bwd(lib, **kw)
    assert rc == code, (name, rc, msg)
    assert msg


IQBN_ERRORS = [
    ("null gamma", dict(g=None), E_NULL),
    ("null var", dict(var=None), E_NULL),
    ("bad dtype", dict(dtype=-1), E_DTYPE),
    ("c = 0", dict(c=0), E_SHAPE),
    ("h = 0", dict(h=0), E_SHAPE),
    ("eps = 0", dict(eps=0.0), E_SHAPE),
    ("eps < 0", dict(eps=-1.0), E_SHAPE),
    ("eps nan", dict(eps=float("nan")), E_SHAPE),
    ("x misaligned", dict(x=X + 2), E_ALIGN),
    ("mean misaligned", dict(mean=MEAN + 2), E_ALIGN),
    ("out partially overlaps x", dict(out=X + 16), E_ALIAS),
    ("mean overlaps var", dict(var=MEAN + 4), E_ALIAS),
    ("var inside x", dict(var=X + 64), E_ALIAS),
    ("too large", dict(n=1 << 14, h=512, w=512, c=4), E_UNSUP),
]


@pytest.mark.parametrize("fn_name", ["quan_iqbn_forward", "quan_iqbn_relu_forward", "quan_iqbn_forward_noalloc"])
@pytest.mark.parametrize("name,kw,code", IQBN_ERRORS, ids=[c[0] for c in IQBN_ERRORS])
def test_iqbn_rejects(lib, name, kw, code, fn_name):
    rc, msg = iqbn(lib, fn_name=fn_name, **kw)
    assert rc == code, (name, rc, msg)
    assert msg


def test_iqbn_noalloc_rejects_more_scratch_than_it_holds(lib):
    """12288 rows of 4000 columns: 512 statistics blocks per column group
    need (2 * 512 + 3) * 4000 floats = 16.4 MB of scratch, beyond the fixed
    8 MiB array; refused before any device work, with a message naming the
    sizes.  quan_iqbn_forward (which allocates) accepts the same arguments
    up to the same point, i.e. the shape itself is valid."""
    rc, msg = iqbn(lib, fn_name="quan_iqbn_forward_noalloc", n=1, c=1000, h=128, w=96)
    assert rc == E_UNSUP and "scratch" in msg, (rc, msg)


def test_error_message_is_per_call(lib):
    rc, msg = conv(lib, x=None)
    assert rc == E_NULL and "non-NULL" in msg
    rc, msg = iqbn(lib, eps=0.0)
    assert rc == E_SHAPE and "eps" in msg


def test_release_without_use(lib):
    assert lib.quan_release() == OK


def test_binding_layout_helpers():
    import torch
    x = torch.randn(2, 4, 3, 5, 6)
    y = quan.to_device_layout(x)
    assert torch.equal(x, y)
    assert quan.is_device_layout(y)
    assert not quan.is_device_layout(x)
    assert y.stride() == quan.device_strides(2, 3, 5, 6)
    e = quan.empty_qmap(2, 3, 5, 6, torch.float32, "cpu")
    assert quan.is_device_layout(e) and tuple(e.shape) == (2, 4, 3, 5, 6)


# ---- descriptor entry points: layout, shape and dtype from (shape, strides) --

E_LAYOUT = -9


def qt(addr, shape, strides=None, dtype=1):
    """A quan_tensor with dense row-major strides unless given."""
    d = quan.QuanTensor()
    d.data = addr or 0
    d.dtype = dtype
    d.ndim = len(shape)
    if strides is None:
        strides, step = [0] * len(shape), 1
        for i in range(len(shape) - 1, -1, -1):
            strides[i] = step
            step *= shape[i]
    for i, (n, st) in enumerate(zip(shape, strides)):
        d.shape[i] = n
        d.strides[i] = st
    return d


def qmap(addr, n, c, h, w, dtype=1):
    """A [N, 4, C, H, W] map stored channels-last by component."""
    return qt(addr, (n, 4, c, h, w), quan.device_strides(n, c, h, w), dtype)


def conv_desc(lib, **kw):
    a = dict(x=qmap(X, 2, 4, 16, 16), wr=qt(WR, (4, 4, 3, 3)), wi=qt(WI, (4, 4, 3, 3)),
             wj=qt(WJ, (4, 4, 3, 3)), wk=qt(WK, (4, 4, 3, 3)), bias=qt(B, (4, 4)),
             stride=(1, 1), pad=(1, 1), dil=(1, 1), out=qmap(OUT, 2, 4, 16, 16))
    a.update(kw)
    ref = lambda d: ctypes.byref(d) if d is not None else None
    pair = lambda p: (ctypes.c_int32 * 2)(*p) if p is not None else None
    rc = lib.quan_qconv2d_forward_desc(ref(a["x"]), ref(a["wr"]), ref(a["wi"]), ref(a["wj"]), ref(a["wk"]),
                                       ref(a["bias"]), pair(a["stride"]), pair(a["pad"]), pair(a["dil"]),
                                       ref(a["out"]), None)
    return rc, lib.quan_last_error().decode()


CONV_DESC_ERRORS = [
    ("x NCHW-ordered memory", dict(x=qt(X, (2, 4, 4, 16, 16))), E_LAYOUT),
    ("x NHWC but component-minor", dict(x=qt(X, (2, 4, 4, 16, 16), (4096, 1, 4, 256, 16))), E_LAYOUT),
    ("out NCHW-ordered memory", dict(out=qt(OUT, (2, 4, 4, 16, 16))), E_LAYOUT),
    ("w_k OHWI strides", dict(wk=qt(WK, (4, 4, 3, 3), (36, 1, 12, 4))), E_LAYOUT),
    ("bias transposed", dict(bias=qt(B, (4, 4), (1, 4))), E_LAYOUT),
    ("x ndim 4", dict(x=qt(X, (2, 16, 16, 16))), E_SHAPE),
    ("x 3 components", dict(x=qt(X, (2, 3, 4, 16, 16), (3072, 4, 1, 192, 12))), E_SHAPE),
    ("w_i c_in mismatch", dict(wi=qt(WI, (4, 5, 3, 3))), E_SHAPE),
    ("w_j k mismatch", dict(wj=qt(WJ, (4, 4, 5, 5))), E_SHAPE),
    ("bias extent", dict(bias=qt(B, (4, 5))), E_SHAPE),
    ("out wrong Ho", dict(out=qmap(OUT, 2, 4, 15, 16)), E_SHAPE),
    ("out wrong c_out", dict(out=qmap(OUT, 2, 8, 16, 16)), E_SHAPE),
    ("empty output", dict(pad=(0, 0), x=qmap(X, 2, 4, 2, 16), out=qmap(OUT, 2, 4, 1, 14)), E_SHAPE),
    ("stride 0", dict(stride=(0, 1)), E_SHAPE),
    ("x bad dtype", dict(x=qmap(X, 2, 4, 16, 16, dtype=5)), E_DTYPE),
    ("w_j f32 with bf16 x", dict(wj=qt(WJ, (4, 4, 3, 3), dtype=0)), E_DTYPE),
    ("out f32 with bf16 x", dict(out=qmap(OUT, 2, 4, 16, 16, dtype=0)), E_DTYPE),
    ("NULL x descriptor", dict(x=None), E_NULL),
    ("NULL x data", dict(x=qmap(0, 2, 4, 16, 16)), E_NULL),
    ("NULL w_r descriptor", dict(wr=None), E_NULL),
    ("NULL out", dict(out=None), E_NULL),
    ("NULL stride", dict(stride=None), E_NULL),
    ("extent 2^31", dict(x=qmap(X, 2 ** 31, 4, 16, 16)), E_UNSUP),
    # descriptors accepted, then the plain entry point's own checks
    ("x misaligned", dict(x=qmap(X + 2, 2, 4, 16, 16)), E_ALIGN),
    ("out overlaps x", dict(out=qmap(X + 256, 2, 4, 16, 16)), E_ALIAS),
    # an axis of extent 1 is never stepped: its stride is not checked
    ("unit axis, any stride", dict(x=qt(X + 2, (1, 4, 4, 16, 16), (7, 4, 1, 256, 16)),
                                   out=qmap(OUT, 1, 4, 16, 16)), E_ALIGN),
]


@pytest.mark.parametrize("name,kw,code", CONV_DESC_ERRORS, ids=[c[0] for c in CONV_DESC_ERRORS])
def test_qconv2d_desc_rejects(lib, name, kw, code):
    rc, msg = conv_desc(lib, **kw)
    assert rc == code, (name, rc, msg)
    assert msg


def iqbn_desc(lib, relu=False, **kw):
    a = dict(x=qmap(X, 2, 4, 8, 8), g=qt(G, (4, 4), dtype=0), b=qt(BE, (4, 4), dtype=0), eps=1e-5,
             out=qmap(OUT, 2, 4, 8, 8), mean=qt(MEAN, (4, 4), dtype=0), var=qt(VAR, (4, 4), dtype=0))
    a.update(kw)
    ref = lambda d: ctypes.byref(d) if d is not None else None
    fn = lib.quan_iqbn_relu_forward_desc if relu else lib.quan_iqbn_forward_desc
    rc = fn(ref(a["x"]), ref(a["g"]), ref(a["b"]), a["eps"], ref(a["out"]), ref(a["mean"]), ref(a["var"]),
            None)
    return rc, lib.quan_last_error().decode()


IQBN_DESC_ERRORS = [
    ("x NCHW-ordered memory", dict(x=qt(X, (2, 4, 4, 8, 8))), E_LAYOUT),
    ("out NCHW-ordered memory", dict(out=qt(OUT, (2, 4, 4, 8, 8))), E_LAYOUT),
    ("gamma transposed", dict(g=qt(G, (4, 4), (1, 4), dtype=0)), E_LAYOUT),
    ("var strided", dict(var=qt(VAR, (4, 4), (8, 1), dtype=0)), E_LAYOUT),
    ("x ndim 3", dict(x=qt(X, (2, 4, 64))), E_SHAPE),
    ("out shape differs", dict(out=qmap(OUT, 2, 4, 8, 9)), E_SHAPE),
    ("mean extent", dict(mean=qt(MEAN, (4, 5), dtype=0)), E_SHAPE),
    ("beta ndim", dict(b=qt(BE, (16,), dtype=0)), E_SHAPE),
    ("gamma bf16", dict(g=qt(G, (4, 4), dtype=1)), E_DTYPE),
    ("out dtype differs", dict(out=qmap(OUT, 2, 4, 8, 8, dtype=0)), E_DTYPE),
    ("x bad dtype", dict(x=qmap(X, 2, 4, 8, 8, dtype=9)), E_DTYPE),
    ("NULL var", dict(var=None), E_NULL),
    ("NULL gamma data", dict(g=qt(0, (4, 4), dtype=0)), E_NULL),
    ("eps 0", dict(eps=0.0), E_SHAPE),
    ("x misaligned", dict(x=qmap(X + 8, 2, 4, 8, 8)), E_ALIGN),
    ("mean overlaps var", dict(mean=qt(VAR + 4, (4, 4), dtype=0)), E_ALIAS),
]


@pytest.mark.parametrize("relu", [False, True])
@pytest.mark.parametrize("name,kw,code", IQBN_DESC_ERRORS, ids=[c[0] for c in IQBN_DESC_ERRORS])
def test_iqbn_desc_rejects(lib, name, kw, code, relu):
    rc, msg = iqbn_desc(lib, relu=relu, **kw)
    assert rc == code, (name, rc, msg)
    assert msg


def test_descriptor_of_torch_tensors():
    import torch
    x = quan.empty_qmap(2, 3, 5, 6, torch.bfloat16, "cpu")
    d = quan.describe(x)
    assert d.ndim == 5 and d.dtype == quan.QUAN_BF16
    assert tuple(d.shape[:5]) == (2, 4, 3, 5, 6)
    assert tuple(d.strides[:5]) == quan.device_strides(2, 3, 5, 6)
    w = torch.zeros(4, 3, 3, 3)
    dw = quan.describe(w)
    assert dw.ndim == 4 and dw.dtype == quan.QUAN_F32 and tuple(dw.strides[:4]) == (27, 9, 3, 1)
    assert quan.describe(None) is None
