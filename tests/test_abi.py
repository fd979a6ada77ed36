"""The C ABI on the host: the library loads, exports every declared entry point, and rejects bad
arguments before touching a device (no GPU needed)."""
import ctypes as C
import os
import re

import pytest

import paper_2003_12203_amd as ft
from paper_2003_12203_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ftcnn.h")


def declared():
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:int|size_t|const char \*)\s*(ftcnn_\w+)\s*\(", txt, re.M)))


def test_library_exports_every_declared_symbol():
    L = _lib.load()
    names = declared()
    assert len(names) >= 11, names
    for n in names:
        assert hasattr(L, n), n
    assert sorted(_lib.EXPORTS) == names


def test_struct_sizes_match_header_layout():
    assert C.sizeof(_lib.ConvDesc) == 12 * 4
    assert C.sizeof(_lib.Checksums) == 17 * 8   # 15 checksum arrays, the bias and its sums
    assert C.sizeof(_lib.ReportHeader) == 14 * 4
    assert C.sizeof(_lib.Fix) == 5 * 4
    assert C.sizeof(_lib.Policy) == 4 * 4 + 2 * 8
    assert C.sizeof(_lib.Fault) == 6 * 4 + 8
    assert ft.report_bytes(0) == C.sizeof(_lib.ReportHeader)
    assert ft.report_bytes(7) == C.sizeof(_lib.ReportHeader) + 7 * C.sizeof(_lib.Fix)


def test_checksums_field_order_matches_header():
    import re
    text = open(os.path.join(ROOT, "include", "ftcnn.h")).read()
    body = text[text.index("typedef struct {\n    double *cd1"):text.index("} ftcnn_checksums;")]
    body = re.sub(r"/\*.*?\*/", "", body, flags=re.S)
    names = re.findall(r"\*\s*(\w+)", body)
    assert names == [f[0] for f in _lib.Checksums._fields_]


@pytest.mark.parametrize("h,r,u,p,e", [(227, 11, 4, 0, 55), (224, 7, 2, 3, 112), (56, 1, 2, 0, 28),
                                       (13, 3, 1, 1, 13), (416, 3, 1, 1, 416), (3, 3, 1, 0, 1)])
def test_out_shape(h, r, u, p, e):
    d = ft.make_desc(2, 3, h, h, 4, r, r, u, p)
    assert ft.out_shape(d) == (e, e)
    assert ft.workspace_bytes(d) > 0
    assert ft.workspace_bytes(d) % 256 == 0


def test_non_square():
    d = ft.make_desc(1, 2, 13, 11, 3, 3, 5, 1, 2)
    assert ft.out_shape(d) == (15, 11)


@pytest.mark.parametrize("kw,code", [
    (dict(n=0), -2), (dict(stride=0), -2), (dict(pad=-1), -2), (dict(r=20), -2),
    (dict(groups=2), -2), (dict(groups=0), -2), (dict(ch=4, m=6, groups=4), -2),
    (dict(dtype_raw=7), -3), (dict(wbase=2), -1),
])
def test_bad_descriptor(kw, code):
    args = dict(n=2, ch=3, h=8, w=8, m=4, r=3, s=3, stride=1, pad=0, groups=1, dtype=ft.F32, wbase=0)
    if "dtype_raw" in kw:
        args["dtype"] = kw.pop("dtype_raw")
    args.update(kw)
    d = _lib.ConvDesc(args["n"], args["ch"], args["h"], args["w"], args["m"], args["r"], args["s"],
                      args["stride"], args["pad"], args["groups"], args["dtype"], args["wbase"])
    E, F = C.c_int32(), C.c_int32()
    assert _lib.load().ftcnn_out_shape(C.byref(d), C.byref(E), C.byref(F)) == code
    assert ft.workspace_bytes(d) == 0
    assert ft.last_error()


def test_bf16_filter_count_bound():
    """The bf16 epilogue's fp32 runs are exact only while every weight m + wbase stays within
    2^16: 65536 filters pass with wbase 0, not with wbase 1; fp32 layers have no such bound."""
    ok = ft.make_desc(1, 1, 4, 4, 65536, 1, 1, dtype="bf16")
    assert ft.out_shape(ok) == (4, 4)
    over = ft.make_desc(1, 1, 4, 4, 65536, 1, 1, dtype="bf16", wbase=1)
    E, F = C.c_int32(), C.c_int32()
    assert _lib.load().ftcnn_out_shape(C.byref(over), C.byref(E), C.byref(F)) == -6
    assert "65536" in ft.last_error()
    assert ft.out_shape(ft.make_desc(1, 1, 4, 4, 65537, 1, 1, dtype="f32")) == (4, 4)


def test_grouped_descriptor_accepted():
    d = ft.make_desc(2, 4, 8, 8, 6, 3, 3, groups=2)
    assert ft.out_shape(d) == (6, 6)
    dense = ft.workspace_bytes(ft.make_desc(2, 4, 8, 8, 6, 3, 3))
    assert ft.workspace_bytes(d) > dense   # room for the block-diagonal expansion of W


def test_null_pointers_rejected_without_launch():
    L = _lib.load()
    d = ft.make_desc(2, 3, 8, 8, 4, 3, 3)
    assert L.ftcnn_conv_fwd(C.byref(d), None, None, None, None) == -1
    assert L.ftcnn_encode(C.byref(d), 0, None, None, None, None, None) == -1
    assert L.ftcnn_encode(C.byref(d), 5, C.c_void_p(16), C.c_void_p(16), C.c_void_p(16), None, None) == -1
    ck = _lib.Checksums()
    pol = ft.make_policy()
    assert L.ftcnn_verify(C.byref(d), C.c_void_p(256), C.byref(ck), C.byref(pol), C.c_void_p(256), 4,
                          C.c_void_p(256), None) == -1
    bad = ft.make_policy(kappa=-1.0)
    assert L.ftcnn_verify(C.byref(d), C.c_void_p(256), C.byref(ck), C.byref(bad), C.c_void_p(256), 4,
                          C.c_void_p(256), None) == -1
    assert L.ftcnn_checksum_conv(C.byref(d), 1 << 9, None, None, C.byref(ck), None) == -1
    f = (_lib.Fault * 1)(_lib.Fault(5, 0, 0, 0, 0, 3, 0.0))
    assert L.ftcnn_inject(C.byref(d), C.c_void_p(256), f, 1, None) == -1   # n out of range
    f = (_lib.Fault * 1)(_lib.Fault(0, 0, 0, 0, 0, 40, 0.0))
    assert L.ftcnn_inject(C.byref(d), C.c_void_p(256), f, 1, None) == -1   # bit out of range
    assert L.ftcnn_inject(C.byref(d), C.c_void_p(256), f, 65, None) == -1
    ws_mis = C.c_void_p(256 + 8)
    assert L.ftcnn_verify(C.byref(d), C.c_void_p(256), C.byref(ck), C.byref(pol), C.c_void_p(256), 4,
                          ws_mis, None) == -1  # ck arrays missing are reported first


def test_relu_pool_rejects_bad_arguments_without_launch():
    L = _lib.load()
    X, Y = C.c_void_p(1 << 20), C.c_void_p(1 << 24)
    assert L.ftcnn_relu_pool(ft.F32, 2, 3, 8, 8, 4, 4, X, Y, None) == -6      # window not built
    assert L.ftcnn_relu_pool(ft.F32, 2, 3, 8, 8, 3, 1, X, Y, None) == -6
    assert L.ftcnn_relu_pool(7, 2, 3, 8, 8, 2, 2, X, Y, None) == -3           # dtype
    assert L.ftcnn_relu_pool(ft.BF16, 2, 0, 8, 8, 2, 2, X, Y, None) == -2     # empty
    assert L.ftcnn_relu_pool(ft.BF16, 2, 3, 2, 8, 3, 2, X, Y, None) == -2     # map below the window
    assert L.ftcnn_relu_pool(ft.F32, 2, 3, 8, 8, 2, 2, None, Y, None) == -1
    # pooling in place (or into an overlapping range) would read windows already overwritten
    assert L.ftcnn_relu_pool(ft.F32, 2, 3, 8, 8, 2, 2, X, X, None) == -1
    assert L.ftcnn_relu_pool(ft.F32, 2, 3, 8, 8, 2, 2, X, C.c_void_p((1 << 20) + 4 * 2 * 3 * 64 - 4), None) == -1


def test_relu_pool_encode_rejects_bad_arguments_without_launch():
    L = _lib.load()
    X, Y, c = C.c_void_p(1 << 20), C.c_void_p(1 << 24), C.c_void_p(1 << 28)
    assert L.ftcnn_relu_pool_encode(ft.F32, 2, 3, 8, 8, 2, 2, 0, X, Y, None, c, None) == -1
    assert L.ftcnn_relu_pool_encode(ft.F32, 2, 3, 8, 8, 2, 2, 2, X, Y, c, c, None) == -1     # wbase
    assert L.ftcnn_relu_pool_encode(ft.F32, 2, 3, 8, 8, 3, 1, 0, X, Y, c, c, None) == -6
    assert L.ftcnn_relu_pool_encode(ft.F32, 2, 3, 8, 8, 2, 2, 0, X, X, c, c, None) == -1     # overlap
    d = ft.make_desc(2, 32, 8, 8, 16, 3, 3, 1, 1)
    ck = _lib.Checksums()
    rep = C.c_void_p(256)
    # the given checksums are required
    assert L.ftcnn_conv_fwd_sums_given(C.byref(d), X, X, Y, C.byref(ck), rep, 4, None, 0, C.c_void_p(256),
                                       None) == -1
    assert L.ftcnn_conv_fwd_sums_given(C.byref(d), X, X, Y, None, rep, 4, None, 0, C.c_void_p(256), None) == -1


def test_chain_shapes_checked_on_host():
    from paper_2003_12203_amd import network
    assert network.pooling(55, 27) == (3, 2) and network.pooling(224, 112) == (2, 2)
    assert network.pooling(13, 13) == (1, 1)
    with pytest.raises(ft.FtcnnError):
        network.pooling(8, 3)


def test_chain_links_and_mismatches_on_host():
    """network.Chain works out the operations between layers on the host (no device work): ReLU
    alone for equal sizes, AlexNet's 3x3/2 and VGG's 2x2/2 pooling, and it rejects layers that do
    not feed each other."""
    from paper_2003_12203_amd import network
    vgg = [(2, 3, 16, 16, 8, 3, 3, 1, 1), (2, 8, 16, 16, 8, 3, 3, 1, 1), (2, 8, 8, 8, 4, 3, 3, 1, 1)]
    assert network.Chain(vgg, "f32", device="cpu").links == [(1, 1), (2, 2)]
    alex = [(2, 3, 29, 29, 8, 5, 5, 2, 0), (2, 8, 6, 6, 4, 3, 3, 1, 1)]   # 13 -> 3x3/2 -> 6
    assert network.Chain(alex, "f32", device="cpu").links == [(3, 2)]
    with pytest.raises(ft.FtcnnError):   # 8 filters feed a layer of 6 channels
        network.Chain([(2, 3, 16, 16, 8, 3, 3, 1, 1), (2, 6, 16, 16, 8, 3, 3, 1, 1)], "f32", device="cpu")
    with pytest.raises(ft.FtcnnError):   # 16 -> 7: no 2x2/2 or 3x3/2 pooling fits exactly
        network.Chain([(2, 3, 16, 16, 8, 3, 3, 1, 1), (2, 8, 7, 7, 8, 3, 3, 1, 1)], "f32", device="cpu")


def test_noalloc_rejects_layers_beyond_the_static_scratch_without_launch():
    """ftcnn_protected_conv_noalloc checks the layer's scratch need against its static array (128 MiB)
    on the host, before any device work: 1024 images x 1024 filters of 64 x 64 outputs need about
    1 GiB of epilogue partial sums even without channels-last copies."""
    L = _lib.load()
    d = ft.make_desc(1024, 32, 64, 64, 1024, 1, 1)
    ck = _lib.Checksums()
    pol = ft.make_policy()
    p = C.c_void_p(256)
    assert L.ftcnn_protected_conv_noalloc(C.byref(d), p, p, p, C.byref(ck), C.byref(pol), p, 4, None) == -4
    assert "static scratch" in ft.last_error()
    # a bad descriptor is still a shape error
    bad = ft.make_desc(0, 3, 8, 8, 4, 3, 3)
    assert L.ftcnn_protected_conv_noalloc(C.byref(bad), p, p, p, C.byref(ck), C.byref(pol), p, 4, None) == -2
