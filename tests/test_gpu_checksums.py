"""GPU parity of encode, checksum convolutions and verification against the oracle."""
import numpy as np
import pytest
import torch

import paper_2003_12203_amd as ft
import workloads as wl
from gpu_util import TOL, assert_close_scaled, dev, gpu_flags, host, layer_for
from oracle import core
from oracle import workflow as wf

pytestmark = pytest.mark.gpu

SHAPES = [
    wl.config(0).layers[0],
    wl.config(1).layers[0].with_(n=3),
    wl.config(1).layers[2].with_(n=5),
    wl.config(3).layers[7].with_(n=4, h=28, w=28),     # 1x1 stride-2 projection, bf16
    wl.config(4).layers[14].with_(n=3),                # 1x1, 1024 channels
    wl.vgg19_bf16().layers[9].with_(n=2),
]


def _cfg_for(spec):
    return wl.Config(91, "ck", (spec,), "uniform", "he")


@pytest.mark.parametrize("spec", SHAPES, ids=lambda s: f"{s.ch}x{s.h}-{s.m}-r{s.r}u{s.stride}-{s.dtype}-n{s.n}")
@pytest.mark.parametrize("wbase", [0, 1])
def test_encode_checksum_conv_verify(spec, wbase):
    cfg = _cfg_for(spec)
    D, W = wl.gen_d(cfg, 0, spec), wl.gen_w(cfg, 0, spec)
    lay = layer_for(spec, wbase=wbase)
    lay.want_row_col()
    Dd, Wd = dev(D, spec.dtype), dev(W, spec.dtype)
    lay.encode_weights(Wd)
    lay.encode_input(Dd)
    O = lay.empty_output()
    lay.conv(Dd, Wd, O)
    lay.checksum_conv(ft.CO1 | ft.CO2 | ft.CO3 | ft.CO4 | ft.CO5 | ft.CO6 | ft.CO7, Dd, Wd)
    lay.verify(O)
    torch.cuda.synchronize()
    b = {k: v.cpu().numpy() for k, v in lay.buf.items()}

    cd1, cd2 = wf.encode(D, wbase)
    cw1, cw2 = wf.encode(W, wbase)
    # float64 sums of exact products: equal up to float64 rounding
    np.testing.assert_allclose(b["cd1"], cd1.ravel(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(b["cd2"], cd2.ravel(), rtol=1e-12, atol=1e-10)
    np.testing.assert_allclose(b["cw1"], cw1.ravel(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(b["cw2"], cw2.ravel(), rtol=1e-12, atol=1e-10)
    ck = wf.Checksums(cd1, cd2, cw1, cw2)
    wf.coc_checksums(ck, spec.stride, spec.pad)
    co1, co3 = wf.row_checksums(ck, W, spec.stride, spec.pad)
    co2, co4 = wf.col_checksums(ck, D, spec.stride, spec.pad)
    for name, ref in [("co5", ck.co5), ("co6", ck.co6), ("co7", ck.co7), ("co1", co1), ("co3", co3),
                      ("co2", co2), ("co4", co4)]:
        assert_close_scaled(b[name].reshape(ref.shape), ref, 1e-11, name)

    # verify: the oracle's summations over the GPU's own output
    Og = host(O)
    so5, so6, so7, q5, flags = wf.verify(Og, ck.co5, spec.ch * spec.r * spec.s, spec.dtype, wf.Policy(wbase=wbase))
    for name, ref in [("so5", so5), ("so6", so6), ("so7", so7), ("q5", q5)]:
        assert_close_scaled(b[name].reshape(ref.shape), ref, 1e-11, name)
    assert not flags.any(), "clean layer flagged by the oracle"
    assert not gpu_flags(lay).any(), "clean layer flagged by the GPU"
    rep = lay.read_report()
    assert not rep.detected and rep.n_flagged == 0 and rep.status == ft.STATUS_CLEAN
    # the GPU output itself agrees with the oracle's convolution
    ref_o = wf.store(core.conv(D, W, spec.stride, spec.pad), spec.dtype)
    assert_close_scaled(Og, ref_o, TOL[spec.dtype], "O")


def test_verify_is_deterministic():
    spec = wl.config(1).layers[1].with_(n=8)
    cfg = _cfg_for(spec)
    lay = layer_for(spec)
    Dd, Wd = dev(wl.gen_d(cfg, 0, spec), "f32"), dev(wl.gen_w(cfg, 0, spec), "f32")
    lay.encode_weights(Wd)
    lay.encode_input(Dd)
    O = lay.empty_output()
    lay.conv(Dd, Wd, O)
    lay.checksum_conv(ft.CO5 | ft.CO6 | ft.CO7)
    lay.verify(O)
    first = {k: lay.buf[k].clone() for k in ("so5", "so6", "so7", "q5", "cd1", "cd2")}
    lay.encode_input(Dd)
    lay.verify(O)
    torch.cuda.synchronize()
    for k, v in first.items():
        assert torch.equal(v, lay.buf[k]), k


def test_integer_checksums_exact():
    """Integer inputs: every checksum identity of Sec. 3 holds exactly on the GPU."""
    spec = wl.LayerSpec("int", 5, 6, 12, 12, 9, 3, 3, 1, 1, "f32")
    D, W = wl.gen_int_d(spec, 3), wl.gen_int_w(spec, 3)
    lay = layer_for(spec)
    Dd, Wd = dev(D, "f32"), dev(W, "f32")
    lay.encode_weights(Wd)
    lay.encode_input(Dd)
    O = lay.empty_output()
    lay.conv(Dd, Wd, O)
    lay.checksum_conv(ft.CO5 | ft.CO6 | ft.CO7)
    lay.verify(O)
    torch.cuda.synchronize()
    b = {k: v.cpu().numpy() for k, v in lay.buf.items()}
    np.testing.assert_array_equal(b["co5"], b["so5"])
    np.testing.assert_array_equal(b["co6"], b["so6"])
    np.testing.assert_array_equal(b["co7"], b["so7"])


def test_co6_alone_needs_no_cw1():
    """Co6 = Cd1 (x) Cw2 (Sec. 3.2) reads Cd1 and Cw2 only: asked for alone with ck->cw1 NULL,
    ftcnn_checksum_conv computes it without touching Cw1, and Co5/Co7 stay untouched."""
    spec = SHAPES[2]
    cfg = _cfg_for(spec)
    D, W = wl.gen_d(cfg, 0, spec), wl.gen_w(cfg, 0, spec)
    lay = layer_for(spec)
    Dd, Wd = dev(D, spec.dtype), dev(W, spec.dtype)
    lay.encode_weights(Wd)
    lay.encode_input(Dd)
    for k in ("co5", "co6", "co7"):
        lay.buf[k].fill_(-7.0)
    ck = ft._lib.Checksums()
    for k, t in lay.buf.items():
        setattr(ck, k, t.data_ptr())
    ck.cw1 = None
    ft.checksum_conv(lay.desc, ft.CO6, None, None, ck)
    torch.cuda.synchronize()
    cd1, cd2 = wf.encode(D, 0)
    cw1, cw2 = wf.encode(W, 0)
    c = wf.Checksums(cd1, cd2, cw1, cw2)
    wf.coc_checksums(c, spec.stride, spec.pad)
    got = lay.buf["co6"].cpu().numpy().reshape(c.co6.shape)
    assert_close_scaled(got, c.co6, 1e-11, "co6")
    assert (lay.buf["co5"] == -7.0).all() and (lay.buf["co7"] == -7.0).all()
